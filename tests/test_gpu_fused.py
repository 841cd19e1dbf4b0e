"""GPU parity of the single-launch step (RETRO_STEP_FUSED=1) against the CPU
oracle, to the same bar as the multi-launch step: selections, masks, A and
sequence lengths bit for bit; outputs and log-normalisers within 2e-3 (bf16)
and 1e-5 (fp32) max-abs.  Shapes the single launch does not cover fall back to
the multi-launch step inside the library and are still checked."""
import pytest

import workloads as W
from gpu_harness import run_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_09001_amd import binding
    binding.load_library()


@pytest.fixture(autouse=True)
def _fused(monkeypatch):
    monkeypatch.setenv("RETRO_STEP_FUSED", "1")


def test_fused_tiny_fp32():
    run_parity(W.config(0), W.config(0).steps, label="fused tiny-fp32")


def test_fused_llama_layer_32k_shuffled():
    run_parity(W.config(1), 24, page_perm_seed=4, label="fused 32k shuffled")


def test_fused_batched_serving_ragged():
    run_parity(W.config(2), 10, page_perm_seed=2, label="fused batch16 ragged")


def test_fused_long_generation_multi_token_steps():
    spec = W.config(3).replace(batch=2, prefill=(16384, 16384))
    run_parity(spec, 24, label="fused long-generation b2 8 tok/step")


@pytest.mark.parametrize("budget,window", [(1024, 0), (8192, 64)])
def test_fused_extreme_context(budget, window):
    spec = W.config(4).replace(budget=budget, window=window)
    run_parity(spec, 6, label=f"fused 131k B={budget} W={window}")


def test_fused_short_sequences_and_partial_pages():
    spec = W.Spec("edge-short", batch=3, num_kv_heads=2, group=3, head_dim=64, page_size=16,
                  budget=64, window=5, steps=20, dtype="bf16", prefill=(1, 17, 40), seed=9)
    run_parity(spec, 20, page_perm_seed=3, label="fused edge short")


def test_fused_fp32_head_dim_128_many_rows():
    spec = W.Spec("edge-f32-d128", batch=1, num_kv_heads=2, group=8, head_dim=128, page_size=16,
                  budget=512, window=20, steps=24, dtype="f32", prefill=(3000,), seed=12)
    run_parity(spec, 24, label="fused edge f32 d128 R=168")
