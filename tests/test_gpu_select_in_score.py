"""GPU parity of the step with the page selection at the end of the score
launch (RETRO_SELECT_IN_SCORE=1) instead of in front of the attention, on
shapes whose default step selects in the attention launch.  Same bar as the
other parity tests: selections, masks, A and sequence lengths bit for bit;
outputs and log-normalisers within 2e-3 (bf16) and 1e-5 (fp32) max-abs."""
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
def _select_in_score(monkeypatch):
    monkeypatch.setenv("RETRO_SELECT_IN_SCORE", "1")


def test_select_in_score_tiny_fp32():
    run_parity(W.config(0), W.config(0).steps, label="select-in-score tiny-fp32")


def test_select_in_score_llama_layer_32k_shuffled():
    run_parity(W.config(1), 24, page_perm_seed=4, label="select-in-score 32k shuffled")


def test_select_in_score_batched_serving_ragged():
    run_parity(W.config(2), 10, page_perm_seed=2, label="select-in-score batch16 ragged")


def test_select_in_score_short_sequences_and_partial_pages():
    spec = W.Spec("edge-short", batch=3, num_kv_heads=2, group=3, head_dim=64, page_size=16,
                  budget=64, window=5, steps=20, dtype="bf16", prefill=(1, 17, 40), seed=9)
    run_parity(spec, 20, page_perm_seed=3, label="select-in-score edge short")
