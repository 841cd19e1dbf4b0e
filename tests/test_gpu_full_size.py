"""GPU parity at the workloads' full sizes and step counts, with every step
captured in a HIP graph and replayed (the launch configuration of bench.py).
Selections, masks, A and sequence lengths are checked bit for bit at every
step; outputs on sampled rows against brute-force softmax over each row's
attended tokens (tests/full_size.py)."""
import pytest

import workloads as W
from full_size import run_full

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_09001_amd import binding
    binding.load_library()


def test_full_tiny_fp32():
    assert run_full(W.config(0), label="full tiny-fp32") > 0


def test_full_llama_layer_32k():
    assert run_full(W.config(1), label="full 32k") > 0


def test_full_batched_serving():
    # outputs of sampled rows at every one of the 128 steps
    spec = W.config(2)
    assert run_full(spec, check_steps=set(range(spec.steps)), label="full batch16") > 0


@pytest.mark.timeout(900)
def test_full_long_generation():
    # 16384 -> 49152 tokens over 4096 steps, 8 tokens per step, batch 4; outputs
    # of sampled rows at the window's ramp-up and every 64th step
    spec = W.config(3)
    checks = {spec.window} | set(range(63, spec.steps, 64))
    assert run_full(spec, check_steps=checks, rows_per_check=16, label="full long-generation") > 0


@pytest.mark.parametrize("budget", [1024, 2048, 4096, 8192])
@pytest.mark.parametrize("window", [0, 4, 16, 64])
def test_full_extreme_context(budget, window):
    spec = W.config(4).replace(budget=budget, window=window)
    assert run_full(spec, check_steps={spec.steps - 1}, rows_per_check=32,
                    label=f"full 131k B={budget} W={window}") > 0


def test_full_extreme_context_dense():
    # budget covering the whole context: every page selected, the current row is dense attention
    spec = W.config(4).replace(budget=131072 + 4096, window=4)
    assert run_full(spec, check_steps={spec.steps - 1}, rows_per_check=32,
                    label="full 131k dense") > 0


def test_full_llama_layer_32k_separate_score_launch():
    # the three-launch sequence (scores, selection + attention, combine) at full length
    assert run_full(W.config(1), flags=1, label="full 32k separate scores") > 0
