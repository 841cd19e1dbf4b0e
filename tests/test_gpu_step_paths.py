"""GPU parity of the step's other launch sequences, on shapes whose default
step runs scores, selection and attention in one launch, chosen through
retro_dims.flags: the scores in a launch of their own with the selection in
front of the attention (RETRO_FLAG_SEPARATE_SCORES), and the selection at the
end of the score launch (RETRO_FLAG_SELECT_IN_SCORES).  Same bar as the other
parity tests: scores, selections, masks, A and sequence lengths bit for bit;
outputs and log-normalisers within 2e-3 (bf16) and 1e-5 (fp32) max-abs."""
import pytest

import workloads as W
from gpu_harness import run_parity

pytestmark = pytest.mark.gpu

PATHS = {"separate-scores": 1, "select-in-scores": 2}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2508_09001_amd import binding
    binding.load_library()


@pytest.fixture(params=sorted(PATHS))
def path(request):
    return request.param


def test_path_tiny_fp32(path):
    run_parity(W.config(0), W.config(0).steps, flags=PATHS[path], label=f"{path} tiny-fp32")


def test_path_llama_layer_32k_shuffled(path):
    run_parity(W.config(1), 24, page_perm_seed=4, flags=PATHS[path], label=f"{path} 32k shuffled")


def test_path_batched_serving_ragged(path):
    run_parity(W.config(2), 10, page_perm_seed=2, flags=PATHS[path],
               label=f"{path} batch16 ragged")


def test_path_short_sequences_and_partial_pages(path):
    spec = W.Spec("edge-short", batch=3, num_kv_heads=2, group=3, head_dim=64, page_size=16,
                  budget=64, window=5, steps=20, dtype="bf16", prefill=(1, 17, 40), seed=9)
    run_parity(spec, 20, page_perm_seed=3, flags=PATHS[path], label=f"{path} edge short")
