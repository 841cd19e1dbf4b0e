"""GPU parity of retro_append_kv_tokens (AppendKV of Alg. 1 for several tokens per
sequence in one call) against the oracle's one-token appends in order: the
stored keys and values, the page digests (Sec. 2.1), last_loaded (Alg. 2's
current-page rule) and seq_lens, bit for bit; and whole decode steps of the
long-generation workload (8 tokens per step) with the step's first 7 tokens
appended in one call.  The drop at an unmapped page (no page table in the
oracle) is checked against the one-token entry point, which drops the same way.
"""
import numpy as np
import pytest

import oracle
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


def _state(layer):
    import torch
    torch.cuda.synchronize()
    return dict(kc=layer.k_cache.float().cpu().numpy(), vc=layer.v_cache.float().cpu().numpy(),
                pt=layer.page_table.cpu().numpy(), dg=layer.digest.float().cpu().numpy(),
                A=layer.last_loaded.cpu().numpy(), lens=layer.seq_lens.cpu().numpy())


def _compare_with_oracle(layer, orc, P, label):
    s = _state(layer)
    assert np.array_equal(s["lens"], orc.seq_lens), f"{label}: seq_lens"
    assert np.array_equal(s["A"], orc.A), f"{label}: last_loaded"
    for b, n in enumerate(s["lens"]):
        pos = np.arange(int(n))
        ph = s["pt"][b, pos // P]
        slot = pos % P
        k = s["kc"][ph, :, slot, :]          # [n][h_k][d]
        v = s["vc"][ph, :, :, slot]          # [n][h_k][d]
        assert np.array_equal(k.transpose(1, 0, 2), orc.K[b, :, :n]), f"{label}: keys of seq {b}"
        assert np.array_equal(v.transpose(1, 0, 2), orc.V[b, :, :n]), f"{label}: values of seq {b}"
        npg = -(-int(n) // P)
        assert np.array_equal(s["dg"][b, :, :npg, 0], orc.kmin[b, :, :npg]), f"{label}: digest min {b}"
        assert np.array_equal(s["dg"][b, :, :npg, 1], orc.kmax[b, :, :npg]), f"{label}: digest max {b}"


def _tokens(rng, n, spec):
    shape = (n, spec.batch, spec.num_kv_heads, spec.head_dim)
    k = rng.standard_normal(shape, dtype=np.float32)
    v = rng.standard_normal(shape, dtype=np.float32)
    if spec.dtype == "bf16":
        k, v = W.round_bf16(k), W.round_bf16(v)
    return k, v


@pytest.mark.parametrize("cfg", [0, 1])
def test_append_tokens_matches_sequential_oracle_appends(cfg):
    """Calls that start mid-page (slot 13), cross page boundaries and exceed one
    64-token launch, on a shuffled page table; fp32 (tiny) and bf16 (Llama-class
    heads) caches."""
    from paper_2508_09001_amd.layer import RetroLayer
    import torch
    base = W.config(cfg)
    spec = base.replace(batch=2, prefill=(29, 45), steps=3, tokens_per_step=60)
    rng = np.random.default_rng(11 + cfg)
    perm = rng.permutation(spec.batch * spec.max_pages).astype(np.int32)
    layer = RetroLayer.for_spec(spec, page_table=torch.from_numpy(perm.reshape(spec.batch, -1)))
    orc = oracle.Oracle.for_spec(spec)
    for b, n0 in enumerate(spec.prefill):
        k, v = _tokens(rng, n0, spec.replace(batch=1))
        orc.prefill(b, k[:, 0], v[:, 0])
        layer.prefill(b, k[:, 0], v[:, 0])
    _compare_with_oracle(layer, orc, spec.page_size, "prefill")
    for step, n in [(0, 7), (1, 70), (2, 1), (3, 0)]:
        k, v = _tokens(rng, n, spec)
        for j in range(n):
            orc.append(step, k[j], v[j])
        layer.append_tokens(step, k, v)
        _compare_with_oracle(layer, orc, spec.page_size, f"{n} tokens at step {step}")


def test_append_tokens_drop_at_unmapped_page_like_one_token_appends():
    """A call running into an unmapped logical page appends the tokens before it
    and drops the rest, leaving seq_lens at the page's start, as the same tokens
    appended one call each do."""
    from paper_2508_09001_amd.layer import RetroLayer
    import torch
    spec = W.config(0).replace(batch=2, prefill=(29, 10), steps=2, tokens_per_step=40)
    P = spec.page_size
    pt = np.arange(spec.batch * spec.max_pages, dtype=np.int32).reshape(spec.batch, -1)
    pt[0, 3] = -1                      # sequence 0: positions 48..63 unmapped
    pt[1, 2] = spec.batch * spec.max_pages + 5   # sequence 1: page 2 past the pool
    rng = np.random.default_rng(5)
    layers = [RetroLayer.for_spec(spec, page_table=torch.from_numpy(pt.copy())) for _ in range(2)]
    for b, n0 in enumerate(spec.prefill):
        k, v = _tokens(rng, n0, spec.replace(batch=1))
        for lay in layers:
            lay.prefill(b, k[:, 0], v[:, 0])
    k, v = _tokens(rng, 40, spec)
    layers[0].append_tokens(1, k, v)
    for j in range(40):
        layers[1].append(1, k[j], v[j])
    a, b_ = _state(layers[0]), _state(layers[1])
    assert a["lens"].tolist() == [3 * P, 2 * P] == b_["lens"].tolist()
    for key in ("kc", "vc", "dg", "A"):
        assert np.array_equal(a[key], b_[key]), key


@pytest.mark.timeout(900)
def test_long_generation_steps_with_multi_token_appends():
    """Whole decode steps of the long-generation workload (batch 4, 8 tokens per
    step): the first 7 tokens of every step through one retro_append_kv_tokens
    call, the last through retro_step; selections, masks, A, seq_lens and scores
    bit for bit, outputs within tolerance, on a shuffled page table."""
    spec = W.config(3)
    run_parity(spec, 24, page_perm_seed=4, multi_append=True,
               label="long-generation b4, 7 tokens per call + step token, 24 steps")
