"""retro_step_noalloc (the step with the library's static scratch as its
workspace) against retro_step with a workspace of its own: the same inputs give
the same outputs and state, bit for bit, on two workloads in a row, the second
smaller (another geometry: the static scratch is cleared for it)."""
from __future__ import annotations

import pytest

import workloads as W

pytestmark = pytest.mark.gpu


def _pair_steps(spec, steps, label):
    import numpy as np
    import torch
    from gpu_harness import _gpu_layer
    ref, na = _gpu_layer(spec, 5), _gpu_layer(spec, 5)
    gen = W.Generator(spec)
    for b, (k, v) in enumerate(gen.prefill()):
        ref.prefill(b, k, v)
        na.prefill(b, k, v)
    qw = W.QueryWindow(spec)
    for t in range(steps):
        k_new, v_new, q = gen.step(t)
        win = qw.push(q).copy()
        for lay in (ref, na):
            for jj in range(k_new.shape[0] - 1):
                lay.append(t, k_new[jj], v_new[jj])
        print(f"[noalloc] {label} step {t}", flush=True)
        ref.step(t, win, k_new[-1], v_new[-1])
        na.step(t, win, k_new[-1], v_new[-1], noalloc=True)
        torch.cuda.synchronize()
        for name in ("o_out", "lse_out", "selected", "mask", "num_selected", "last_loaded",
                     "seq_lens", "o_cache", "lse_cache"):
            a = getattr(ref, name).cpu().numpy()
            b = getattr(na, name).cpu().numpy()
            assert np.array_equal(a, b, equal_nan=True), f"{label} step {t}: {name} differs"
        assert np.isfinite(ref.o_out.cpu().numpy()).all(), f"{label} step {t}: non-finite output"


def test_noalloc_step_matches_retro_step():
    spec = W.config(1)
    _pair_steps(spec, spec.window + 3, "32k layer")
    # a smaller workload right after: another geometry on the same static scratch
    _pair_steps(W.config(0), 6, "tiny fp32")


def test_noalloc_rejects_a_step_beyond_its_scratch():
    import ctypes as C
    from paper_2508_09001_amd import binding as B
    # a workload whose workspace exceeds the static scratch: refused before any launch
    spec = W.config(1).replace(batch=160, prefill=(32768,) * 160)
    dims = B.Dims(spec.batch, spec.num_kv_heads, spec.group, spec.head_dim, spec.page_size,
                  spec.budget, spec.window, spec.max_pages, spec.batch * spec.max_pages,
                  B.RETRO_BF16, 0.0, 0, 0)
    assert B.retro_workspace_size(dims) > 64 << 20
    st = B.load_library().retro_step_noalloc(C.byref(dims), 0, None, None, None,
                                             C.byref(B.KVCache()), C.byref(B.Selection()),
                                             C.byref(B.OutputCache()), None, None, None)
    assert st == B.RETRO_ESCRATCH, B.retro_status_string(st)
