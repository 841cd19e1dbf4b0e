"""Full-size parity in the launch configuration of bench.py.

Every step of a workload runs on the GPU through ``retro_step`` captured in a
HIP graph and replayed (as bench.py times it).  The CPU oracle runs the same
steps' page selection (scores, top-k, Alg. 2), and every step's page scores, selection,
mask M, last_loaded A and sequence lengths must match bit for bit.  Outputs are
checked on sampled window rows at sampled steps against a brute-force fp64
softmax over the exact set of tokens that row has attended so far, derived here
from the selection history by the set form of eq. (update-sup) (a page is
eligible for a past query if it was not selected at any step since that query,
and holds no key newer than it): the full oracle attention would take minutes
at these sizes.
"""
from __future__ import annotations

import sys
import time
from typing import List, Optional

import numpy as np

import oracle
import workloads as W
from gpu_harness import TOL, _gpu_layer, compare_scores
from oracle_shadow import softmax_attend


def attended_tokens(sel_hist: List[np.ndarray], num_hist: List[np.ndarray],
                    len_hist: List[np.ndarray], b: int, h: int, tau: int, t: int, P: int):
    """Token positions window row tau has attended by the end of step t."""
    qpos = int(len_hist[tau][b]) - 1
    seen_pages = set()
    toks = set()
    for m in range(tau, t + 1):
        L = int(len_hist[m][b])
        S = set(int(p) for p in sel_hist[m][b, h, :num_hist[m][b, h]])
        if m == tau:
            pages = S
        else:
            pages = {p for p in S - seen_pages if min((p + 1) * P, L) - 1 <= qpos}
        for p in pages:
            toks.update(range(p * P, min((p + 1) * P, L)))
        seen_pages |= S
    return toks


def run_full(spec, steps: Optional[int] = None, *, check_steps=None, rows_per_check: int = 48,
             graph: bool = True, label: str = "", flags: int = 0) -> int:
    import torch
    steps = spec.steps if steps is None else steps
    if check_steps is None:  # the window's ramp-up, eight evenly spaced steps, the last
        check_steps = {steps - 1, min(steps - 1, spec.window)} | {i * steps // 8 for i in range(1, 8)}
    check_steps = set(check_steps)
    tol = TOL[spec.dtype]
    print(f"[full] {label or spec.name}: batch={spec.batch} hk={spec.num_kv_heads} G={spec.group} "
          f"d={spec.head_dim} P={spec.page_size} B={spec.budget} W={spec.window} steps={steps} "
          f"graph={graph}", flush=True)
    t_start = time.time()
    gen = W.Generator(spec)
    orc = oracle.Oracle.for_spec(spec)
    layer = _gpu_layer(spec, None, flags=flags)
    for b, (k, v) in enumerate(gen.prefill()):
        orc.prefill(b, k, v)
        layer.prefill(b, k, v)
    qw = W.QueryWindow(spec)
    tdt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
    scale = 1.0 / np.sqrt(spec.head_dim)
    G, Wn, P = spec.group, spec.window, spec.page_size
    rng = np.random.default_rng(4242)
    sel_hist, num_hist, len_hist = [], [], []
    rows_checked, worst_o, worst_z = 0, 0.0, 0.0
    for t in range(steps):
        k_new, v_new, q = gen.step(t)
        win = qw.push(q).copy()
        ref = orc.step(t, k_new, v_new, win, attend=False)
        T = k_new.shape[0]
        for j in range(T - 1):
            layer.append(t, k_new[j], v_new[j])
        win_d = torch.from_numpy(win).to("cuda", tdt)
        kn_d = torch.from_numpy(np.ascontiguousarray(k_new[-1])).to("cuda", tdt)
        vn_d = torch.from_numpy(np.ascontiguousarray(v_new[-1])).to("cuda", tdt)
        if graph:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                layer.step(t, win_d, kn_d, vn_d)
            g.replay()
        else:
            layer.step(t, win_d, kn_d, vn_d)
        torch.cuda.synchronize()
        compare_scores(t, layer, ref)
        sel = layer.selected.cpu().numpy()
        num = layer.num_selected.cpu().numpy()
        assert np.array_equal(num, ref["num_selected"]), f"step {t}: num_selected differs"
        if not np.array_equal(sel, ref["selected"]):
            bad = np.argwhere(sel != ref["selected"])[:5]
            raise AssertionError(f"step {t}: selected pages differ at {bad.tolist()}")
        assert np.array_equal(layer.mask.cpu().numpy(), ref["mask"]), f"step {t}: mask M differs"
        assert np.array_equal(layer.last_loaded.cpu().numpy(), orc.A), f"step {t}: A differs"
        lens = layer.seq_lens.cpu().numpy()
        assert np.array_equal(lens, ref["seq_lens"]), f"step {t}: seq_lens differ"
        sel_hist.append(sel.copy())
        num_hist.append(num.copy())
        len_hist.append(lens.copy())
        if t in check_steps:
            o = layer.o_out.cpu().numpy().astype(np.float64)
            z = layer.lse_out.cpu().numpy().astype(np.float64)
            for _ in range(rows_per_check):
                b = int(rng.integers(spec.batch))
                qh = int(rng.integers(spec.num_q_heads))
                r = int(rng.integers(Wn + 1))
                tau = t - Wn + r
                if tau < 0:
                    assert np.all(o[b, r, qh] == 0.0) and z[b, r, qh] == -np.inf, \
                        f"step {t}: row {r} before the first step is not empty"
                    continue
                h = qh // G
                toks = attended_tokens(sel_hist, num_hist, len_hist, b, h, tau, t, P)
                eo_ref, ez_ref = softmax_attend(win[b, r, qh], orc.K[b, h], orc.V[b, h], toks, scale)
                if not toks:
                    assert z[b, r, qh] == -np.inf, f"step {t}: empty row {r} has Z {z[b, r, qh]}"
                    continue
                eo = float(np.max(np.abs(o[b, r, qh] - eo_ref)))
                ez = abs(float(z[b, r, qh]) - float(ez_ref))
                worst_o, worst_z = max(worst_o, eo), max(worst_z, ez)
                rows_checked += 1
                assert eo <= tol, f"step {t} row (b={b}, qh={qh}, r={r}): max |dO| = {eo:.3g} > {tol}"
                assert ez <= tol, f"step {t} row (b={b}, qh={qh}, r={r}): |dZ| = {ez:.3g} > {tol}"
        if (t + 1) % 512 == 0:
            print(f"[full] {label or spec.name}: step {t + 1}/{steps} ({time.time() - t_start:.0f} s)",
                  flush=True)
    print(f"[full] {label or spec.name}: ok, {steps} steps bit-exact selection; {rows_checked} sampled "
          f"rows, max|dO|={worst_o:.3g} max|dZ|={worst_z:.3g} ({time.time() - t_start:.0f} s)",
          flush=True)
    sys.stdout.flush()
    return rows_checked
