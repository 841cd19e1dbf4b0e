"""Drive the GPU library and the CPU oracle side by side on the same seeded inputs."""
from __future__ import annotations

import sys
from typing import Optional

import numpy as np

import oracle
import workloads as W

TOL = {"bf16": 2e-3, "f32": 1e-5}   # max-abs on outputs and log-normalisers


def _gpu_layer(spec, page_perm_seed: Optional[int], device="cuda", flags: int = 0,
               pool_pages: Optional[int] = None, page_table: Optional[np.ndarray] = None):
    """A RetroLayer for spec.  page_perm_seed: logical pages map to a seeded random
    choice of distinct physical pages (a shuffled table) from a pool of pool_pages
    physical pages (default batch * max_pages); page_table: that table given
    explicitly, [batch][max_pages]."""
    import torch
    from paper_2508_09001_amd.layer import RetroLayer
    pt = None
    pool = spec.batch * spec.max_pages if pool_pages is None else pool_pages
    if page_table is not None:
        pt = torch.from_numpy(np.ascontiguousarray(page_table, np.int32))
    elif page_perm_seed is not None:
        rng = np.random.default_rng(page_perm_seed)
        perm = rng.permutation(pool)[:spec.batch * spec.max_pages].astype(np.int32)
        pt = torch.from_numpy(perm.reshape(spec.batch, spec.max_pages))
    return RetroLayer.for_spec(spec, page_table=pt, device=device, flags=flags,
                               num_phys_pages=pool)


class Stats:
    def __init__(self):
        self.o = 0.0
        self.z = 0.0
        self.steps = 0
        self.rows_checked = 0


def compare_scores(t, layer, ref):
    """The step's page scores, eq. (quest_score) in the fixed fp32 order, bit for bit
    on every page of every sequence (steps that keep the selection of an earlier
    step, with top-k reuse, score nothing and are skipped)."""
    if ref.get("scores") is None:
        return
    s = layer.scores().cpu().numpy()
    P = layer.P
    for b, L in enumerate(ref["seq_lens"]):
        n = -(-int(L) // P)
        got = s[b, :, :n].view(np.uint32)
        want = np.ascontiguousarray(ref["scores"][b, :, :n]).view(np.uint32)
        if not np.array_equal(got, want):
            bad = np.argwhere(got != want)[:5]
            raise AssertionError(f"step {t}: page scores of sequence {b} differ at (head, page) "
                                 f"{bad.tolist()}")


def compare_step(t, layer, ref, tol, stats: Stats, outputs=True):
    import torch
    torch.cuda.synchronize()
    compare_scores(t, layer, ref)
    sel = layer.selected.cpu().numpy()
    num = layer.num_selected.cpu().numpy()
    msk = layer.mask.cpu().numpy()
    A = layer.last_loaded.cpu().numpy()
    assert np.array_equal(num, ref["num_selected"]), f"step {t}: num_selected differs"
    if not np.array_equal(sel, ref["selected"]):
        bad = np.argwhere(sel != ref["selected"])[:5]
        raise AssertionError(f"step {t}: selected pages differ at {bad.tolist()}")
    assert np.array_equal(msk, ref["mask"]), f"step {t}: mask M differs"
    assert np.array_equal(A, ref["A"]), f"step {t}: last_loaded (A) differs"
    assert np.array_equal(layer.seq_lens.cpu().numpy(), ref["seq_lens"]), f"step {t}: seq_lens"
    if outputs:
        o = layer.o_out.cpu().numpy().astype(np.float64)
        z = layer.lse_out.cpu().numpy().astype(np.float64)
        zr = ref["lse_out"]
        fin = np.isfinite(zr)
        assert np.array_equal(fin, np.isfinite(z)), f"step {t}: empty-row pattern differs"
        assert np.all(z[~fin] == -np.inf)
        eo = float(np.max(np.abs(o - ref["o_out"])))
        ez = float(np.max(np.abs(z[fin] - zr[fin]), initial=0.0))
        stats.o = max(stats.o, eo)
        stats.z = max(stats.z, ez)
        stats.rows_checked += int(fin.sum())
        assert eo <= tol, f"step {t}: max |O - O_ref| = {eo:.3g} > {tol}"
        assert ez <= tol, f"step {t}: max |Z - Z_ref| = {ez:.3g} > {tol}"
    stats.steps += 1


def reembedded_kv(orc, n: int, rng, dtype: str):
    """Synthetic UpdateKV inputs: the n most recent stored keys / values of every
    sequence, perturbed by 5 % (keys) and 10 % (values) of their rms, the size of
    one retrospective update's change the paper reports for keys and values
    (appendix, evolving query representations); [batch][n][h_k][d]."""
    b_, hk, d = orc.batch, orc.hk, orc.d
    ku = np.zeros((b_, n, hk, d), np.float32)
    vu = np.zeros((b_, n, hk, d), np.float32)
    for b in range(b_):
        L = int(orc.seq_lens[b])
        for j in range(n):
            pos = L - n + j
            if pos < 0:
                continue
            k, v = orc.K[b, :, pos], orc.V[b, :, pos]
            ku[b, j] = k + 0.05 * np.sqrt(np.mean(k * k)) * rng.standard_normal(k.shape)
            vu[b, j] = v + 0.10 * np.sqrt(np.mean(v * v)) * rng.standard_normal(v.shape)
    if dtype == "bf16":
        ku, vu = W.round_bf16(ku), W.round_bf16(vu)
    return ku.astype(np.float32), vu.astype(np.float32)


def run_parity(spec, steps: int, *, page_perm_seed: Optional[int] = None, split_calls=False,
               check_outputs_from: int = 0, tol: Optional[float] = None, label: str = "",
               update_kv: bool = False, flags: int = 0,
               pool_pages: Optional[int] = None,
               page_table: Optional[np.ndarray] = None, multi_append: bool = False) -> Stats:
    """Run `steps` decode steps on GPU and oracle; compare every step's selection,
    mask and A exactly, and the outputs of the steps >= check_outputs_from (the
    oracle runs attention only from check_outputs_from - W on, which is enough
    for the cached rows it then checks)."""
    import torch
    tol = TOL[spec.dtype] if tol is None else tol
    print(f"[parity] {label or spec.name}: batch={spec.batch} hk={spec.num_kv_heads} "
          f"G={spec.group} d={spec.head_dim} P={spec.page_size} B={spec.budget} W={spec.window} "
          f"steps={steps} tps={spec.tokens_per_step} perm={page_perm_seed} split={split_calls} "
          f"update_kv={update_kv} flags={flags} pool={pool_pages} multi_append={multi_append}",
          flush=True)
    gen = W.Generator(spec)
    orc = oracle.Oracle.for_spec(spec)
    layer = _gpu_layer(spec, page_perm_seed, flags=flags, pool_pages=pool_pages,
                       page_table=page_table)
    for b, (k, v) in enumerate(gen.prefill()):
        orc.prefill(b, k, v)
        layer.prefill(b, k, v)
    qw = W.QueryWindow(spec)
    stats = Stats()
    attend_from = max(0, check_outputs_from - spec.window)
    rng_upd = np.random.default_rng(1234)
    for t in range(steps):
        k_new, v_new, q = gen.step(t)
        win = qw.push(q).copy()
        if update_kv and spec.window > 0 and t > 0:
            # UpdateKV of the window's past tokens, before the step's append (Alg. 1)
            ku, vu = reembedded_kv(orc, spec.window, rng_upd, spec.dtype)
            orc.update_kv(ku, vu)
            layer.update_kv(ku, vu)
        ref = orc.step(t, k_new, v_new, win, attend=t >= attend_from)
        ref["A"] = orc.A
        T = k_new.shape[0]
        if multi_append and T > 1:  # the tokens before the last in one call
            layer.append_tokens(t, k_new[:-1], v_new[:-1])
        else:
            for j in range(T - 1):
                layer.append(t, k_new[j], v_new[j])
        if split_calls:
            layer.append(t, k_new[-1], v_new[-1])
            layer.select(t, win[:, -1])
            layer.attend(t, win)
            layer.merge(t)
        else:
            layer.step(t, win, k_new[-1], v_new[-1])
        compare_step(t, layer, ref, tol, stats, outputs=t >= check_outputs_from)
    torch.cuda.synchronize()
    print(f"[parity] {label or spec.name}: ok, max|dO|={stats.o:.3g} max|dZ|={stats.z:.3g} "
          f"over {stats.rows_checked} rows", flush=True)
    sys.stdout.flush()
    return stats
