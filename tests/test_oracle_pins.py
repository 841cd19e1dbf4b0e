"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's formulas: each compares it with a
hand-worked fixture (tests/golden), a closed form, a textbook routine, an error
bound, or brute force over sets derived independently (tests/oracle_shadow.py).
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import workloads as W
from oracle_shadow import Shadow, softmax_attend

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
U32 = 2.0 ** -24


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _tiny_spec(**kw):
    base = dict(name="tiny", batch=2, num_kv_heads=2, group=2, head_dim=16, page_size=4,
                budget=16, window=3, steps=40, dtype="f32", prefill=(61, 38), seed=11)
    base.update(kw)
    return W.Spec(**base)


def _run(spec, steps=None, attend=True):
    g = W.Generator(spec)
    o = oracle.Oracle.for_spec(spec)
    for b, (k, v) in enumerate(g.prefill()):
        o.prefill(b, k, v)
    qw = W.QueryWindow(spec)
    outs = []
    for t in range(spec.steps if steps is None else steps):
        k, v, q = g.step(t)
        win = qw.push(q).copy()
        out = o.step(t, k, v, win, attend=attend)
        out["q_window"] = win
        outs.append(out)
    return g, o, outs


# ----------------------------------------------------------------------------- digests
@pytest.mark.parametrize("tps", [1, 3])
def test_digest_is_elementwise_min_max_of_stored_keys(tps):
    spec = _tiny_spec(tokens_per_step=tps, steps=12)
    g, o, _ = _run(spec, attend=False)
    for b in range(spec.batch):
        L = int(o.seq_lens[b])
        for p in range(-(-L // spec.page_size)):
            lo, hi = p * spec.page_size, min((p + 1) * spec.page_size, L)
            keys = g.keys[b][lo:hi]                      # [n][h_k][d], the generator's copy
            np.testing.assert_array_equal(o.kmin[b, :, p], keys.min(axis=0))
            np.testing.assert_array_equal(o.kmax[b, :, p], keys.max(axis=0))


# ----------------------------------------------------------------------------- UpdateKV
def test_update_kv_overwrites_recent_tokens_and_recomputes_digests():
    """UpdateKV (Alg. 1; Sec. 3.3): the n most recent stored tokens of each sequence
    take the new keys and values, nothing else changes, and every page digest is
    again the element-wise min / max over the page's stored keys: here the update
    lowers a page maximum, which widening could not produce."""
    P, d, hk = 4, 8, 2
    o = oracle.Oracle(batch=2, num_kv_heads=hk, group=1, head_dim=d, page_size=P, budget=P,
                      window=0, max_tokens=40)
    rng = np.random.default_rng(5)
    lens = [13, 2]
    for b, L in enumerate(lens):
        k = rng.standard_normal((L, hk, d)).astype(np.float32)
        v = rng.standard_normal((L, hk, d)).astype(np.float32)
        k[L - 1, 0, 3] = 50.0                       # the page maximum, about to be replaced
        o.prefill(b, k, v)
    K0, V0 = o.K.copy(), o.V.copy()
    old_max = o.kmax[0, 0, (lens[0] - 1) // P, 3]
    n = 3                                           # sequence 1 holds only 2 tokens
    ku = rng.standard_normal((2, n, hk, d)).astype(np.float32)
    vu = rng.standard_normal((2, n, hk, d)).astype(np.float32)
    o.update_kv(ku, vu)
    for b, L in enumerate(lens):
        for j in range(n):
            pos = L - n + j
            if pos < 0:
                continue
            np.testing.assert_array_equal(o.K[b, :, pos], ku[b, j])
            np.testing.assert_array_equal(o.V[b, :, pos], vu[b, j])
        keep = max(L - n, 0)
        np.testing.assert_array_equal(o.K[b, :, :keep], K0[b, :, :keep])
        np.testing.assert_array_equal(o.V[b, :, :keep], V0[b, :, :keep])
        for page in range(-(-L // P)):
            toks = o.K[b, :, page * P:min((page + 1) * P, L)]
            np.testing.assert_array_equal(o.kmin[b, :, page], toks.min(axis=1))
            np.testing.assert_array_equal(o.kmax[b, :, page], toks.max(axis=1))
    assert o.kmax[0, 0, (lens[0] - 1) // P, 3] < old_max


# ----------------------------------------------------------------------------- score
def _score_setup(dtype, d, G, seed):
    spec = _tiny_spec(head_dim=d, group=G, dtype=dtype, prefill=(70, 70), steps=0, seed=seed)
    g = W.Generator(spec)
    o = oracle.Oracle.for_spec(spec)
    for b, (k, v) in enumerate(g.prefill()):
        o.prefill(b, k, v)
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((spec.batch, spec.num_q_heads, d)).astype(np.float32) * 3
    if dtype == "bf16":
        q = W.round_bf16(q)
    return spec, g, o, q


@pytest.mark.parametrize("dtype,d,G", [("f32", 16, 2), ("bf16", 64, 4), ("f32", 128, 8),
                                       ("bf16", 128, 1)])
def test_score_within_fp32_error_bound_of_exact_value(dtype, d, G):
    """eq. (quest_score) over the reals vs the fp32 evaluation: the error of a
    pairwise sum of d terms plus a sequential sum of G terms (plus one rounding
    per product for fp32 inputs) is at most (log2 d + G + 1) u sum|terms|."""
    spec, g, o, q = _score_setup(dtype, d, G, seed=d + G)
    s = o.score(q)
    for b in range(spec.batch):
        n = -(-int(o.seq_lens[b]) // spec.page_size)
        for h in range(spec.num_kv_heads):
            qq = q[b, h * G:(h + 1) * G].astype(np.float64)          # [G][d]
            lo = o.kmin[b, h, :n].astype(np.float64)                   # [n][d]
            hi = o.kmax[b, h, :n].astype(np.float64)
            terms = np.maximum(qq[None] * lo[:, None], qq[None] * hi[:, None])  # [n][G][d]
            exact = terms.sum(axis=(1, 2))
            bound = (math.log2(d) + G + 1) * U32 * np.abs(terms).sum(axis=(1, 2)) * 1.01
            err = np.abs(s[b, h, :n].astype(np.float64) - exact)
            assert np.all(err <= bound + 1e-30), (err - bound).max()


def test_score_of_single_token_page_is_sum_of_dot_products():
    """A page holding one key k has Kmin = Kmax = k, so eq. (quest_score) reduces
    to sum_g q_g . k."""
    spec = _tiny_spec(prefill=(1,), batch=1, steps=0, head_dim=32, group=3)
    g = W.Generator(spec)
    o = oracle.Oracle.for_spec(spec)
    k, v = g.prefill()[0]
    o.prefill(0, k, v)
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, spec.num_q_heads, 32)).astype(np.float32)
    s = o.score(q)
    for h in range(spec.num_kv_heads):
        qq = q[0, h * 3:(h + 1) * 3].astype(np.float64)
        kk = k[0, h].astype(np.float64)
        exact = float((qq @ kk).sum())
        assert abs(float(s[0, h, 0]) - exact) <= (5 + 3 + 1) * U32 * float(np.abs(qq * kk).sum())


def test_score_upper_bounds_every_key_of_the_page():
    """For every key l of page j and every query, Q.k_l <= score_j(Q): each term
    Q_i k_{l,i} lies between Q_i Kmin_i and Q_i Kmax_i (Quest's upper bound)."""
    spec, g, o, q = _score_setup("f32", 64, 4, seed=3)
    s = o.score(q)
    for b in range(spec.batch):
        L = int(o.seq_lens[b])
        for h in range(spec.num_kv_heads):
            qq = q[b, h * 4:(h + 1) * 4].astype(np.float64)
            keys = g.keys[b][:L, h].astype(np.float64)                # [L][d]
            dots = (keys @ qq.T).sum(axis=1)                           # [L]
            pages = np.arange(L) // spec.page_size
            slack = (6 + 4 + 1) * U32 * (np.abs(keys) @ np.abs(qq).T).sum(axis=1)
            assert np.all(dots <= s[b, h, pages].astype(np.float64) + 2 * slack)


def test_score_evaluation_order_golden():
    gold = _load("score_order.json")
    d = gold["head_dim"]
    o = oracle.Oracle(batch=1, num_kv_heads=1, group=1, head_dim=d, page_size=1, budget=1,
                      window=0, max_tokens=1)
    key = np.array(gold["key"], np.float32).reshape(1, 1, d)
    o.prefill(0, key, np.zeros_like(key))
    s = o.score(np.array(gold["q"], np.float32).reshape(1, 1, d))
    assert float(s[0, 0, 0]) == gold["expected_fp32"]
    assert math.copysign(1.0, float(s[0, 0, 0])) == 1.0      # never a negative zero


# ----------------------------------------------------------------------------- top-k
@pytest.mark.parametrize("n,budget_pages", [(37, 8), (129, 16), (5, 16), (64, 64), (300, 1)])
def test_select_equals_stable_sort_by_score_then_index(n, budget_pages):
    P = 4
    o = oracle.Oracle(batch=2, num_kv_heads=3, group=1, head_dim=8, page_size=P,
                      budget=budget_pages * P, window=0, max_tokens=400 * P)
    rng = np.random.default_rng(n)
    scores = np.zeros((2, 3, o.max_pages), np.float32)
    # heavy ties, signed zeros included
    scores[:, :, :n] = rng.integers(-3, 4, size=(2, 3, n)).astype(np.float32)
    scores[0, 0, :n:7] = -0.0
    o.seq_lens[:] = [n * P - 1, (n - 1) * P + 1]
    sel, num = o.select(scores)
    for b in range(2):
        nb = -(-int(o.seq_lens[b]) // P)
        k = min(budget_pages, nb)
        for h in range(3):
            idx = np.arange(nb)
            order = np.lexsort((idx, -scores[b, h, :nb].astype(np.float64)))
            want = np.sort(order[:k])
            assert num[b, h] == k
            np.testing.assert_array_equal(sel[b, h, :k], want)
            assert np.all(sel[b, h, k:] == -1)


def test_relative_budget_pages():
    """Relative budget (Sec. 4 ablation, Table 1's setting: fraction 0.15 of the
    context, at least 256 tokens): k = min(floor(max(256, floor(0.15 L)) / P),
    pages of the sequence), the counts below worked by hand for P = 16."""
    P = 16
    lens = [100, 1707, 1813, 1814, 10000, 20000]
    # 100 tokens: 7 pages; 256/16; floor(271.95) = 271 -> 16; 272/16; 1500/16; 3000/16
    want_k = [7, 16, 16, 17, 93, 187]
    o = oracle.Oracle(batch=len(lens), num_kv_heads=1, group=1, head_dim=8, page_size=P,
                      budget=256, window=0, max_tokens=20000, budget_permille=150)
    assert o.k_max == 187                 # the budget of a full 1250-page row
    rng = np.random.default_rng(3)
    scores = rng.standard_normal((len(lens), 1, o.max_pages)).astype(np.float32)
    o.seq_lens[:] = lens
    sel, num = o.select(scores)
    for b, (L, k) in enumerate(zip(lens, want_k)):
        assert num[b, 0] == k
        nb = -(-L // P)
        order = np.lexsort((np.arange(nb), -scores[b, 0, :nb].astype(np.float64)))
        np.testing.assert_array_equal(sel[b, 0, :k], np.sort(order[:k]))
        assert np.all(sel[b, 0, k:] == -1)
    fixed = oracle.Oracle(batch=len(lens), num_kv_heads=1, group=1, head_dim=8, page_size=P,
                          budget=256, window=0, max_tokens=20000)
    assert fixed.k_max == 16
    fixed.seq_lens[:] = lens
    _, num = fixed.select(scores)
    assert list(num[:, 0]) == [7, 16, 16, 16, 16, 16]


# ----------------------------------------------------------------------------- Alg. 2
def test_alg2_golden_walk():
    gold = _load("alg2_walk.json")
    P, W_ = gold["page_size"], gold["window"]
    o = oracle.Oracle(batch=1, num_kv_heads=1, group=1, head_dim=2, page_size=P,
                      budget=3 * P, window=W_, max_tokens=gold["prefill_tokens"] + 5)
    z = np.zeros((gold["prefill_tokens"], 1, 2), np.float32)
    o.prefill(0, z, z)
    for st in gold["steps"]:
        t = st["t"]
        o.append(t, np.zeros((1, 1, 2), np.float32), np.zeros((1, 1, 2), np.float32))
        assert (int(o.seq_lens[0]) - 1) // P == st["p_curr"]
        sel = np.full((1, 1, o.k_max), -1, np.int32)
        sel[0, 0, :3] = st["S"]
        num = np.array([[3]], np.int32)
        M = o.build_mask(t, sel, num)
        assert list(M[0, 0, :3]) == st["M"], t
        assert list(o.A[0, 0, :7]) == st["A_after"], t
        st["_M"] = dict(zip(st["S"], st["M"]))
    for e in gold["eligible_past"]:
        st = gold["steps"][e["t"]]
        got = sorted(p for p, m in st["_M"].items() if m < e["tau"])   # the paper's mask rule
        assert got == e["pages"], e


@pytest.mark.parametrize("tps,P,W_", [(1, 4, 3), (3, 4, 5), (1, 8, 1), (5, 4, 2)])
def test_mask_rule_equals_set_semantics_and_never_double_counts(tps, P, W_):
    """Alg. 2's A/M bookkeeping (M_p < tau) selects exactly the pages of
    eq. (update-sup) minus those holding keys newer than tau, for every past
    query of every step; and no token reaches a query twice."""
    spec = _tiny_spec(tokens_per_step=tps, page_size=P, window=W_, steps=48,
                      budget=4 * P, prefill=(9 * P + 1, 5 * P + 3))
    _, o, outs = _run(spec, attend=False)
    sh = Shadow(spec.batch, spec.num_kv_heads, P, W_)
    for t, out in enumerate(outs):
        want = sh.record(t, out["selected"], out["num_selected"], out["seq_lens"])
        for b in range(spec.batch):
            for h in range(spec.num_kv_heads):
                k = out["num_selected"][b, h]
                sel = out["selected"][b, h, :k]
                M = out["mask"][b, h, :k]
                for tau in range(max(0, t - W_), t):
                    got = set(int(p) for p, m in zip(sel, M) if m < tau)
                    assert got == want[(b, h, tau)], (t, b, h, tau)


# ----------------------------------------------------------------------------- attention
def test_attention_and_merge_closed_form_golden():
    gold = _load("attention_closed_form.json")
    d, P = gold["head_dim"], gold["page_size"]
    o = oracle.Oracle(batch=1, num_kv_heads=1, group=1, head_dim=d, page_size=P, budget=2 * P,
                      window=1, max_tokens=4, sm_scale=gold["sm_scale"])
    k = np.array(gold["keys"], np.float32).reshape(4, 1, d)
    v = np.array(gold["values"], np.float32).reshape(4, 1, d)
    o.prefill(0, k, v)
    qw = np.zeros((1, 2, 1, d), np.float32)
    qw[0, :, 0] = gold["q"]             # same query at both window rows
    tol = 1e-6
    for sel_pages, M, key in [([0, 1], [-1, -1], "both"), ([0], [-1], "page0"), ([1], [-1], "page1")]:
        sel = np.full((1, 1, 2), -1, np.int32)
        sel[0, 0, :len(sel_pages)] = sel_pages
        Mm = np.full((1, 1, 2), -1, np.int32)
        Mm[0, 0, :len(M)] = M
        op, zp = o.attend(1, qw, sel, np.array([[len(sel_pages)]], np.int32), Mm)
        np.testing.assert_allclose(op[0, 1, 0], gold[key]["O"], atol=tol)
        assert abs(zp[0, 1, 0] - gold[key]["Z_value"]) < tol
    # Past row tau=0 at step 1: page 0 was loaded at step 0 (M=0, skipped),
    # page 1 is new (M=-1): the supplement is page 1 alone...
    sel = np.array([[[0, 1]]], np.int32)
    op, zp = o.attend(1, qw, sel, np.array([[2]], np.int32), np.array([[[0, -1]]], np.int32))
    np.testing.assert_allclose(op[0, 0, 0], gold["page1"]["O"], atol=tol)
    # ...and merging it into the cached page-0 output gives attention over both.
    om, zm = oracle.lse_merge(gold["page0"]["O"], gold["page0"]["Z_value"], op[0, 0, 0], zp[0, 0, 0])
    np.testing.assert_allclose(om, gold["both"]["O"], atol=tol)
    assert abs(zm - gold["both"]["Z_value"]) < tol


def test_lse_merge_identity_commutativity_associativity():
    rng = np.random.default_rng(0)
    d = 8
    a, b, c = (rng.standard_normal(d) for _ in range(3))
    za, zb, zc = 1.5, -0.25, 3.0
    o, z = oracle.lse_merge(a, za, b, -np.inf)
    np.testing.assert_array_equal(o, a)
    assert z == za
    o, z = oracle.lse_merge(a, -np.inf, b, -np.inf)
    assert np.all(o == 0) and z == -np.inf
    o1, z1 = oracle.lse_merge(a, za, b, zb)
    o2, z2 = oracle.lse_merge(b, zb, a, za)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-14)
    assert abs(z1 - z2) < 1e-14
    l, zl = oracle.lse_merge(*oracle.lse_merge(a, za, b, zb), c, zc)
    r, zr = oracle.lse_merge(a, za, *oracle.lse_merge(b, zb, c, zc))
    np.testing.assert_allclose(l, r, atol=1e-13)
    assert abs(zl - zr) < 1e-13
    # weights are the normalisers e^Z (eq. merged_attn)
    ea, eb = math.exp(za), math.exp(zb)
    np.testing.assert_allclose(o1, (ea * a + eb * b) / (ea + eb), atol=1e-14)
    assert abs(z1 - math.log(ea + eb)) < 1e-14


@pytest.mark.parametrize("tps,W_", [(1, 3), (2, 5), (1, 1)])
def test_every_window_row_equals_softmax_over_its_attended_union(tps, W_):
    """After any number of supplements, a past query's cached output equals plain
    softmax attention over the union of the (disjoint) token sets it has attended,
    so the merged output at finalisation equals attention over the whole union."""
    spec = _tiny_spec(tokens_per_step=tps, window=W_, steps=30)
    g, o, outs = _run(spec)
    sh = Shadow(spec.batch, spec.num_kv_heads, spec.page_size, W_)
    qs = {}
    for t, out in enumerate(outs):
        sh.record(t, out["selected"], out["num_selected"], out["seq_lens"])
        qs[t] = out["q_window"][:, -1].copy()
        for b in range(spec.batch):
            for qh in range(spec.num_q_heads):
                h = qh // spec.group
                for r in range(W_ + 1):
                    tau = t - W_ + r
                    if tau < 0:
                        assert out["lse_out"][b, r, qh] == -np.inf
                        assert np.all(out["o_out"][b, r, qh] == 0)
                        continue
                    toks = sh.seen[(b, h, tau)]
                    O, Z = softmax_attend(qs[tau][b, qh], g.keys[b][:, h], _values(o, b, h), toks,
                                          o.dims.sm_scale)
                    np.testing.assert_allclose(out["o_out"][b, r, qh], O, atol=1e-10)
                    assert abs(out["lse_out"][b, r, qh] - Z) < 1e-10


def _values(o, b, h):
    return o.V[b, h]


def test_full_budget_current_row_is_dense_causal_attention():
    """With a budget covering the whole context every page is selected, so the
    current query's output is dense causal attention (softmax(qK^T/sqrt d)V over
    all stored tokens) and no past query ever gets a supplement."""
    spec = _tiny_spec(budget=4 * 200, steps=10, window=3)
    g, o, outs = _run(spec)
    for t, out in enumerate(outs):
        for b in range(spec.batch):
            L = int(out["seq_lens"][b])
            for qh in range(spec.num_q_heads):
                h = qh // spec.group
                q = out["q_window"][b, -1, qh].astype(np.float64)
                k = g.keys[b][:L, h].astype(np.float64)
                v = o.V[b, h, :L].astype(np.float64)
                s = (k @ q) / math.sqrt(spec.head_dim)
                w = np.exp(s - s.max())
                np.testing.assert_allclose(out["o_out"][b, -1, qh], w @ v / w.sum(), atol=1e-6)
                assert abs(out["lse_out"][b, -1, qh] - (s.max() + math.log(w.sum()))) < 1e-6
                for r in range(spec.window):
                    if t - spec.window + r >= 0:
                        assert out["lse_part"][b, r, qh] == -np.inf


def test_window_zero_is_plain_quest_sparse_attention():
    """W = 0 leaves only the current query: its output is softmax attention over
    the tokens of the k best pages (eq. update-org), pages chosen here with an
    independent numpy sort of the page scores."""
    spec = _tiny_spec(window=0, steps=12)
    g, o, outs = _run(spec)
    for out in outs:
        for b in range(spec.batch):
            L = int(out["seq_lens"][b])
            n = -(-L // spec.page_size)
            k = min(spec.budget // spec.page_size, n)
            for qh in range(spec.num_q_heads):
                h = qh // spec.group
                sc = out["scores"][b, h, :n].astype(np.float64)
                pages = np.lexsort((np.arange(n), -sc))[:k]
                toks = [p * spec.page_size + s for p in pages for s in range(spec.page_size)
                        if p * spec.page_size + s < L]
                O, Z = softmax_attend(out["q_window"][b, 0, qh], g.keys[b][:, h], o.V[b, h], toks,
                                      o.dims.sm_scale)
                np.testing.assert_allclose(out["o_out"][b, 0, qh], O, atol=1e-10)
                assert abs(out["lse_out"][b, 0, qh] - Z) < 1e-10


# ----------------------------------------------------------------------------- top-k reuse
def test_topk_reuse_golden_walk():
    """The selection-reuse baseline (Table 4, f = 2) on a hand-worked walk: refresh
    steps select as PageSelect does, reuse steps keep the last refresh's pages
    whatever the scores say, and Alg. 2's mask runs on the pages in use."""
    gold = _load("topk_reuse_walk.json")
    P = gold["page_size"]
    keys = np.array(gold["prefill_keys"], np.float32).reshape(-1, 1, 2)
    n_steps = len(gold["steps"])
    for f in (gold["reuse_interval"], 1):
        o = oracle.Oracle(batch=1, num_kv_heads=1, group=1, head_dim=2, page_size=P,
                          budget=gold["budget_pages"] * P, window=gold["window"],
                          max_tokens=len(keys) + n_steps, reuse_interval=f)
        o.prefill(0, keys, np.zeros_like(keys))
        for st in gold["steps"]:
            t = st["t"]
            win = np.zeros((1, 2, 1, 2), np.float32)
            win[0, 1, 0] = st["q"]
            tok = np.zeros((1, 1, 2), np.float32)
            out = o.step(t, tok, tok, win, attend=False)
            want = st["selected"] if f == gold["reuse_interval"] else st["fresh_selected"]
            k = int(out["num_selected"][0, 0])
            assert list(out["selected"][0, 0, :k]) == want, (f, t)
            assert (out["scores"] is None) == (f == 2 and t % 2 == 1), (f, t)
            if f == gold["reuse_interval"]:
                assert list(out["mask"][0, 0, :k]) == st["mask"], (f, t)
        if f == gold["reuse_interval"]:
            assert list(o.A[0, 0, :len(gold["last_loaded_after"])]) == gold["last_loaded_after"]


@pytest.mark.parametrize("f", [2, 3])
def test_topk_reuse_steps_keep_the_pages_and_add_no_past_context(f):
    """On a reuse step the pages are the last refresh's, every one of them was
    loaded at the step before (mask t - 1), so no past query of the window gains
    a page (eq. update-sup adds nothing), and its merged output is the cached one."""
    spec = _tiny_spec(reuse_interval=f, steps=24)
    _, o, outs = _run(spec)
    for t, out in enumerate(outs):
        if t % f == 0:
            assert out["scores"] is not None
            last = t
            continue
        assert out["scores"] is None
        assert np.array_equal(out["selected"], outs[last]["selected"]), t
        assert np.array_equal(out["num_selected"], outs[last]["num_selected"]), t
        for b in range(spec.batch):
            for h in range(spec.num_kv_heads):
                k = out["num_selected"][b, h]
                assert np.all(out["mask"][b, h, :k] == t - 1), (t, b, h)
        # rows of past queries (not the one leaving, whose result is final) keep
        # their previous merged output: nothing supplementary reached them
        for r in range(1, spec.window):
            tau = t - spec.window + r
            if tau < 0:
                continue
            prev = outs[t - 1]
            assert np.allclose(out["o_out"][:, r], prev["o_out"][:, r + 1], rtol=0, atol=0), (t, r)
            assert np.array_equal(out["lse_out"][:, r], prev["lse_out"][:, r + 1]), (t, r)
