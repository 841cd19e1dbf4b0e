"""Multi-layer decode with re-embedding (Sec. 3.3) on the GPU against the oracle.

* fp32, free running: the GPU stack and the oracle stack each run from the same
  seeded embeddings, weights and prompts; every layer's selection and mask must
  match bit for bit at every step, and the outputs within 1e-4 (fp32 products
  over d_model terms, accumulated in a different order than the oracle's fp64,
  feed the next layer: a few 1e-6 per layer, see the design notes).
* bf16, layer by layer: each layer's projections are checked against the
  oracle's fp64 products of the same bf16 inputs (within one bf16 rounding), then
  the GPU's own bf16 queries, keys and values are handed to the oracle layer, so
  that selection, mask, A and every page digest compare bit for bit and the
  merged outputs within 2e-3, as for a single layer.  With UpdateKV folded into
  the projection launch the past rows' keys and values are read back from the
  GPU cache.
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads as W
from oracle.decoder import round_to

pytestmark = pytest.mark.gpu


def _inputs(spec, layers):
    inp = W.DecoderInputs(spec, layers)
    return inp, inp.weights()


def _build(spec, layers, fuse_update=True):
    import torch
    from oracle.decoder import OracleDecoder
    from paper_2508_09001_amd.decode import RetroDecoder, layer_kwargs
    inp, weights = _inputs(spec, layers)
    dec = RetroDecoder(weights, fuse_update=fuse_update, **layer_kwargs(spec))
    orc = OracleDecoder(spec, weights)
    for layer in range(layers):
        for b, (k, v) in enumerate(inp.prefill(layer)):
            dec.prefill(layer, b, k, v)
            orc.layers[layer].prefill(b, k, v)
    torch.cuda.synchronize()
    return inp, dec, orc


def _window(emb, inp, t):
    return np.concatenate([emb[:, 1:], inp.embedding(t)[:, None]], axis=1)


def _np(x):
    return x.float().cpu().numpy() if x.dtype.is_floating_point else x.cpu().numpy()


def _same_selection(t, layer, g, r, A_gpu, A_ref):
    assert np.array_equal(_np(g["num_selected"]), r["num_selected"]), f"t={t} l={layer}: k"
    assert np.array_equal(_np(g["selected"]), r["selected"]), f"t={t} l={layer}: selection"
    assert np.array_equal(_np(g["mask"]), r["mask"]), f"t={t} l={layer}: mask"
    assert np.array_equal(A_gpu, A_ref), f"t={t} l={layer}: A"


def test_decoder_fp32_free_running_matches_oracle():
    import torch
    spec = W.Spec(name="dec-f32", batch=2, num_kv_heads=2, group=4, head_dim=64, page_size=16,
                  budget=64, window=4, steps=9, dtype="f32", prefill=(300, 211))
    layers = 3
    print(f"[decoder] {spec.name}: layers={layers}", flush=True)
    inp, dec, orc = _build(spec, layers)
    emb = np.zeros((spec.batch, spec.window + 1, inp.d_model), np.float32)
    worst = 0.0
    for t in range(spec.steps):
        emb = _window(emb, inp, t)
        tg, tr = [], []
        h_gpu = dec.step(t, torch.from_numpy(emb).cuda(), tg)
        h_ref = orc.step(t, emb, tr)
        torch.cuda.synchronize()
        for layer in range(layers):
            _same_selection(t, layer, tg[layer], tr[layer],
                            _np(dec.layers[layer].last_loaded), orc.layers[layer].A)
            eo = np.max(np.abs(_np(tg[layer]["o_out"]) - tr[layer]["o_out"]))
            assert eo <= 1e-4, f"t={t} l={layer}: max |O - O_ref| = {eo:.3g}"
            worst = max(worst, float(eo))
        eh = np.max(np.abs(_np(h_gpu) - h_ref))
        assert eh <= 1e-4, f"t={t}: max |H - H_ref| = {eh:.3g}"
        worst = max(worst, float(eh))
    print(f"[decoder] {spec.name}: ok, worst abs error {worst:.3g}", flush=True)


def _cache_rows(lay, b, positions):
    """Keys and values [n][h_k][d] of sequence b at the given positions, read back
    from the layer's paged cache."""
    pt = lay.page_table.cpu().numpy()
    kc, vc = lay.k_cache.float().cpu().numpy(), lay.v_cache.float().cpu().numpy()
    P = lay.P
    k = np.stack([kc[pt[b, p // P], :, p % P, :] for p in positions])
    v = np.stack([vc[pt[b, p // P], :, :, p % P] for p in positions])
    return k, v


@pytest.mark.parametrize("window,budget_permille,fuse,batch", [(4, 0, True, 2), (8, 150, True, 2),
                                                               (0, 0, True, 2), (4, 0, False, 2),
                                                               (16, 0, True, 2), (16, 0, True, 4)])
def test_decoder_bf16_layers_match_oracle_on_the_same_inputs(window, budget_permille, fuse, batch):
    """fuse: UpdateKV inside the projection launch (the past rows' keys and values
    are then read back from the cache and the digests compared exactly)."""
    import torch
    spec = W.Spec(name="dec-bf16-llama-heads", batch=batch, num_kv_heads=8, group=4,
                  head_dim=128, page_size=16, budget=256, window=window,
                  steps=7 if window < 16 else 20, dtype="bf16",
                  prefill=(1500, 2047, 777, 1024)[:batch], budget_permille=budget_permille)
    layers = 2
    print(f"[decoder] {spec.name}: W={window} permille={budget_permille} fuse={fuse} "
          f"batch={batch} layers={layers}", flush=True)
    inp, dec, orc = _build(spec, layers, fuse_update=fuse)
    emb = np.zeros((spec.batch, spec.window + 1, inp.d_model), np.float32)
    worst = {"proj": 0.0, "o": 0.0, "y": 0.0}
    for t in range(spec.steps):
        emb = _window(emb, inp, t)
        n_upd = orc.n_update()
        assert n_upd == dec.n_update()
        tg = []
        dec.step(t, torch.from_numpy(emb).cuda(), tg)
        torch.cuda.synchronize()
        for layer in range(layers):
            g = tg[layer]
            x = _np(g["x"])
            if layer == 0:
                np.testing.assert_array_equal(x, W.round_bf16(emb))
            q = _np(g["q"])
            refs = orc.project(layer, x)
            if fuse:
                # rows W-n .. W-1 went straight to the cache, row W to k_new / v_new
                k = np.zeros_like(refs[1])
                v = np.zeros_like(refs[2])
                k[:, -1], v[:, -1] = _np(g["k_new"]), _np(g["v_new"])
                for b in range(spec.batch):
                    L = int(orc.layers[layer].seq_lens[b])
                    pos = list(range(L - n_upd, L))
                    if pos:
                        kb, vb = _cache_rows(dec.layers[layer], b, pos)
                        k[b, spec.window - n_upd:spec.window] = kb
                        v[b, spec.window - n_upd:spec.window] = vb
                rows = list(range(spec.window - n_upd, spec.window + 1))
                checks = ((q, refs[0]), (k[:, rows], refs[1][:, rows]),
                          (v[:, rows], refs[2][:, rows]))
            else:
                k, v = _np(g["k"]), _np(g["v"])
                checks = zip((q, k, v), refs)
            for got, ref in checks:
                err = np.abs(got - ref)
                assert np.all(err <= 2.0 ** -7 * np.abs(ref) + 1e-3), f"t={t} l={layer}: proj"
                worst["proj"] = max(worst["proj"], float(err.max()))
            r = orc.attend_layer(layer, t, q, k, v, n_upd)
            _same_selection(t, layer, g, r, _np(dec.layers[layer].last_loaded),
                            orc.layers[layer].A)
            # digests of every stored page (the re-embedded ones recomputed)
            dg = _np(dec.layers[layer].digest).reshape(spec.batch, spec.num_kv_heads,
                                                       spec.max_pages, 2, spec.head_dim)
            ol = orc.layers[layer]
            for b in range(spec.batch):
                npg = -(-int(ol.seq_lens[b]) // spec.page_size)
                np.testing.assert_array_equal(dg[b, :, :npg, 0], ol.kmin[b, :, :npg])
                np.testing.assert_array_equal(dg[b, :, :npg, 1], ol.kmax[b, :, :npg])
            o = _np(g["o_out"])
            eo = float(np.max(np.abs(o - r["o_out"])))
            assert eo <= 2e-3, f"t={t} l={layer}: max |O - O_ref| = {eo:.3g}"
            worst["o"] = max(worst["o"], eo)
            y_ref = orc.out_proj(layer, o)
            ey = np.abs(_np(g["y"]) - y_ref)
            assert np.all(ey <= 2.0 ** -7 * np.abs(y_ref) + 1e-3), f"t={t} l={layer}: o-proj"
            worst["y"] = max(worst["y"], float(ey.max()))
            if "x_next" in g:   # library projections: the next input is bf16(h)
                np.testing.assert_array_equal(_np(g["x_next"]), round_to(_np(g["h_out"]), "bf16"))
        orc.decoded += 1
    print(f"[decoder] {spec.name}: ok, worst {worst}", flush=True)


def _proj_case(rows, K, nq, nkv, seed):
    import torch
    from paper_2508_09001_amd import binding as B
    rng = np.random.default_rng(seed)
    n = nq + 2 * nkv
    x = W.round_bf16(rng.standard_normal((rows, K), dtype=np.float32))
    w = W.round_bf16(rng.standard_normal((K, n), dtype=np.float32) * np.float32(K ** -0.5))
    xd = torch.from_numpy(x).cuda().to(torch.bfloat16)
    wd = torch.from_numpy(w).cuda().to(torch.bfloat16)
    wp = torch.empty_like(wd)
    B.retro_pack_weight(wd, K, n, wp)
    q = torch.empty(rows, nq, dtype=torch.bfloat16, device="cuda")
    k = torch.empty(rows, nkv, dtype=torch.bfloat16, device="cuda")
    v = torch.empty(rows, nkv, dtype=torch.bfloat16, device="cuda")
    B.retro_project_qkv(xd, rows, K, wp, nq, nkv, q, k, v)
    torch.cuda.synchronize()
    ref = x.astype(np.float64) @ w.astype(np.float64)
    got = np.concatenate([q.float().cpu().numpy(), k.float().cpu().numpy(),
                          v.float().cpu().numpy()], axis=1)
    return got, ref, round_to(ref, "bf16")


@pytest.mark.parametrize("rows,K,nq,nkv", [(1, 1024, 256, 64), (5, 2048, 512, 128),
                                           (17, 4096, 4096, 1024), (34, 1024, 128, 32),
                                           (48, 3072, 64, 16), (20, 1024, 16, 16),
                                           (72, 2048, 256, 64), (112, 1024, 64, 16)])
def test_project_qkv_matches_fp64_products(rows, K, nq, nkv):
    print(f"[proj] qkv rows={rows} K={K} nq={nq} nkv={nkv}", flush=True)
    got, ref, ref_b = _proj_case(rows, K, nq, nkv, seed=rows * 7 + K)
    # fp32 accumulation, then one rounding to bf16: within one bf16 step of the
    # fp64 product, and equal to its rounding for almost every element
    assert np.all(np.abs(got - ref) <= 2.0 ** -7 * np.abs(ref) + 1e-6)
    assert np.mean(got == ref_b) > 0.98


@pytest.mark.parametrize("rows,K,n", [(1, 1024, 512), (17, 4096, 4096), (40, 2048, 256),
                                      (18, 1024, 48), (72, 4096, 1024), (100, 1024, 256)])
def test_project_out_adds_the_residual(rows, K, n):
    import torch
    from paper_2508_09001_amd import binding as B
    print(f"[proj] out rows={rows} K={K} n={n}", flush=True)
    rng = np.random.default_rng(rows + K + n)
    o = rng.standard_normal((rows, K)).astype(np.float32)
    w = W.round_bf16(rng.standard_normal((K, n), dtype=np.float32) * np.float32(K ** -0.5))
    h0 = rng.standard_normal((rows, n)).astype(np.float32)
    wd = torch.from_numpy(w).cuda().to(torch.bfloat16)
    wp = torch.empty_like(wd)
    B.retro_pack_weight(wd, K, n, wp)
    h = torch.from_numpy(h0).cuda()
    xn = torch.empty(rows, n, dtype=torch.bfloat16, device="cuda")
    B.retro_project_out(torch.from_numpy(o).cuda(), rows, K, wp, n, h, xn)
    torch.cuda.synchronize()
    y_ref = round_to(round_to(o, "bf16").astype(np.float64) @ w.astype(np.float64), "bf16")
    hn = h.cpu().numpy()
    err = np.abs(hn.astype(np.float64) - (h0.astype(np.float64) + y_ref))
    assert np.all(err <= 2.0 ** -7 * np.abs(y_ref) + 1e-6 * (1 + np.abs(h0)))
    np.testing.assert_array_equal(xn.float().cpu().numpy(), round_to(hn, "bf16"))


@pytest.mark.parametrize("rows,K,n,accumulate", [(1, 256, 512, False), (5, 1000, 96, False),
                                                 (18, 2500, 300, True), (40, 64, 1024, True)])
def test_project_f32_matches_fp64_products(rows, K, n, accumulate):
    """fp32 projections of fp32 stacks: each element is an fp32 fused
    multiply-add chain, within the textbook bound gamma_K * sum |x| |w| of the
    fp64 product (plus one rounding of the residual add), and the same bits on a
    second call."""
    import torch
    from paper_2508_09001_amd import binding as B
    print(f"[proj] f32 rows={rows} K={K} n={n} accumulate={accumulate}", flush=True)
    rng = np.random.default_rng(rows * 131 + K + n)
    x = rng.standard_normal((rows, K)).astype(np.float32)
    w = (rng.standard_normal((K, n)) * K ** -0.5).astype(np.float32)
    h0 = rng.standard_normal((rows, n)).astype(np.float32) if accumulate else \
        np.zeros((rows, n), np.float32)
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.from_numpy(h0).cuda()
    B.retro_project_f32(xd, rows, K, wd, n, y, accumulate=accumulate)
    y2 = torch.from_numpy(h0).cuda()
    B.retro_project_f32(xd, rows, K, wd, n, y2, accumulate=accumulate)
    torch.cuda.synchronize()
    got = y.cpu().numpy().astype(np.float64)
    ref = h0.astype(np.float64) + x.astype(np.float64) @ w.astype(np.float64)
    u = 2.0 ** -24
    gamma = K * u / (1 - K * u)
    bound = gamma * (np.abs(x).astype(np.float64) @ np.abs(w).astype(np.float64)) + \
        u * np.abs(ref) * (2 if accumulate else 0)
    assert np.all(np.abs(got - ref) <= bound + 1e-30)
    assert torch.equal(y, y2)


def test_projection_shape_errors_are_reported_before_any_launch():
    import torch
    from paper_2508_09001_amd import binding as B
    x = torch.zeros(4, 1024, dtype=torch.bfloat16, device="cuda")
    wp = torch.zeros(1024, 96, dtype=torch.bfloat16, device="cuda")
    q = torch.zeros(4, 64, dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros(4, 16, dtype=torch.bfloat16, device="cuda")
    for rows, K in [(113, 1024), (4, 512), (4, 1000)]:
        with pytest.raises(RuntimeError):
            B.retro_project_qkv(x, rows, K, wp, 64, 16, q, kv, kv)
    B.retro_project_qkv(x, 0, 1024, wp, 64, 16, q, kv, kv)   # no rows: nothing to do
    with pytest.raises(RuntimeError):
        B.retro_pack_weight(wp, 1000, 96, wp)
