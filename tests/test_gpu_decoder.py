"""Multi-layer decode with re-embedding (Sec. 3.3) on the GPU against the oracle.

* fp32, free running: the GPU stack and the oracle stack each run from the same
  seeded embeddings, weights and prompts; every layer's selection and mask must
  match bit for bit at every step, and the outputs within 1e-4 (fp32 products
  over d_model terms, accumulated in a different order than the oracle's fp64,
  feed the next layer: a few 1e-6 per layer, see the design notes).
* bf16, layer by layer: each layer's projections are checked against the
  oracle's fp64 products of the same bf16 inputs (within one bf16 rounding), then
  the GPU's own bf16 queries, keys and values are handed to the oracle layer, so
  that selection, mask and A compare bit for bit and the merged outputs within
  2e-3, as for a single layer.
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


def _inputs(spec, layers):
    inp = W.DecoderInputs(spec, layers)
    return inp, inp.weights()


def _build(spec, layers):
    import torch
    from oracle.decoder import OracleDecoder
    from paper_2508_09001_amd.decode import RetroDecoder, layer_kwargs
    inp, weights = _inputs(spec, layers)
    dec = RetroDecoder(weights, **layer_kwargs(spec))
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


@pytest.mark.parametrize("window,budget_permille", [(4, 0), (8, 150), (0, 0)])
def test_decoder_bf16_layers_match_oracle_on_the_same_inputs(window, budget_permille):
    import torch
    spec = W.Spec(name="dec-bf16-llama-heads", batch=2, num_kv_heads=8, group=4, head_dim=128,
                  page_size=16, budget=256, window=window, steps=7, dtype="bf16",
                  prefill=(1500, 2047), budget_permille=budget_permille)
    layers = 2
    print(f"[decoder] {spec.name}: W={window} permille={budget_permille} layers={layers}",
          flush=True)
    inp, dec, orc = _build(spec, layers)
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
            q, k, v = (_np(g[n]) for n in ("q", "k", "v"))
            for got, ref in zip((q, k, v), orc.project(layer, x)):
                err = np.abs(got - ref)
                assert np.all(err <= 2.0 ** -7 * np.abs(ref) + 1e-3), f"t={t} l={layer}: proj"
                worst["proj"] = max(worst["proj"], float(err.max()))
            r = orc.attend_layer(layer, t, q, k, v, n_upd)
            _same_selection(t, layer, g, r, _np(dec.layers[layer].last_loaded),
                            orc.layers[layer].A)
            o = _np(g["o_out"])
            eo = float(np.max(np.abs(o - r["o_out"])))
            assert eo <= 2e-3, f"t={t} l={layer}: max |O - O_ref| = {eo:.3g}"
            worst["o"] = max(worst["o"], eo)
            y_ref = orc.out_proj(layer, o)
            ey = np.abs(_np(g["y"]) - y_ref)
            assert np.all(ey <= 2.0 ** -7 * np.abs(y_ref) + 1e-3), f"t={t} l={layer}: o-proj"
            worst["y"] = max(worst["y"], float(ey.max()))
        orc.decoded += 1
    print(f"[decoder] {spec.name}: ok, worst {worst}", flush=True)
