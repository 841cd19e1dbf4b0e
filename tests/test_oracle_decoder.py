"""Pins of the multi-layer decode oracle (re-embedding across layers, Sec. 3.3).

* With a budget that covers every page, nothing is ever unseen, so the
  retrospective supplements are empty, the merged outputs equal the original
  ones and the re-embedded keys and values equal the stored ones: the stack must
  reproduce plain dense causal decoding, written out here with numpy's softmax.
* Layer 0's inputs are token embeddings, which do not change, so its stored keys
  are never altered by re-embedding and its current-row outputs do not depend on
  the window; deeper layers' stored keys do change once past outputs are updated.
* After every step the stored keys and values of the re-embedded rows are the
  projections of that step's window rows (row alignment of UpdateKV).
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads as W
from oracle.decoder import OracleDecoder, round_to


def _spec(**kw):
    base = dict(name="dec-tiny", batch=2, num_kv_heads=2, group=2, head_dim=16, page_size=4,
                budget=8, window=3, steps=9, dtype="f32", prefill=(13, 10))
    base.update(kw)
    return W.Spec(**base)


def _run(spec, layers=3, keep_trace=False):
    inp = W.DecoderInputs(spec, layers)
    dec = OracleDecoder(spec, inp.weights())
    for layer in range(layers):
        for b, (k, v) in enumerate(inp.prefill(layer)):
            dec.layers[layer].prefill(b, k, v)
    emb = np.zeros((spec.batch, spec.window + 1, inp.d_model), np.float32)
    outs, traces = [], []
    for t in range(spec.steps):
        emb = np.concatenate([emb[:, 1:], inp.embedding(t)[:, None]], axis=1)
        tr = [] if keep_trace else None
        outs.append(dec.step(t, emb, tr))
        traces.append(tr)
    return inp, dec, outs, traces


def _dense(spec, inp, layers):
    """Dense causal decoding of the same stack: every token attends every earlier
    token and itself, keys and values are computed once."""
    ws = [{k: np.asarray(v, np.float64) for k, v in w.items()} for w in inp.weights()]
    s, d = spec, spec.head_dim
    scale = float(np.float32(1.0 / np.sqrt(d)))
    kv = [[[k.astype(np.float64), v.astype(np.float64)] for k, v in inp.prefill(layer)]
          for layer in range(layers)]
    outs = []
    for t in range(spec.steps):
        h = inp.embedding(t).astype(np.float64)                      # [b][d_model]
        for layer in range(layers):
            x = round_to(h, s.dtype).astype(np.float64)
            q = round_to(x @ ws[layer]["wq"], s.dtype).reshape(s.batch, s.num_q_heads, d)
            k = round_to(x @ ws[layer]["wk"], s.dtype).reshape(s.batch, s.num_kv_heads, d)
            v = round_to(x @ ws[layer]["wv"], s.dtype).reshape(s.batch, s.num_kv_heads, d)
            o = np.zeros((s.batch, s.num_q_heads, d))
            for b in range(s.batch):
                kv[layer][b][0] = np.concatenate([kv[layer][b][0], k[b][None]])
                kv[layer][b][1] = np.concatenate([kv[layer][b][1], v[b][None]])
                K, V = kv[layer][b]
                for hq in range(s.num_q_heads):
                    g = hq // s.group
                    logits = (K[:, g].astype(np.float32) @ q[b, hq].astype(np.float32)
                              ).astype(np.float64) * scale
                    p = np.exp(logits - logits.max())
                    o[b, hq] = (p / p.sum()) @ V[:, g]
            o_s = round_to(o.reshape(s.batch, -1), s.dtype).astype(np.float64)
            h = h + round_to(o_s @ ws[layer]["wo"], s.dtype)
        outs.append(h)
    return outs


@pytest.mark.parametrize("window", [0, 3])
def test_full_budget_stack_is_dense_causal_decoding(window):
    spec = _spec(budget=64, window=window)       # 64 tokens >= every context here
    inp, _, outs, _ = _run(spec)
    ref = _dense(spec, inp, 3)
    for t in range(spec.steps):
        np.testing.assert_allclose(outs[t][:, -1], ref[t], rtol=1e-6, atol=1e-6)
        # decoded past rows keep their original values too
        for r in range(1, min(window, t) + 1):
            np.testing.assert_allclose(outs[t][:, -1 - r], ref[t - r], rtol=1e-6, atol=1e-6)


def test_full_budget_bf16_stack_is_dense_causal_decoding():
    spec = _spec(budget=64, dtype="bf16")
    inp, _, outs, _ = _run(spec, layers=2)
    ref = _dense(spec, inp, 2)
    for t in range(spec.steps):
        np.testing.assert_allclose(outs[t][:, -1], ref[t], rtol=1e-5, atol=1e-5)


def test_reembedding_leaves_layer0_and_changes_deeper_layers():
    spec = _spec()
    inp, dec, outs, traces = _run(spec, keep_trace=True)
    _, dec0, _, traces0 = _run(spec.replace(window=0), keep_trace=True)
    # first-time keys of every decoded token at every layer
    for t in range(spec.steps):
        np.testing.assert_allclose(traces[t][0]["o_out"][:, -1], traces0[t][0]["o_out"][:, -1],
                                   rtol=0, atol=0)
    changed = []
    for layer in range(3):
        for b in range(spec.batch):
            n0 = spec.prefill[b]
            first = np.stack([traces[t][layer]["k"][b, -1] for t in range(spec.steps)])
            stored = dec.layers[layer].K[b][:, n0:n0 + spec.steps].transpose(1, 0, 2)
            if layer == 0:
                np.testing.assert_array_equal(stored, first)
            else:
                changed.append(not np.array_equal(stored, first))
    assert any(changed), "no deeper layer's stored key was re-embedded"


def test_update_rows_hold_projections_of_the_latest_window():
    spec = _spec()
    inp, dec, _, traces = _run(spec, keep_trace=True)
    t_last = spec.steps - 1
    n_upd = min(spec.window, t_last)
    for layer in range(3):
        tr = traces[t_last][layer]
        for b in range(spec.batch):
            n = spec.prefill[b] + spec.steps
            stored_k = dec.layers[layer].K[b][:, n - 1 - n_upd:n].transpose(1, 0, 2)
            stored_v = dec.layers[layer].V[b][:, n - 1 - n_upd:n].transpose(1, 0, 2)
            np.testing.assert_array_equal(stored_k, tr["k"][b, spec.window - n_upd:])
            np.testing.assert_array_equal(stored_v, tr["v"][b, spec.window - n_upd:])
