"""CPU oracle of a multi-layer synthetic decode with retrospective re-embedding.

TEST INFRASTRUCTURE ONLY (like the rest of ``oracle/``): only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use it.

What it computes (Sec. 3.3, "Influences on deeper layers", with Alg. 1 in every
layer): at decode step t every layer l sees the W+1 window rows tau = t-W .. t.
Row t is embedded for the first time; the W past rows carry the (possibly
updated) outputs of the layer below, so their queries, keys and values are
computed again ("re-embedding"):

* ``X(l) = H(l)`` rounded to the storage type, ``Q, K, V = X(l) Wq, X(l) Wk, X(l) Wv``
  (fp64 products, rounded to the storage type);
* UpdateKV overwrites the stored keys and values of the past rows that were
  themselves decoded (rows of prompt positions are left alone), AppendKV stores
  row t's, and the layer's step (selection, mask, attention over the window,
  merge with the output cache) runs as in ``Oracle.step``;
* ``H(l+1) = H(l) + O(l) Wo``: the merged outputs, rounded to the storage type,
  through the output projection, whose result is rounded to the storage type and
  added to the residual stream.

``H(0)`` holds the token embeddings of the window (zero for rows before the first
decode step).  Feed-forward blocks and normalisation are left out: the paper's
figure of this mechanism omits them too, and they do not touch the KV cache.
The rounding points are those of a bf16 GEMM with a bf16 result; the residual
stream itself is kept in fp64.
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np

from . import Oracle


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round to float32, then (bf16) to the nearest bf16 with ties to even;
    returns float32 values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype != "bf16":
        return x
    bits = x.view(np.uint32).astype(np.uint64)
    keep = (bits + 0x7FFF + ((bits >> 16) & 1)) >> 16
    return (keep << 16).astype(np.uint32).view(np.float32).reshape(x.shape)


class OracleDecoder:
    """``num_layers`` Oracle layers joined by random-weight projections."""

    def __init__(self, spec, weights: List[dict], sm_scale: Optional[float] = None):
        self.spec = spec
        self.dtype = spec.dtype
        self.W = spec.window
        self.weights = [{k: np.asarray(v, np.float64) for k, v in w.items()} for w in weights]
        self.layers = [Oracle.for_spec(spec, sm_scale=sm_scale) for _ in weights]
        self.decoded = 0   # decode steps run so far

    # -- the three parts of one layer ---------------------------------------------
    def project(self, layer: int, x: np.ndarray):
        """x [batch][W+1][d_model] (storage-type values) -> q [b][W+1][h_q][d],
        k, v [b][W+1][h_k][d]."""
        s, w = self.spec, self.weights[layer]
        x = np.asarray(x, np.float64)
        b, rows = x.shape[:2]
        q = round_to(x @ w["wq"], self.dtype).reshape(b, rows, s.num_q_heads, s.head_dim)
        k = round_to(x @ w["wk"], self.dtype).reshape(b, rows, s.num_kv_heads, s.head_dim)
        v = round_to(x @ w["wv"], self.dtype).reshape(b, rows, s.num_kv_heads, s.head_dim)
        return q, k, v

    def attend_layer(self, layer: int, t: int, q, k, v, n_upd: int) -> Dict[str, np.ndarray]:
        """UpdateKV for the last n_upd past rows, then the layer's step at t."""
        lay, W = self.layers[layer], self.W
        if n_upd > 0:
            lay.update_kv(k[:, W - n_upd:W], v[:, W - n_upd:W])
        return lay.step(t, k[:, W], v[:, W], q)

    def out_proj(self, layer: int, o: np.ndarray) -> np.ndarray:
        """o [b][W+1][h_q][d] (fp64 merged outputs) -> [b][W+1][d_model]."""
        b, rows = o.shape[:2]
        o_s = np.asarray(round_to(o.reshape(b, rows, -1), self.dtype), np.float64)
        return np.asarray(round_to(o_s @ self.weights[layer]["wo"], self.dtype), np.float64)

    # -- one decode step of the whole stack -----------------------------------------
    def n_update(self) -> int:
        """Past rows whose keys and values are re-embedded this step: the decoded ones
        among the W."""
        return min(self.W, self.decoded)

    def step(self, t: int, emb_window: np.ndarray, trace: Optional[list] = None) -> np.ndarray:
        """emb_window [batch][W+1][d_model]: embeddings of the window's tokens.
        Returns the residual stream after the last layer, [batch][W+1][d_model]."""
        h = np.asarray(emb_window, np.float64).copy()
        n_upd = self.n_update()
        for layer in range(len(self.layers)):
            x = round_to(h, self.dtype)
            q, k, v = self.project(layer, x)
            out = self.attend_layer(layer, t, q, k, v, n_upd)
            y = self.out_proj(layer, out["o_out"])
            if trace is not None:
                trace.append(dict(x=x, q=q, k=k, v=v, y=y, **out))
            h = h + y
        self.decoded += 1
        return h
