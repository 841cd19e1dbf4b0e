"""Multi-layer decode with retrospective re-embedding (Sec. 3.3, "Influences on
deeper layers"; Alg. 1 in every layer).

At step t every layer sees the W+1 window rows t-W .. t.  The newest row is
embedded for the first time; the W past rows carry the layer below's updated
outputs, so their queries, keys and values are computed again: UpdateKV
(``retro_update_kv``) overwrites the stored keys and values of the decoded past
rows, and the layer's step (``retro_step``) appends the newest token and attends
all W+1 queries.  Layers are joined by a residual stream kept in fp32:
``H(l+1) = H(l) + O(l) Wo``.

The projections are dense products over (W+1) * batch rows, the case the paper's
linear-layer analysis (Appendix, linear layer overhead) prices: bound by reading
the weights.  In bf16 they run in the library too (``retro_project_qkv``: one
launch for the query, key and value projections of a layer, weights pre-tiled by
``retro_pack_weight``; ``retro_project_out``: the output projection fused with the
residual add and the next layer's bf16 input), both bf16 in, fp32 accumulation,
bf16 out.  fp32 stacks use ``retro_project_f32`` (fp32 fused multiply-add
chains on the unpacked weights, the output projection added into the residual
stream in place).
Feed-forward blocks and normalisation are left out: they do not touch the KV
cache.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import binding as B
from .layer import RetroLayer


class RetroDecoder:
    """``len(weights)`` RetroLayers joined by query/key/value and output projections.

    ``weights``: per layer a dict of ``wq [d_model][h_q*d]``, ``wk``, ``wv
    [d_model][h_k*d]`` and ``wo [h_q*d][d_model]`` (host arrays or device tensors);
    ``d_model = h_q * d``.  ``layer_kw`` are the RetroLayer arguments shared by all
    layers (batch, num_kv_heads, group, head_dim, page_size, budget, window,
    max_pages, dtype, budget_permille, ...).  ``library_projections=False`` keeps
    the products on torch.matmul (for comparison); with the library projections,
    ``fuse_update`` folds UpdateKV into the query / key / value launch
    (``retro_project_qkv_update``) instead of a ``retro_update_kv`` of its own.
    """

    def __init__(self, weights: Sequence[dict], device: str = "cuda",
                 library_projections: bool = True, fuse_update: bool = True, **layer_kw):
        self.device = torch.device(device)
        self.layers: List[RetroLayer] = [RetroLayer(device=device, **layer_kw)
                                         for _ in weights]
        lay = self.layers[0]
        self.dtype = lay.dtype
        self.W, self.batch, self.hq, self.hk, self.d = lay.W, lay.batch, lay.hq, lay.hk, lay.d
        self.d_model = self.hq * self.d
        self.weights = []
        for w in weights:
            dw = {}
            for name in ("wq", "wk", "wv", "wo"):
                x = w[name]
                if not isinstance(x, torch.Tensor):
                    x = torch.from_numpy(x)
                dw[name] = x.to(device=self.device, dtype=self.dtype).contiguous()
            if dw["wq"].shape != (self.d_model, self.hq * self.d) or \
               dw["wk"].shape != (self.d_model, self.hk * self.d) or \
               dw["wv"].shape != (self.d_model, self.hk * self.d) or \
               dw["wo"].shape != (self.hq * self.d, self.d_model):
                raise ValueError("projection shapes do not match the layer geometry")
            self.weights.append(dw)
        self.decoded = 0  # decode steps run so far
        # bf16: library projections (weights pre-tiled; they need k % 1024 == 0 and
        # at most 112 rows)
        rows = self.batch * (self.W + 1)
        self.fused = (library_projections and self.dtype == torch.bfloat16 and
                      self.d_model % 1024 == 0 and
                      (self.hq * self.d) % 1024 == 0 and rows <= 112)
        if self.fused:
            nq, nkv = self.hq * self.d, self.hk * self.d
            self.packed = []
            for dw in self.weights:
                wqkv = torch.cat([dw["wq"], dw["wk"], dw["wv"]], dim=1).contiguous()
                pq = torch.empty_like(wqkv)
                po = torch.empty_like(dw["wo"])
                B.retro_pack_weight(wqkv, self.d_model, nq + 2 * nkv, pq)
                B.retro_pack_weight(dw["wo"], nq, self.d_model, po)
                self.packed.append((pq, po))
            torch.cuda.synchronize(self.device)
            dev, td = self.device, self.dtype
            self.h = torch.zeros(self.batch, self.W + 1, self.d_model, dtype=torch.float32,
                                 device=dev)
            self.x = torch.zeros(self.batch, self.W + 1, self.d_model, dtype=td, device=dev)
            self.q = torch.zeros(self.batch, self.W + 1, self.hq, self.d, dtype=td, device=dev)
            self.k = torch.zeros(self.batch, self.W + 1, self.hk, self.d, dtype=td, device=dev)
            self.v = torch.zeros_like(self.k)
            self.k_new = torch.zeros(self.batch, self.hk, self.d, dtype=td, device=dev)
            self.v_new = torch.zeros_like(self.k_new)
        self.fuse_update = self.fused and fuse_update
        # fp32: library projections on the unpacked weights (retro_project_f32)
        self.f32_library = library_projections and self.dtype == torch.float32
        if self.f32_library:
            dev = self.device
            self.h = torch.zeros(self.batch, self.W + 1, self.d_model, dtype=torch.float32,
                                 device=dev)
            self.q = torch.zeros(self.batch, self.W + 1, self.hq, self.d, dtype=torch.float32,
                                 device=dev)
            self.k = torch.zeros(self.batch, self.W + 1, self.hk, self.d, dtype=torch.float32,
                                 device=dev)
            self.v = torch.zeros_like(self.k)

    def prefill(self, layer: int, seq: int, k, v, stream=None) -> None:
        """Prompt keys and values [n][h_k][d] of one sequence in one layer."""
        self.layers[layer].prefill(seq, k, v, stream)

    def n_update(self) -> int:
        """Past rows re-embedded this step: the decoded ones among the W."""
        return min(self.W, self.decoded)

    def step(self, t: int, emb_window: torch.Tensor, trace: Optional[list] = None
             ) -> torch.Tensor:
        """One decode step of the whole stack on the current stream.

        emb_window: [batch][W+1][d_model] device tensor, the embeddings of the
        window's tokens (row W the newest; zero rows before the first decode step).
        Returns the residual stream after the last layer, [batch][W+1][d_model]
        fp32 (with the library projections, a buffer of the decoder that the next
        step overwrites).  ``trace`` (a list) receives per layer the tensors the
        layer saw and produced (for tests).
        """
        b, rows, W = self.batch, self.W + 1, self.W
        if tuple(emb_window.shape) != (b, rows, self.d_model):
            raise ValueError("emb_window must be [batch][W+1][d_model]")
        n_upd = self.n_update()
        if self.fused:
            return self._step_fused(t, emb_window, n_upd, trace)
        if self.f32_library:
            return self._step_f32(t, emb_window, n_upd, trace)
        h = emb_window.to(device=self.device, dtype=torch.float32)
        for lay, w in zip(self.layers, self.weights):
            x = h.to(self.dtype)
            q = torch.matmul(x, w["wq"]).view(b, rows, self.hq, self.d)
            k = torch.matmul(x, w["wk"]).view(b, rows, self.hk, self.d)
            v = torch.matmul(x, w["wv"]).view(b, rows, self.hk, self.d)
            if n_upd > 0:
                lay.update_kv(k[:, W - n_upd:W], v[:, W - n_upd:W])
            lay.step(t, q, k[:, W], v[:, W])
            y = torch.matmul(lay.o_out.to(self.dtype).view(b, rows, self.d_model), w["wo"])
            if trace is not None:
                trace.append(dict(x=x.clone(), q=q.clone(), k=k.clone(), v=v.clone(),
                                  o_out=lay.o_out.clone(), lse_out=lay.lse_out.clone(),
                                  selected=lay.selected.clone(), mask=lay.mask.clone(),
                                  num_selected=lay.num_selected.clone(), y=y.clone()))
            h = h + y.float()
        self.decoded += 1
        return h

    def _step_f32(self, t, emb_window, n_upd, trace):
        """fp32 stack: every product in the library (retro_project_f32), the
        residual stream itself the next layer's input."""
        b, rows, W = self.batch, self.W + 1, self.W
        nq, nkv, r = self.hq * self.d, self.hk * self.d, self.batch * (self.W + 1)
        self.h.copy_(emb_window)
        for lay, w in zip(self.layers, self.weights):
            h_in = self.h.clone() if trace is not None else None
            B.retro_project_f32(self.h, r, self.d_model, w["wq"], nq, self.q)
            B.retro_project_f32(self.h, r, self.d_model, w["wk"], nkv, self.k)
            B.retro_project_f32(self.h, r, self.d_model, w["wv"], nkv, self.v)
            if n_upd > 0:
                lay.update_kv(self.k[:, W - n_upd:W], self.v[:, W - n_upd:W])
            lay.step(t, self.q, self.k[:, W], self.v[:, W])
            B.retro_project_f32(lay.o_out, r, nq, w["wo"], self.d_model, self.h, accumulate=True)
            if trace is not None:
                trace.append(dict(x=h_in, q=self.q.clone(), k=self.k.clone(), v=self.v.clone(),
                                  o_out=lay.o_out.clone(), lse_out=lay.lse_out.clone(),
                                  selected=lay.selected.clone(), mask=lay.mask.clone(),
                                  num_selected=lay.num_selected.clone(), y=self.h - h_in))
        self.decoded += 1
        return self.h

    def _step_fused(self, t, emb_window, n_upd, trace):
        b, rows, W = self.batch, self.W + 1, self.W
        nq, nkv = self.hq * self.d, self.hk * self.d
        self.h.copy_(emb_window)
        self.x.copy_(emb_window)
        for lay, (pq, po) in zip(self.layers, self.packed):
            h_in = self.h.clone() if trace is not None else None
            x_in = self.x.clone() if trace is not None else None
            if self.fuse_update:
                B.retro_project_qkv_update(lay.dims, lay.cache, self.x, self.d_model, pq, n_upd,
                                           self.q, self.k_new, self.v_new)
                k_new, v_new = self.k_new, self.v_new
            else:
                B.retro_project_qkv(self.x, b * rows, self.d_model, pq, nq, nkv, self.q, self.k,
                                    self.v)
                if n_upd > 0:
                    lay.update_kv(self.k[:, W - n_upd:W], self.v[:, W - n_upd:W])
                k_new, v_new = self.k[:, W], self.v[:, W]
            lay.step(t, self.q, k_new, v_new)
            B.retro_project_out(lay.o_out, b * rows, nq, po, self.d_model, self.h, self.x)
            if trace is not None:
                kv = (dict(k_new=self.k_new.clone(), v_new=self.v_new.clone())
                      if self.fuse_update else dict(k=self.k.clone(), v=self.v.clone()))
                trace.append(dict(x=x_in, q=self.q.clone(), **kv,
                                  o_out=lay.o_out.clone(), lse_out=lay.lse_out.clone(),
                                  selected=lay.selected.clone(), mask=lay.mask.clone(),
                                  num_selected=lay.num_selected.clone(), h_in=h_in,
                                  h_out=self.h.clone(), x_next=self.x.clone(),
                                  y=self.h - h_in))
        self.decoded += 1
        return self.h


def layer_kwargs(spec, **over) -> dict:
    """RetroLayer arguments of a workload Spec (shared by every layer)."""
    kw = dict(batch=spec.batch, num_kv_heads=spec.num_kv_heads, group=spec.group,
              head_dim=spec.head_dim, page_size=spec.page_size, budget=spec.budget,
              window=spec.window, max_pages=spec.max_pages, dtype=spec.dtype,
              budget_permille=spec.budget_permille)
    kw.update(over)
    return kw


__all__ = ["RetroDecoder", "layer_kwargs"]
