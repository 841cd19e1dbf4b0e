"""Device buffers of one attention layer and convenience wrappers of the C ABI.

PyTorch only allocates device memory here; every step of the decode path runs in
the gfx950 library (binding.py).  Layouts are the ones documented in
include/retro.h.
"""
from __future__ import annotations

import math
from typing import Optional

import torch

from . import binding as B

_TORCH_DTYPE = {"bf16": torch.bfloat16, "f32": torch.float32}
_RETRO_DTYPE = {"bf16": B.RETRO_BF16, "f32": B.RETRO_F32}


class RetroLayer:
    """State of one layer: paged KV cache, digests, retrospective mask, selection,
    output cache, outputs and workspace, all on one device."""

    def __init__(self, batch: int, num_kv_heads: int, group: int, head_dim: int, page_size: int,
                 budget: int, window: int, max_pages: int, dtype: str = "bf16",
                 num_phys_pages: Optional[int] = None, page_table: Optional[torch.Tensor] = None,
                 sm_scale: float = 0.0, budget_permille: int = 0, flags: int = 0,
                 reuse_interval: int = 0,
                 device: str = "cuda"):
        self.device = torch.device(device)
        if num_phys_pages is None:
            num_phys_pages = batch * max_pages
        self.dims = B.Dims(batch, num_kv_heads, group, head_dim, page_size, budget, window,
                           max_pages, num_phys_pages, _RETRO_DTYPE[dtype], sm_scale,
                           budget_permille, flags, reuse_interval)
        self.k_max = B.retro_k_max(self.dims)
        self.ws_bytes = B.retro_workspace_size(self.dims)
        self.batch, self.hk, self.G, self.d = batch, num_kv_heads, group, head_dim
        self.hq, self.P, self.W = num_kv_heads * group, page_size, window
        self.dtype = _TORCH_DTYPE[dtype]
        dev, td = self.device, self.dtype
        hk, d, P = num_kv_heads, head_dim, page_size
        self.k_cache = torch.zeros(num_phys_pages, hk, P, d, dtype=td, device=dev)
        self.v_cache = torch.zeros(num_phys_pages, hk, d, P, dtype=td, device=dev)
        # per logical page of each sequence, as the header lays it out (not per
        # physical page: the pool may hold more or fewer pages than batch * max_pages)
        self.digest = torch.zeros(batch, hk, max_pages, 2, d, dtype=td, device=dev)
        if page_table is None:
            page_table = torch.arange(batch * max_pages, dtype=torch.int32).view(batch, max_pages)
        self.page_table = page_table.to(device=dev, dtype=torch.int32).contiguous()
        self.seq_lens = torch.zeros(batch, dtype=torch.int32, device=dev)
        self.last_loaded = torch.full((batch, hk, max_pages), -1, dtype=torch.int32, device=dev)
        self.selected = torch.full((batch, hk, self.k_max), -1, dtype=torch.int32, device=dev)
        self.mask = torch.full((batch, hk, self.k_max), -1, dtype=torch.int32, device=dev)
        self.num_selected = torch.zeros(batch, hk, dtype=torch.int32, device=dev)
        Wc = max(window, 1)
        self.o_cache = torch.zeros(batch, Wc, self.hq, d, dtype=torch.float32, device=dev)
        self.lse_cache = torch.full((batch, Wc, self.hq), -math.inf, dtype=torch.float32,
                                    device=dev)
        self.o_out = torch.zeros(batch, window + 1, self.hq, d, dtype=torch.float32, device=dev)
        self.lse_out = torch.zeros(batch, window + 1, self.hq, dtype=torch.float32, device=dev)
        self.o_part = torch.zeros_like(self.o_out)
        self.lse_part = torch.zeros_like(self.lse_out)
        self.workspace = torch.zeros(max(self.ws_bytes, 256), dtype=torch.uint8, device=dev)
        self.cache = B.KVCache(self.k_cache.data_ptr(), self.v_cache.data_ptr(),
                               self.digest.data_ptr(), self.page_table.data_ptr(),
                               self.seq_lens.data_ptr(), self.last_loaded.data_ptr())
        self.sel = B.Selection(self.selected.data_ptr(), self.mask.data_ptr(),
                               self.num_selected.data_ptr())
        self.ocache = B.OutputCache(self.o_cache.data_ptr(), self.lse_cache.data_ptr())
        self._lens = [0] * batch  # host mirror of seq_lens, for prefill positions

    @classmethod
    def for_spec(cls, spec, **kw) -> "RetroLayer":
        args = dict(batch=spec.batch, num_kv_heads=spec.num_kv_heads, group=spec.group,
                    head_dim=spec.head_dim, page_size=spec.page_size, budget=spec.budget,
                    window=spec.window, max_pages=spec.max_pages, dtype=spec.dtype,
                    budget_permille=spec.budget_permille,
                    reuse_interval=getattr(spec, "reuse_interval", 0))
        args.update(kw)
        return cls(**args)

    def _dev(self, x) -> torch.Tensor:
        if not isinstance(x, torch.Tensor):
            x = torch.from_numpy(x)
        return x.to(device=self.device, dtype=self.dtype).contiguous()

    # -- calls ----------------------------------------------------------------------
    def prefill(self, seq: int, k, v, stream=None) -> None:
        k, v = self._dev(k), self._dev(v)
        n = k.shape[0]
        B.retro_prefill_kv(self.dims, self.cache, seq, self._lens[seq], n, k, v, stream)
        self._lens[seq] += n
        self._keep = (k, v)  # keep sources alive until the copy has run

    def append(self, step: int, k_new, v_new, stream=None) -> None:
        k_new, v_new = self._dev(k_new), self._dev(v_new)
        B.retro_append_kv(self.dims, step, self.cache, k_new, v_new, stream)
        for b in range(self.batch):
            self._lens[b] += 1

    def append_tokens(self, step: int, k_new, v_new, stream=None) -> None:
        """Several tokens per sequence in one call: k_new / v_new [n][batch][h_k][d]."""
        k_new, v_new = self._dev(k_new), self._dev(v_new)
        n = int(k_new.shape[0])
        B.retro_append_kv_tokens(self.dims, step, self.cache, n, k_new, v_new, stream)
        for b in range(self.batch):
            self._lens[b] += n
        self._keep_append = (k_new, v_new)
        self._keep = (k_new, v_new)

    def select(self, step: int, q_cur, stream=None) -> None:
        q_cur = self._dev(q_cur)
        B.retro_select_pages(self.dims, step, q_cur, self.cache, self.sel, self.workspace,
                             self.ws_bytes, stream)
        self._keep = q_cur

    def attend(self, step: int, q_window, stream=None) -> None:
        q_window = self._dev(q_window)
        B.retro_decode_attend(self.dims, step, q_window, self.cache, self.sel, self.o_part,
                              self.lse_part, self.workspace, self.ws_bytes, stream)
        self._keep = q_window

    def attend_partials(self, step: int, q_window: torch.Tensor, stream=None) -> None:
        """Attention kernel only (partials stay in the workspace); q_window on device."""
        B.retro_decode_attend_partials(self.dims, step, q_window, self.cache, self.sel,
                                       self.workspace, self.ws_bytes, stream)

    def update_kv(self, k_upd, v_upd, stream=None) -> None:
        """UpdateKV: new keys / values [batch][n][h_k][d] for the n most recent stored
        tokens of every sequence (their pages' digests are recomputed)."""
        k_upd, v_upd = self._dev(k_upd), self._dev(v_upd)
        B.retro_update_kv(self.dims, self.cache, int(k_upd.shape[1]), k_upd, v_upd, stream)
        self._keep_upd = (k_upd, v_upd)

    def step_attend_partials(self, step: int, q_window: torch.Tensor, stream=None) -> None:
        """The step's launch that ends in the attention partials (scores where the step
        computes them there, selection, attention) alone; overwrites the selection
        outputs, not last_loaded."""
        B.retro_step_attend_partials(self.dims, step, q_window, self.cache, self.sel,
                                       self.workspace, self.ws_bytes, stream)

    def scores(self, stream=None) -> torch.Tensor:
        """The page scores [batch][h_k][max_pages] fp32 of the last call that computed
        them (entries past a sequence's pages are unspecified)."""
        out = torch.empty(self.batch, self.hk, self.dims.max_pages, dtype=torch.float32,
                          device=self.device)
        B.retro_copy_scores(self.dims, self.workspace, self.ws_bytes, out, stream)
        return out

    def merge(self, step: int, stream=None) -> None:
        B.retro_merge_output_cache(self.dims, step, self.o_part, self.lse_part, self.ocache,
                                   self.o_out, self.lse_out, stream)

    def step(self, step: int, q_window, k_new, v_new, stream=None, noalloc: bool = False) -> None:
        """One retro_step (noalloc: retro_step_noalloc, the library's static scratch in
        place of this layer's workspace)."""
        q_window, k_new, v_new = self._dev(q_window), self._dev(k_new), self._dev(v_new)
        if noalloc:
            B.retro_step_noalloc(self.dims, step, q_window, k_new, v_new, self.cache, self.sel,
                                 self.ocache, self.o_out, self.lse_out, stream)
        else:
            B.retro_step(self.dims, step, q_window, k_new, v_new, self.cache, self.sel,
                         self.ocache, self.o_out, self.lse_out, self.workspace, self.ws_bytes,
                         stream)
        for b in range(self.batch):
            self._lens[b] += 1
        self._keep = (q_window, k_new, v_new)
