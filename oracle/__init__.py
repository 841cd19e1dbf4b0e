"""CPU oracle for the retrospective sparse-attention decode step.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The GPU library never
loads it and shares no code with it.

The arithmetic lives in ``retro_oracle.c`` (plain C, fp32 canonical page scores,
fp64 attention and merge); this module only owns the state arrays and marshals
them.  Every function cites the passage of the paper it follows in the C source.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "retro_oracle.c")
_LIB = os.path.join(_HERE, "libretro_oracle.so")


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no contraction, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off",
                               "-fno-fast-math", "-Wall", "-Wextra", "-Werror", "-fPIC", "-shared",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Dims(C.Structure):
    _fields_ = [("batch", C.c_int32), ("num_kv_heads", C.c_int32), ("group", C.c_int32),
                ("head_dim", C.c_int32), ("page_size", C.c_int32), ("budget", C.c_int32),
                ("window", C.c_int32), ("max_tokens", C.c_int32), ("sm_scale", C.c_double),
                ("budget_permille", C.c_int32)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = C.CDLL(_LIB)
        P = C.c_void_p
        D = C.POINTER(_Dims)
        i32 = C.c_int32
        lib.oracle_k_max.argtypes = [D]
        lib.oracle_k_max.restype = i32
        lib.oracle_prefill.argtypes = [D, i32, i32, P, P, P, P, P, P, P]
        lib.oracle_prefill.restype = C.c_int
        lib.oracle_append.argtypes = [D, i32, P, P, P, P, P, P, P, P]
        lib.oracle_append.restype = C.c_int
        lib.oracle_update_kv.argtypes = [D, i32, P, P, P, P, P, P, P]
        lib.oracle_update_kv.restype = None
        lib.oracle_score.argtypes = [D, P, P, P, P, P]
        lib.oracle_score.restype = None
        lib.oracle_select.argtypes = [D, P, P, P, P]
        lib.oracle_select.restype = None
        lib.oracle_build_mask.argtypes = [D, i32, P, P, P, P]
        lib.oracle_build_mask.restype = None
        lib.oracle_attend.argtypes = [D, i32, P, P, P, P, P, P, P, P, P]
        lib.oracle_attend.restype = None
        lib.oracle_merge.argtypes = [D, i32, P, P, P, P, P, P]
        lib.oracle_merge.restype = None
        lib.oracle_lse_merge.argtypes = [i32, P, C.c_double, P, C.c_double, P, P]
        lib.oracle_lse_merge.restype = None
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = i32
        _lib = lib
    return _lib


def _p(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().oracle_num_threads())


def lse_merge(oa, za, ob, zb):
    """Merge two partial outputs (eq. merged_attn); returns (O, Z) in fp64."""
    lib = _load()
    oa = np.ascontiguousarray(oa, np.float64)
    ob = np.ascontiguousarray(ob, np.float64)
    o = np.zeros_like(oa)
    z = np.zeros(1, np.float64)
    lib.oracle_lse_merge(oa.size, _p(oa), float(za), _p(ob), float(zb), _p(o), _p(z))
    return o, float(z[0])


class Oracle:
    """State of one attention layer of one batch, held on the host."""

    def __init__(self, batch: int, num_kv_heads: int, group: int, head_dim: int,
                 page_size: int, budget: int, window: int, max_tokens: int,
                 sm_scale: Optional[float] = None, budget_permille: int = 0,
                 reuse_interval: int = 0):
        self.lib = _load()
        # top-k reuse (the selection-reuse baseline of the motivational study,
        # Table 4): the page selection is refreshed on steps t with t mod f == 0
        # and kept, unscored, on the others; 0 or 1: every step
        self.reuse_interval = reuse_interval
        self._kept = None
        if sm_scale is None:
            sm_scale = float(np.float32(1.0 / np.sqrt(head_dim)))
        self.dims = _Dims(batch, num_kv_heads, group, head_dim, page_size, budget, window,
                          max_tokens, sm_scale, budget_permille)
        self._d = C.byref(self.dims)
        self.batch, self.hk, self.G, self.d = batch, num_kv_heads, group, head_dim
        self.P, self.W, self.max_tokens = page_size, window, max_tokens
        self.hq = num_kv_heads * group
        self.max_pages = -(-max_tokens // page_size)
        self.k_max = int(self.lib.oracle_k_max(self._d))
        b, hk, d = batch, num_kv_heads, head_dim
        self.K = np.zeros((b, hk, max_tokens, d), np.float32)
        self.V = np.zeros((b, hk, max_tokens, d), np.float32)
        self.kmin = np.zeros((b, hk, self.max_pages, d), np.float32)
        self.kmax = np.zeros((b, hk, self.max_pages, d), np.float32)
        self.A = np.full((b, hk, self.max_pages), -1, np.int32)
        self.seq_lens = np.zeros(b, np.int32)
        self.o_cache = np.zeros((b, max(window, 1), self.hq, d), np.float64)
        self.lse_cache = np.full((b, max(window, 1), self.hq), -np.inf, np.float64)

    @classmethod
    def for_spec(cls, spec, sm_scale: Optional[float] = None, **over) -> "Oracle":
        kw = dict(batch=spec.batch, num_kv_heads=spec.num_kv_heads, group=spec.group,
                  head_dim=spec.head_dim, page_size=spec.page_size, budget=spec.budget,
                  window=spec.window, max_tokens=spec.max_tokens, sm_scale=sm_scale,
                  budget_permille=spec.budget_permille, reuse_interval=spec.reuse_interval)
        kw.update(over)
        return cls(**kw)

    # -- phases ----------------------------------------------------------------
    def prefill(self, b: int, k: np.ndarray, v: np.ndarray) -> None:
        k = np.ascontiguousarray(k, np.float32)
        v = np.ascontiguousarray(v, np.float32)
        rc = self.lib.oracle_prefill(self._d, b, k.shape[0], _p(self.seq_lens), _p(self.K),
                                     _p(self.V), _p(self.kmin), _p(self.kmax), _p(k), _p(v))
        if rc != 0:
            raise ValueError("prefill exceeds max_tokens")

    def append(self, step: int, k_new: np.ndarray, v_new: np.ndarray) -> None:
        k_new = np.ascontiguousarray(k_new, np.float32)
        v_new = np.ascontiguousarray(v_new, np.float32)
        rc = self.lib.oracle_append(self._d, step, _p(self.seq_lens), _p(self.K), _p(self.V),
                                    _p(self.kmin), _p(self.kmax), _p(self.A), _p(k_new),
                                    _p(v_new))
        if rc != 0:
            raise ValueError("append exceeds max_tokens")

    def update_kv(self, k_upd: np.ndarray, v_upd: np.ndarray) -> None:
        """UpdateKV (Alg. 1): k_upd, v_upd [batch][n][h_k][d] replace the n most recent
        stored tokens of every sequence; their pages' digests are recomputed."""
        k_upd = np.ascontiguousarray(k_upd, np.float32)
        v_upd = np.ascontiguousarray(v_upd, np.float32)
        self.lib.oracle_update_kv(self._d, k_upd.shape[1], _p(self.seq_lens), _p(self.K),
                                  _p(self.V), _p(self.kmin), _p(self.kmax), _p(k_upd), _p(v_upd))

    def score(self, q_cur: np.ndarray) -> np.ndarray:
        q_cur = np.ascontiguousarray(q_cur, np.float32)
        s = np.zeros((self.batch, self.hk, self.max_pages), np.float32)
        self.lib.oracle_score(self._d, _p(q_cur), _p(self.kmin), _p(self.kmax),
                              _p(self.seq_lens), _p(s))
        return s

    def select(self, scores: np.ndarray):
        scores = np.ascontiguousarray(scores, np.float32)
        sel = np.zeros((self.batch, self.hk, self.k_max), np.int32)
        num = np.zeros((self.batch, self.hk), np.int32)
        self.lib.oracle_select(self._d, _p(scores), _p(self.seq_lens), _p(sel), _p(num))
        return sel, num

    def refreshes(self, step: int) -> bool:
        """Whether PageSelect runs at this step (always, unless top-k reuse keeps the
        selection of the last refresh step: steps t with t mod f != 0)."""
        f = self.reuse_interval
        return f < 2 or step % f == 0 or self._kept is None

    def build_mask(self, step: int, sel: np.ndarray, num: np.ndarray) -> np.ndarray:
        M = np.zeros_like(sel)
        self.lib.oracle_build_mask(self._d, step, _p(sel), _p(num), _p(self.A), _p(M))
        return M

    def attend(self, step: int, q_window: np.ndarray, sel, num, M):
        q_window = np.ascontiguousarray(q_window, np.float32)
        rows = self.W + 1
        o = np.zeros((self.batch, rows, self.hq, self.d), np.float64)
        z = np.zeros((self.batch, rows, self.hq), np.float64)
        self.lib.oracle_attend(self._d, step, _p(q_window), _p(self.K), _p(self.V),
                               _p(self.seq_lens), _p(sel), _p(num), _p(M), _p(o), _p(z))
        return o, z

    def merge(self, step: int, o_part: np.ndarray, lse_part: np.ndarray):
        rows = self.W + 1
        o_out = np.zeros((self.batch, rows, self.hq, self.d), np.float64)
        z_out = np.zeros((self.batch, rows, self.hq), np.float64)
        self.lib.oracle_merge(self._d, step, _p(np.ascontiguousarray(o_part)),
                              _p(np.ascontiguousarray(lse_part)), _p(self.o_cache),
                              _p(self.lse_cache), _p(o_out), _p(z_out))
        return o_out, z_out

    # -- one decode step (Alg. 1 without its UpdateKV step) ----------------------
    def step(self, t: int, k_new: np.ndarray, v_new: np.ndarray, q_window: np.ndarray,
             attend: bool = True) -> Dict[str, np.ndarray]:
        """k_new, v_new: [T][batch][h_k][d] (T tokens appended this step, the query
        sitting on the last); q_window: [batch][W+1][h_q][d]."""
        k_new = np.asarray(k_new, np.float32)
        v_new = np.asarray(v_new, np.float32)
        if k_new.ndim == 3:
            k_new, v_new = k_new[None], v_new[None]
        for j in range(k_new.shape[0]):
            self.append(t, k_new[j], v_new[j])
        if self.refreshes(t):
            scores = self.score(q_window[:, -1])
            sel, num = self.select(scores)
            self._kept = (sel.copy(), num.copy())
        else:
            # top-k reuse: the pages of the last refresh step, as they were selected;
            # Alg. 2's mask and last_loaded update apply to them unchanged
            scores = None
            sel, num = self._kept[0].copy(), self._kept[1].copy()
        M = self.build_mask(t, sel, num)
        out = dict(scores=scores, selected=sel, num_selected=num, mask=M,
                   seq_lens=self.seq_lens.copy())
        if attend:
            o_part, z_part = self.attend(t, q_window, sel, num, M)
            o_out, z_out = self.merge(t, o_part, z_part)
            out.update(o_part=o_part, lse_part=z_part, o_out=o_out, lse_out=z_out)
        return out
