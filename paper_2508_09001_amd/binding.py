"""ctypes binding of the C ABI declared in include/retro.h.

Argument marshalling only: every function forwards to the gfx950 library of the
same name.  Buffers may be passed as torch tensors (their device pointers are
used) or as raw integer addresses; ``stream`` defaults to torch's current HIP
stream.  A non-zero status raises :class:`RetroError`.  If the compiled library
is absent, loading fails loudly: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libretro_mi355x.so")

RETRO_OK, RETRO_EINVAL, RETRO_EUNSUPPORTED, RETRO_EHIP, RETRO_EWORKSPACE, RETRO_ESCRATCH = \
    0, -1, -2, -3, -4, -5
RETRO_F32, RETRO_BF16 = 0, 1
RETRO_FLAG_SEPARATE_SCORES, RETRO_FLAG_SELECT_IN_SCORES, RETRO_FLAG_TEST_WAIT_TIMEOUT = 1, 2, 4

EXPORTED = ("retro_version", "retro_status_string", "retro_k_max", "retro_workspace_size",
            "retro_prefill_kv", "retro_append_kv", "retro_append_kv_tokens", "retro_update_kv",
            "retro_select_pages",
            "retro_decode_attend", "retro_decode_attend_partials", "retro_step_attend_partials",
            "retro_copy_scores", "retro_merge_output_cache", "retro_step", "retro_step_noalloc",
            "retro_step_launches", "retro_pack_weight", "retro_project_qkv",
            "retro_project_qkv_update", "retro_project_out", "retro_project_f32")


class RetroError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {retro_status_string(status)} ({status})")


class Dims(C.Structure):
    _fields_ = [("batch", C.c_int32), ("num_kv_heads", C.c_int32), ("group", C.c_int32),
                ("head_dim", C.c_int32), ("page_size", C.c_int32), ("budget_tokens", C.c_int32),
                ("window", C.c_int32), ("max_pages", C.c_int32), ("num_phys_pages", C.c_int32),
                ("dtype", C.c_int32), ("sm_scale", C.c_float), ("budget_permille", C.c_int32),
                ("flags", C.c_int32), ("reuse_interval", C.c_int32)]


class KVCache(C.Structure):
    _fields_ = [("k_cache", C.c_void_p), ("v_cache", C.c_void_p), ("digest", C.c_void_p),
                ("page_table", C.c_void_p), ("seq_lens", C.c_void_p),
                ("last_loaded", C.c_void_p)]


class Selection(C.Structure):
    _fields_ = [("selected", C.c_void_p), ("mask", C.c_void_p), ("num_selected", C.c_void_p)]


class OutputCache(C.Structure):
    _fields_ = [("o_cache", C.c_void_p), ("lse_cache", C.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load the compiled library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    # PyTorch-ROCm ships its own HIP runtime under the same soname; load it first
    # so that this library binds to the runtime that owns torch's streams.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it first (__graft_entry__.build())")
    lib = C.CDLL(path)
    P, i32, D = C.c_void_p, C.c_int32, C.POINTER(Dims)
    sig = {
        "retro_version": ([], C.c_char_p),
        "retro_status_string": ([i32], C.c_char_p),
        "retro_k_max": ([D, C.POINTER(C.c_int32)], C.c_int),
        "retro_workspace_size": ([D, C.POINTER(C.c_size_t)], C.c_int),
        "retro_prefill_kv": ([D, C.POINTER(KVCache), i32, i32, i32, P, P, P], C.c_int),
        "retro_append_kv": ([D, i32, C.POINTER(KVCache), P, P, P], C.c_int),
        "retro_append_kv_tokens": ([D, i32, C.POINTER(KVCache), i32, P, P, P], C.c_int),
        "retro_update_kv": ([D, C.POINTER(KVCache), i32, P, P, P], C.c_int),
        "retro_select_pages": ([D, i32, P, C.POINTER(KVCache), C.POINTER(Selection), P,
                                C.c_size_t, P], C.c_int),
        "retro_decode_attend": ([D, i32, P, C.POINTER(KVCache), C.POINTER(Selection), P, P, P,
                                 C.c_size_t, P], C.c_int),
        "retro_decode_attend_partials": ([D, i32, P, C.POINTER(KVCache), C.POINTER(Selection), P,
                                          C.c_size_t, P], C.c_int),
        "retro_step_attend_partials": ([D, i32, P, C.POINTER(KVCache), C.POINTER(Selection), P,
                                          C.c_size_t, P], C.c_int),
        "retro_copy_scores": ([D, P, C.c_size_t, P, P], C.c_int),
        "retro_merge_output_cache": ([D, i32, P, P, C.POINTER(OutputCache), P, P, P], C.c_int),
        "retro_step": ([D, i32, P, P, P, C.POINTER(KVCache), C.POINTER(Selection),
                        C.POINTER(OutputCache), P, P, P, C.c_size_t, P], C.c_int),
        "retro_step_noalloc": ([D, i32, P, P, P, C.POINTER(KVCache), C.POINTER(Selection),
                                C.POINTER(OutputCache), P, P, P], C.c_int),
        "retro_step_launches": ([D, C.POINTER(C.c_int32)], C.c_int),
        "retro_pack_weight": ([P, i32, i32, P, P], C.c_int),
        "retro_project_qkv": ([P, i32, i32, P, i32, i32, P, P, P, P], C.c_int),
        "retro_project_out": ([P, i32, i32, P, i32, P, P, P], C.c_int),
        "retro_project_f32": ([P, i32, i32, P, i32, P, i32, P], C.c_int),
        "retro_project_qkv_update": ([D, C.POINTER(KVCache), P, i32, P, i32, P, P, P, P],
                                     C.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(st: int, where: str) -> None:
    if st != RETRO_OK:
        raise RetroError(st, where)


def retro_version() -> str:
    return load_library().retro_version().decode()


def retro_status_string(status: int) -> str:
    return load_library().retro_status_string(status).decode()


def retro_k_max(dims: Dims) -> int:
    k = C.c_int32(0)
    _check(load_library().retro_k_max(C.byref(dims), C.byref(k)), "retro_k_max")
    return k.value


def retro_workspace_size(dims: Dims) -> int:
    n = C.c_size_t(0)
    _check(load_library().retro_workspace_size(C.byref(dims), C.byref(n)), "retro_workspace_size")
    return n.value


def retro_prefill_kv(dims: Dims, cache: KVCache, seq: int, start_pos: int, n_tokens: int,
                     k_src, v_src, stream=None) -> None:
    _check(load_library().retro_prefill_kv(C.byref(dims), C.byref(cache), seq, start_pos,
                                           n_tokens, _ptr(k_src), _ptr(v_src), _stream(stream)),
           "retro_prefill_kv")


def retro_append_kv(dims: Dims, step: int, cache: KVCache, k_new, v_new, stream=None) -> None:
    _check(load_library().retro_append_kv(C.byref(dims), step, C.byref(cache), _ptr(k_new),
                                          _ptr(v_new), _stream(stream)), "retro_append_kv")


def retro_append_kv_tokens(dims: Dims, step: int, cache: KVCache, n_tokens: int, k_new, v_new,
                           stream=None) -> None:
    _check(load_library().retro_append_kv_tokens(C.byref(dims), step, C.byref(cache), n_tokens,
                                                 _ptr(k_new), _ptr(v_new), _stream(stream)),
           "retro_append_kv_tokens")


def retro_update_kv(dims: Dims, cache: KVCache, n_tokens: int, k_upd, v_upd, stream=None) -> None:
    _check(load_library().retro_update_kv(C.byref(dims), C.byref(cache), n_tokens, _ptr(k_upd),
                                          _ptr(v_upd), _stream(stream)), "retro_update_kv")


def retro_select_pages(dims: Dims, step: int, q_cur, cache: KVCache, sel: Selection, workspace,
                       ws_bytes: int, stream=None) -> None:
    _check(load_library().retro_select_pages(C.byref(dims), step, _ptr(q_cur), C.byref(cache),
                                             C.byref(sel), _ptr(workspace), ws_bytes,
                                             _stream(stream)), "retro_select_pages")


def retro_decode_attend(dims: Dims, step: int, q_window, cache: KVCache, sel: Selection, o_part,
                        lse_part, workspace, ws_bytes: int, stream=None) -> None:
    _check(load_library().retro_decode_attend(C.byref(dims), step, _ptr(q_window),
                                              C.byref(cache), C.byref(sel), _ptr(o_part),
                                              _ptr(lse_part), _ptr(workspace), ws_bytes,
                                              _stream(stream)), "retro_decode_attend")


def retro_decode_attend_partials(dims: Dims, step: int, q_window, cache: KVCache, sel: Selection,
                                 workspace, ws_bytes: int, stream=None) -> None:
    _check(load_library().retro_decode_attend_partials(C.byref(dims), step, _ptr(q_window),
                                                       C.byref(cache), C.byref(sel),
                                                       _ptr(workspace), ws_bytes, _stream(stream)),
           "retro_decode_attend_partials")


def retro_step_attend_partials(dims: Dims, step: int, q_window, cache: KVCache, sel: Selection,
                                 workspace, ws_bytes: int, stream=None) -> None:
    _check(load_library().retro_step_attend_partials(C.byref(dims), step, _ptr(q_window),
                                                       C.byref(cache), C.byref(sel),
                                                       _ptr(workspace), ws_bytes, _stream(stream)),
           "retro_step_attend_partials")


def retro_copy_scores(dims: Dims, workspace, ws_bytes: int, scores, stream=None) -> None:
    _check(load_library().retro_copy_scores(C.byref(dims), _ptr(workspace), ws_bytes,
                                            _ptr(scores), _stream(stream)), "retro_copy_scores")


def retro_merge_output_cache(dims: Dims, step: int, o_part, lse_part, ocache: OutputCache, o_out,
                             lse_out, stream=None) -> None:
    _check(load_library().retro_merge_output_cache(C.byref(dims), step, _ptr(o_part),
                                                   _ptr(lse_part), C.byref(ocache), _ptr(o_out),
                                                   _ptr(lse_out), _stream(stream)),
           "retro_merge_output_cache")


def retro_step(dims: Dims, step: int, q_window, k_new, v_new, cache: KVCache, sel: Selection,
               ocache: OutputCache, o_out, lse_out, workspace, ws_bytes: int,
               stream=None) -> None:
    _check(load_library().retro_step(C.byref(dims), step, _ptr(q_window), _ptr(k_new), _ptr(v_new),
                                     C.byref(cache), C.byref(sel), C.byref(ocache), _ptr(o_out),
                                     _ptr(lse_out), _ptr(workspace), ws_bytes, _stream(stream)),
           "retro_step")


def retro_step_launches(dims: Dims) -> int:
    """Kernel launches retro_step makes for dims on the current device."""
    n = C.c_int32(0)
    _check(load_library().retro_step_launches(C.byref(dims), C.byref(n)), "retro_step_launches")
    return n.value


def retro_step_noalloc(dims: Dims, step: int, q_window, k_new, v_new, cache: KVCache,
                       sel: Selection, ocache: OutputCache, o_out, lse_out, stream=None) -> None:
    _check(load_library().retro_step_noalloc(C.byref(dims), step, _ptr(q_window), _ptr(k_new),
                                             _ptr(v_new), C.byref(cache), C.byref(sel),
                                             C.byref(ocache), _ptr(o_out), _ptr(lse_out),
                                             _stream(stream)),
           "retro_step_noalloc")


def retro_pack_weight(w, k: int, n: int, w_packed, stream=None) -> None:
    _check(load_library().retro_pack_weight(_ptr(w), k, n, _ptr(w_packed), _stream(stream)),
           "retro_pack_weight")


def retro_project_qkv(x, rows: int, k: int, w_packed, n_q: int, n_kv: int, q, k_out, v,
                      stream=None) -> None:
    _check(load_library().retro_project_qkv(_ptr(x), rows, k, _ptr(w_packed), n_q, n_kv, _ptr(q),
                                            _ptr(k_out), _ptr(v), _stream(stream)),
           "retro_project_qkv")


def retro_project_out(o, rows: int, k: int, w_packed, n: int, h, x_next, stream=None) -> None:
    _check(load_library().retro_project_out(_ptr(o), rows, k, _ptr(w_packed), n, _ptr(h),
                                            _ptr(x_next), _stream(stream)), "retro_project_out")


def retro_project_f32(x, rows: int, k: int, w, n: int, y, accumulate: bool = False,
                      stream=None) -> None:
    _check(load_library().retro_project_f32(_ptr(x), rows, k, _ptr(w), n, _ptr(y),
                                            1 if accumulate else 0, _stream(stream)),
           "retro_project_f32")


def retro_project_qkv_update(dims: Dims, cache: KVCache, x, k: int, w_packed, n_update: int, q,
                             k_new, v_new, stream=None) -> None:
    _check(load_library().retro_project_qkv_update(C.byref(dims), C.byref(cache), _ptr(x), k,
                                                   _ptr(w_packed), n_update, _ptr(q),
                                                   _ptr(k_new), _ptr(v_new), _stream(stream)),
           "retro_project_qkv_update")
