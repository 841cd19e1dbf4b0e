"""The C-ABI library (CPU-only checks): it loads, exports every declared symbol,
and rejects bad arguments on the host before anything is enqueued."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_2508_09001_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return binding


def _declared():
    with open(os.path.join(ROOT, "include", "retro.h")) as f:
        text = f.read()
    return set(re.findall(r"^\s*(?:const char\*|retro_status)\s+(retro_\w+)\s*\(", text, re.M))


def test_header_declares_the_documented_entry_points(lib):
    assert _declared() == set(lib.EXPORTED)


def test_library_exports_every_declared_symbol(lib):
    raw = C.CDLL(lib.LIB_PATH)
    for name in _declared():
        assert hasattr(raw, name), name


def test_version_and_status_strings(lib):
    assert "gfx950" in lib.retro_version()
    for st in (0, -1, -2, -3, -4):
        assert lib.retro_status_string(st).startswith("RETRO_")
    assert "unknown" in lib.retro_status_string(7)


def _dims(lib, **kw):
    base = dict(batch=1, num_kv_heads=8, group=4, head_dim=128, page_size=16, budget_tokens=2048,
                window=16, max_pages=2080, num_phys_pages=2080, dtype=lib.RETRO_BF16, sm_scale=0.0)
    base.update(kw)
    return lib.Dims(**base)


@pytest.mark.parametrize("field,value,status", [
    ("batch", 0, -1), ("num_kv_heads", -2, -1), ("group", 0, -1), ("head_dim", 96, -2),
    ("head_dim", 256, -2), ("page_size", 8, -2), ("page_size", 0, -1), ("window", -1, -1),
    ("window", 65, -2), ("group", 17, -2), ("budget_tokens", 8, -1), ("max_pages", 0, -1),
    ("max_pages", 20000, -2), ("dtype", 7, -1), ("sm_scale", -1.0, -1),
    ("sm_scale", float("inf"), -1), ("sm_scale", float("nan"), -1), ("num_phys_pages", 0, -1),
    ("flags", 8, -1), ("flags", -1, -1),
])
def test_bad_dims_are_rejected(lib, field, value, status):
    d = _dims(lib, **{field: value})
    with pytest.raises(lib.RetroError) as e:
        lib.retro_k_max(d)
    assert e.value.status == status


def test_rows_limit(lib):
    with pytest.raises(lib.RetroError) as e:
        lib.retro_k_max(_dims(lib, window=64, group=16))
    assert e.value.status == lib.RETRO_EUNSUPPORTED
    assert lib.retro_k_max(_dims(lib, window=63, group=16)) == 128


def test_k_max_and_workspace(lib):
    assert lib.retro_k_max(_dims(lib)) == 2048 // 16
    assert lib.retro_k_max(_dims(lib, budget_tokens=1 << 20, max_pages=100)) == 100
    assert lib.retro_k_max(_dims(lib, budget_tokens=1000)) == 62          # floor(B / P)
    ws = lib.retro_workspace_size(_dims(lib))
    # at least the scores and one fp32 partial output per (KV head, row)
    assert ws >= 8 * 2080 * 4 + 8 * 17 * 4 * 128 * 4
    assert ws % 256 == 0


def test_null_pointers_and_small_workspace_rejected_before_any_launch(lib):
    d = _dims(lib)
    cache = lib.KVCache(1, 1, 1, 1, 1, 1)
    sel = lib.Selection(1, 1, 1)
    oc = lib.OutputCache(1, 1)
    ws = lib.retro_workspace_size(d)
    raw = lib.load_library()
    S = C.c_int32
    # null query window
    assert raw.retro_step(C.byref(d), 0, None, 1, 1, C.byref(cache), C.byref(sel), C.byref(oc),
                          1, 1, 1, ws, None) == lib.RETRO_EINVAL
    # missing cache member
    bad = lib.KVCache(1, 1, None, 1, 1, 1)
    assert raw.retro_step(C.byref(d), 0, 1, 1, 1, C.byref(bad), C.byref(sel), C.byref(oc),
                          1, 1, 1, ws, None) == lib.RETRO_EINVAL
    # output cache required when W > 0, optional when W == 0
    assert raw.retro_merge_output_cache(C.byref(d), 0, 1, 1, None, 1, 1, None) == lib.RETRO_EINVAL
    # negative step
    assert raw.retro_append_kv(C.byref(d), -1, C.byref(cache), 1, 1, None) == lib.RETRO_EINVAL
    # workspace too small / missing
    assert raw.retro_step(C.byref(d), 0, 1, 1, 1, C.byref(cache), C.byref(sel), C.byref(oc),
                          1, 1, 1, ws - 1, None) == lib.RETRO_EWORKSPACE
    assert raw.retro_select_pages(C.byref(d), 0, 1, C.byref(cache), C.byref(sel), None, ws,
                                  None) == lib.RETRO_EWORKSPACE
    assert raw.retro_decode_attend(C.byref(d), 0, 1, C.byref(cache), C.byref(sel), None, 1, 1, ws,
                                   None) == lib.RETRO_EINVAL
    # prefill range checks
    assert raw.retro_prefill_kv(C.byref(d), C.byref(cache), 1, 0, 4, 1, 1, None) == lib.RETRO_EINVAL
    assert raw.retro_prefill_kv(C.byref(d), C.byref(cache), 0, 2080 * 16 - 2, 4, 1, 1,
                                None) == lib.RETRO_EINVAL
    assert raw.retro_k_max(None, C.byref(S())) == lib.RETRO_EINVAL


def test_project_f32_arguments_checked_on_the_host(lib):
    raw = lib.load_library()
    assert raw.retro_project_f32(None, 1, 4, 1, 4, 1, 0, None) == lib.RETRO_EINVAL
    assert raw.retro_project_f32(1, -1, 4, 1, 4, 1, 0, None) == lib.RETRO_EINVAL
    assert raw.retro_project_f32(1, 1, 0, 1, 4, 1, 0, None) == lib.RETRO_EINVAL
    assert raw.retro_project_f32(1, 0, 4, 1, 4, 1, 0, None) == lib.RETRO_OK  # no rows: nothing to do
    assert raw.retro_project_f32(1, 70000, 4, 1, 4, 1, 1, None) == lib.RETRO_EUNSUPPORTED


def test_append_tokens_arguments_checked_on_the_host(lib):
    d = _dims(lib)
    cache = lib.KVCache(1, 1, 1, 1, 1, 1)
    raw = lib.load_library()
    assert raw.retro_append_kv_tokens(C.byref(d), -1, C.byref(cache), 2, 1, 1, None) == lib.RETRO_EINVAL
    assert raw.retro_append_kv_tokens(C.byref(d), 0, C.byref(cache), -1, 1, 1, None) == lib.RETRO_EINVAL
    assert raw.retro_append_kv_tokens(C.byref(d), 0, C.byref(cache), 2, None, 1, None) == lib.RETRO_EINVAL
    bad = lib.KVCache(1, 1, None, 1, 1, 1)
    assert raw.retro_append_kv_tokens(C.byref(d), 0, C.byref(bad), 2, 1, 1, None) == lib.RETRO_EINVAL
    # no tokens: nothing to do, no launch
    assert raw.retro_append_kv_tokens(C.byref(d), 0, C.byref(cache), 0, None, None, None) == lib.RETRO_OK
