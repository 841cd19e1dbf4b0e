"""MI355X (gfx950) library for one decode step of retrospective sparse attention.

The compute path is the HIP library ``libretro_mi355x.so`` (C ABI in
``include/retro.h``); this package only binds it (``binding``) and offers a
buffer-owning helper (``layer.RetroLayer``).
"""
from .binding import (EXPORTED, RETRO_BF16, RETRO_F32, Dims, KVCache, OutputCache, RetroError,
                      Selection, load_library, retro_append_kv, retro_decode_attend,
                      retro_decode_attend_partials,
                      retro_k_max, retro_merge_output_cache, retro_prefill_kv,
                      retro_select_pages, retro_status_string, retro_step, retro_version,
                      retro_workspace_size)

__all__ = ["EXPORTED", "RETRO_BF16", "RETRO_F32", "Dims", "KVCache", "OutputCache", "RetroError",
           "Selection", "load_library", "retro_append_kv", "retro_decode_attend",
           "retro_decode_attend_partials", "retro_k_max",
           "retro_merge_output_cache", "retro_prefill_kv", "retro_select_pages",
           "retro_status_string", "retro_step", "retro_version", "retro_workspace_size"]
