"""MI355X-native Thinker decoder layer (prefill, decode, mixed steps).

The compute path is libtri.so (hand-written HIP kernels for gfx950 behind the
C ABI in include/tri.h); this package is its thin ctypes binding.
"""
from ._lib import (DeviceBatch, LayerConfig, PagedCache, Profile, TriError, Work, kv_struct,
                   kvcache_append,
                   layer_decode, layer_work, phase_intensity, profile_enable, profile_read,
                   work_dict, work_sum,
                   layer_prefill, lib, linear, linear_workspace_size, make_config, moe_route,
                   status_string, workspace_layout, workspace_size)

__all__ = ["DeviceBatch", "LayerConfig", "PagedCache", "Profile", "TriError", "Work", "kv_struct",
           "kvcache_append",
           "layer_decode", "layer_work", "phase_intensity", "work_dict", "work_sum",
           "layer_prefill", "lib", "linear", "linear_workspace_size", "profile_enable", "profile_read",
           "make_config", "moe_route", "status_string",
           "workspace_layout", "workspace_size"]
