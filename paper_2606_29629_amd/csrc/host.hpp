// Host-side definitions shared by the C-ABI sources: config validation and
// the stage list that both the per-stage timers and the work model index.
#pragma once
#include "../../include/tri.h"

namespace tri {

enum Stage {
  ST_PROLOGUE, ST_QKV, ST_ATTN_PREFILL, ST_ATTN_DECODE, ST_ATTN_COMBINE, ST_OPROJ,
  ST_NORM2, ST_GATEUP, ST_DOWN, ST_ROUTER, ST_MOE_PERMUTE, ST_MOE_GATEUP, ST_MOE_DOWN,
  ST_MOE_COMBINE, ST_APPEND, ST_COUNT
};
static_assert(ST_COUNT <= TRI_MAX_STAGES, "too many stages");

inline constexpr const char* kStageName[ST_COUNT] = {
    "prologue", "qkv_rope", "attn_prefill", "attn_decode", "attn_combine",
    "o_proj", "rmsnorm_mlp", "gate_up", "down", "moe_router", "moe_permute", "moe_gate_up",
    "moe_down", "moe_combine", "kv_append"};

// Validates a layer config (TRI_OK, or the status the entry points return).
tri_status check_config(const tri_layer_config* c);

// The layer entry points' common body (tri_layer_prefill when decode is
// false, tri_layer_decode when true) on a workspace of ws_bytes; with timed =
// false no profiling event is created or recorded.
tri_status layer_call(bool decode, bool timed, const tri_layer_config* cfg,
                      const tri_layer_weights* w, const tri_kv_cache* cache, const tri_batch* b,
                      const void* x_in, void* x_out, int32_t* route_idx, float* route_w, void* ws,
                      size_t ws_bytes, void* stream);

}  // namespace tri
