// libtri C ABI: host-side validation, workspace layout and the launch
// sequences of the decoder layer.  No kernel is launched unless every check
// passes; no device memory is allocated.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "../../include/tri.h"
#include "host.hpp"
#include "kernels.hpp"

using namespace tri;

namespace {
bool is_moe(const tri_layer_config* c) { return (c->flags & TRI_F_MOE) != 0; }
bool is_f32(const tri_layer_config* c) { return c->dtype == TRI_F32; }

// Rotary frequency sections: frequency i < s0 reads position plane 0, i < s01
// plane 1, the rest plane 2 (one plane, s0 = s01 = D/2, without TRI_F_MROPE).
RopeSections rope_sections(const tri_layer_config* c) {
  const int half = c->head_dim / 2;
  if (!(c->flags & TRI_F_MROPE)) return {half, half};
  return {c->mrope_section[0], c->mrope_section[0] + c->mrope_section[1]};
}
}  // namespace

tri_status tri::check_config(const tri_layer_config* c) {
  if (!c) return TRI_ERR_NULL;
  if (c->dtype != TRI_BF16 && c->dtype != TRI_F32) return TRI_ERR_UNSUPPORTED;
  if (c->flags & ~TRI_F_ALL) return TRI_ERR_UNSUPPORTED;
  if (c->hidden <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0)
    return TRI_ERR_SHAPE;
  if (c->head_dim != 64 && c->head_dim != 128) return TRI_ERR_UNSUPPORTED;
  if (c->hidden % 64 != 0 || c->hidden > 8192) return TRI_ERR_UNSUPPORTED;
  if (c->n_q_heads % c->n_kv_heads != 0) return TRI_ERR_SHAPE;
  if (c->n_q_heads / c->n_kv_heads > 32) return TRI_ERR_UNSUPPORTED;
  if ((int64_t)c->n_q_heads * c->head_dim % 64 != 0) return TRI_ERR_UNSUPPORTED;
  if (!(c->rms_eps >= 0.f) || !(c->rope_base > 0.f)) return TRI_ERR_RANGE;
  if (c->flags & TRI_F_MROPE) {
    const int32_t* m = c->mrope_section;
    if (m[0] < 0 || m[1] < 0 || m[2] < 0 || (int64_t)m[0] + m[1] + m[2] != c->head_dim / 2)
      return TRI_ERR_SHAPE;
  }
  if (is_moe(c)) {
    if (c->n_experts < 1 || c->n_experts > 256) return TRI_ERR_UNSUPPORTED;
    if (c->top_k < 1 || c->top_k > c->n_experts || c->top_k > 16) return TRI_ERR_SHAPE;
    if (c->expert_ffn_dim <= 0 || c->expert_ffn_dim % 64 != 0) return TRI_ERR_UNSUPPORTED;
  } else {
    if (c->ffn_dim <= 0 || c->ffn_dim % 64 != 0) return TRI_ERR_UNSUPPORTED;
  }
  return TRI_OK;
}

namespace {

constexpr size_t kAlign = 256;
inline size_t up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Projections with at most this many rows take the weight-streaming path.
constexpr int kSkinnyMaxRows = 128;

tri_status check_batch_scalars(const tri_batch* b) {
  if (!b) return TRI_ERR_NULL;
  if (b->n_seqs < 0 || b->n_tokens < 0 || b->max_q_len < 0 || b->max_ctx_len < 0)
    return TRI_ERR_SHAPE;
  if (b->n_tokens > 0 && b->n_seqs == 0) return TRI_ERR_SHAPE;
  if (b->n_tokens > 0 && b->max_q_len == 0) return TRI_ERR_SHAPE;
  if ((int64_t)b->max_q_len > b->n_tokens) return TRI_ERR_SHAPE;
  if ((int64_t)b->n_seqs > 0 && (int64_t)b->max_q_len * b->n_seqs < b->n_tokens) return TRI_ERR_SHAPE;
  return TRI_OK;
}

struct Layout {
  size_t tok_slot, tok_row, rope, h, q, attn, x1, h2, act, part;
  // MoE (n_pairs = T * top_k)
  size_t route_idx, route_w, rank, counts, perm, inv, seg, tile_off, y, logits;
  // fp32 storage: bf16 operand planes of the activations (one GEMM at a time)
  // and of the weights (q/k/v, O, gate/up, down)
  size_t a3, w_qkv3, w_o3, w_gu3, w_d3;
  size_t total;
};

// Bytes of the flash kernel's split partials, rounded up to the alignment
// (none when no sequence has more than one token: no flash launch).
size_t flash_part_bytes(const tri_layer_config* c, const tri_batch* b) {
  if (b->max_q_len <= 1) return 0;
  return up(attn_prefill_partial_bytes(b->n_seqs, b->n_tokens, b->max_q_len, b->max_ctx_len,
                                       c->n_q_heads, c->head_dim));
}

size_t part_bytes(const tri_layer_config* c, const tri_batch* b) {
  const int T = b->n_tokens, H = c->hidden, D = c->head_dim;
  const int Nqkv = (c->n_q_heads + 2 * c->n_kv_heads) * D;
  // A chunk's flash attention and the single-token sequences' split-KV
  // attention may run at the same time (on two streams), so their partials
  // sit side by side: the flash partials first, then the decode partials.
  size_t p = flash_part_bytes(c, b) +
             attn_decode_partial_bytes(b->n_seqs, c->n_q_heads, D, b->max_ctx_len + 1);
  if (T > 0) {
    // Skinny-path partials.  64-row and 128-row batches split K differently,
    // so a batch reserves them for the largest batch of each kind up to its
    // own size: the size never shrinks as n_tokens grows.
    auto mx = [](size_t a, size_t b2) { return a > b2 ? a : b2; };
    auto skinny = [&](int Ts) {
      size_t g = skinny_partial_bytes(Ts, Nqkv, H, EPI_QKV);
      g = mx(g, skinny_partial_bytes(Ts, H, c->n_q_heads * D, EPI_RESID));
      if (!is_moe(c)) {
        g = mx(g, skinny_partial_bytes(Ts, 2 * c->ffn_dim, H, EPI_SWIGLU));
        g = mx(g, skinny_partial_bytes(Ts, H, c->ffn_dim, EPI_RESID));
      }
      return g;
    };
    p = mx(p, mx(skinny(T < 64 ? T : 64), skinny(T <= kSkinnyMaxRows ? T : kSkinnyMaxRows)));
    // Large-M GEMMs: fp32 partials of their tail tiles (a constant bound, so
    // the size stays non-decreasing in n_tokens).
    if (T > kSkinnyMaxRows) p = mx(p, gemm_tail_bytes());
  }
  return p;
}

// Cache shape checks shared by the layer and the append: logical sizes, and
// for a paged cache the block table, block size and pool.
tri_status check_cache(const tri_kv_cache* c) {
  if (!c) return TRI_ERR_NULL;
  if (!c->k || !c->v) return TRI_ERR_NULL;
  if (c->n_slots <= 0 || c->max_seq <= 0) return TRI_ERR_SHAPE;
  if (c->block_table) {
    if (c->block_size <= 0 || c->n_blocks <= 0) return TRI_ERR_SHAPE;
    if (c->block_size % 64 != 0) return TRI_ERR_UNSUPPORTED;
    if (c->max_seq % c->block_size != 0) return TRI_ERR_SHAPE;
    if (((uintptr_t)c->block_table & 3u) != 0) return TRI_ERR_ALIGN;
  }
  return TRI_OK;
}

KvDev kv_dev(const tri_kv_cache* c) {
  KvDev kv{};
  kv.n_slots = c->n_slots;
  kv.max_seq = c->max_seq;
  kv.table = c->block_table;
  kv.block_size = c->block_table ? c->block_size : 0;
  kv.n_blocks = c->block_table ? c->n_blocks : 0;
  return kv;
}

// fp32 storage: activations in fp32, every projection on bf16 operand planes
// (split3: activations [hi | lo | hi], weights [hi | hi | lo], a 3K
// contraction), attention through the flash kernel for every sequence (no
// split-KV partials), the large GEMMs' tail partials.
Layout layout_f32(const tri_layer_config* c, const tri_batch* b) {
  const size_t T = (size_t)b->n_tokens, H = c->hidden, D = c->head_dim;
  const size_t Hq = c->n_q_heads, Hkv = c->n_kv_heads;
  const bool moe = is_moe(c);
  const size_t P = moe ? T * c->top_k : 0, E = moe ? c->n_experts : 0;
  const size_t F = moe ? (size_t)c->expert_ffn_dim : (size_t)c->ffn_dim;
  const size_t act_rows = moe ? P : T;
  const size_t Nqkv = (Hq + 2 * Hkv) * D;
  const size_t f = 4, pl = 3 * 2;  // fp32 element; three bf16 planes per element
  Layout l{};
  size_t o = 0;
  l.tok_slot = o; o += up(T * 4);
  l.tok_row = o;  o += up(T * 4);
  l.rope = o;     o += up(T * (D / 2) * 8);
  l.h = o;        o += up(T * H * f);
  l.q = o;        o += up(T * Hq * D * f);
  l.attn = o;     o += up(T * Hq * D * f);
  l.x1 = o;       o += up(T * H * f);
  l.h2 = o;       o += up(T * H * f);
  l.act = o;      o += up(act_rows * F * f);
  l.part = o;     o += up(T > 0 ? gemm_tail_bytes() : 0);
  l.route_idx = o; o += up(P * 4);
  l.route_w = o;  o += up(P * 4);
  l.rank = o;     o += up(P * 4);
  l.counts = o;   o += up(E * 4);
  l.perm = o;     o += up(P * 4);
  l.inv = o;      o += up(P * 4);
  l.seg = o;      o += up((E + 1) * 4);
  l.tile_off = o; o += up((E + 1) * 4);
  l.y = o;        o += up(P * H * 4);
  const size_t a_cols = std::max(std::max(H, Hq * D), F);  // widest activation operand
  l.a3 = o;       o += up(std::max(T, act_rows) * a_cols * pl);
  l.w_qkv3 = o;   o += up(Nqkv * H * pl);
  l.w_o3 = o;     o += up(H * Hq * D * pl);
  const size_t experts = moe ? E : 1;
  l.w_gu3 = o;    o += up(experts * 2 * F * H * pl);
  l.w_d3 = o;     o += up(experts * H * F * pl);
  l.total = o;
  return l;
}

Layout layout_of(const tri_layer_config* c, const tri_batch* b) {
  if (is_f32(c)) return layout_f32(c, b);
  const size_t T = (size_t)b->n_tokens, H = c->hidden, D = c->head_dim;
  const bool moe = is_moe(c);
  const size_t P = moe ? T * c->top_k : 0, E = moe ? c->n_experts : 0;
  const size_t act_cols = moe ? (size_t)c->expert_ffn_dim : (size_t)c->ffn_dim;
  const size_t act_rows = moe ? P : T;
  Layout l{};
  size_t o = 0;
  l.tok_slot = o; o += up(T * 4);
  l.tok_row = o;  o += up(T * 4);
  l.rope = o;     o += up(T * (D / 2) * 8);
  l.h = o;        o += up(T * H * 2);
  l.q = o;        o += up(T * c->n_q_heads * D * 2);
  l.attn = o;     o += up(T * c->n_q_heads * D * 2);
  l.x1 = o;       o += up(T * H * 2);
  l.h2 = o;       o += up(T * H * 2);
  l.act = o;      o += up(act_rows * act_cols * 2);
  l.part = o;     o += up(part_bytes(c, b));
  l.route_idx = o; o += up(P * 4);
  l.route_w = o;  o += up(P * 4);
  l.rank = o;     o += up(P * 4);
  l.counts = o;   o += up(E * 4);
  l.perm = o;     o += up(P * 4);
  l.inv = o;      o += up(P * 4);
  l.seg = o;      o += up((E + 1) * 4);
  l.tile_off = o; o += up((E + 1) * 4);
  l.y = o;        o += up(P * H * 4);
  // Router logit planes [S][T][E]: S * T <= max(T, 51200 / ceil(E / 64)) for
  // every split count the GEMM picks (S > 1 only while S * tiles < 800), a
  // bound that never decreases with T.
  const size_t rows = moe ? std::max(T, (size_t)51200 / ((E + 63) / 64)) : 0;
  l.logits = o;   o += up(rows * E * 4);
  l.total = o;
  return l;
}

// ------------------------------------------------------------ profiling --
struct Profiler {
  std::mutex mu;
  bool on = false;
  struct Rec { int stage; hipEvent_t a, b; };
  std::vector<Rec> pending;
  std::vector<hipEvent_t> pool;
  int launches[ST_COUNT] = {};
  double ms[ST_COUNT] = {};
  hipEvent_t get() {
    if (!pool.empty()) { hipEvent_t e = pool.back(); pool.pop_back(); return e; }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
Profiler& prof() { static Profiler p; return p; }

// Records an event pair around one stage when profiling is on.
struct StageTimer {
  int stage;
  hipStream_t s;
  hipEvent_t a = nullptr, b = nullptr;
  StageTimer(int st, hipStream_t str, bool timed = true) : stage(st), s(str) {
    Profiler& p = prof();
    if (!timed || !p.on) return;
    std::lock_guard<std::mutex> g(p.mu);
    a = p.get();
    b = p.get();
    if (a && b) hipEventRecord(a, s);
  }
  ~StageTimer() {
    if (!a || !b) return;
    Profiler& p = prof();
    hipEventRecord(b, s);
    std::lock_guard<std::mutex> g(p.mu);
    p.pending.push_back({stage, a, b});
  }
};

template <typename T>
T* at(void* ws, size_t off) { return (T*)((char*)ws + off); }

// A second stream per device, on which a mixed batch's split-KV attention
// (the single-token sequences) runs beside the flash attention of its
// multi-token sequences: both read the projected q and the cache, and they
// write disjoint output rows and disjoint partials.  Created on first use
// (default priority, non-blocking); the fork and join events are recorded and
// waited on under the device's lock, so concurrent callers cannot pair one
// caller's record with another's wait.
struct SideStream {
  std::mutex mu;
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  bool failed = false;  // creation failed once (e.g. under graph capture): run serially
};
constexpr int kMaxSideDevices = 64;
// The side stream of the current device, or nullptr (run on the caller's
// stream) when the caller's stream belongs to another device.
SideStream* side_stream(hipStream_t caller) {
  static SideStream ss[kMaxSideDevices];
  int dev = -1, sdev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxSideDevices) return nullptr;
  if (caller && (hipStreamGetDevice(caller, &sdev) != hipSuccess || sdev != dev)) {
    (void)hipGetLastError();
    return nullptr;
  }
  return &ss[dev];
}
// With the device's lock held: makes sure the stream and events exist; false
// means "run on the caller's stream".  No stream is created while the
// caller's stream is being captured into a graph (creating one could
// invalidate the capture); an existing side stream joins the capture through
// the fork and join events.
bool side_ready(SideStream& x, hipStream_t caller) {
  if (x.s) return true;
  if (x.failed) return false;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(caller, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone) {
    (void)hipGetLastError();
    return false;
  }
  hipStream_t st = nullptr;
  hipEvent_t f = nullptr, j = nullptr;
  if (hipStreamCreateWithFlags(&st, hipStreamNonBlocking) == hipSuccess &&
      hipEventCreateWithFlags(&f, hipEventDisableTiming) == hipSuccess &&
      hipEventCreateWithFlags(&j, hipEventDisableTiming) == hipSuccess) {
    x.s = st;
    x.fork = f;
    x.join = j;
    return true;
  }
  if (f) (void)hipEventDestroy(f);
  if (st) (void)hipStreamDestroy(st);
  (void)hipGetLastError();  // clear the failed call's error
  x.failed = true;
  return false;
}


#define TRI_HIP(expr)                              \
  do {                                             \
    if ((expr) != hipSuccess) return TRI_ERR_HIP;  \
  } while (0)

tri_status run_linear(const void* A, int lda, const void* B, int M, int N, int K, const Epi& epi,
                      float* part, hipStream_t s) {
  if (M <= kSkinnyMaxRows) TRI_HIP(launch_skinny(A, lda, B, K, M, N, K, epi, part, s));
  else TRI_HIP(launch_gemm(A, lda, B, K, M, N, K, epi, part, s));
  return TRI_OK;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

// The fp32 storage mode's launch sequence (arguments already validated): the
// same stages on fp32 activations, cache and weights.  Every projection runs
// the prefill GEMM on bf16 operand planes (activations [hi | lo | hi] against
// weights [hi | hi | lo] over 3K: the products a_hi b_hi + a_lo b_hi + a_hi
// b_lo, fp32 accumulation), with the same fused epilogues storing fp32; every
// sequence's attention runs the flash kernel on the fp32 matrix instruction.
// Used for tight parity, not for speed: the weight planes are rebuilt on
// every call.
tri_status layer_f32(const tri_layer_config* cfg, const tri_layer_weights* w,
                     const tri_kv_cache* cache, const tri_batch* b, const void* x_in, void* x_out,
                     int32_t* route_idx, float* route_w, void* ws, const Layout& L, bool timed,
                     hipStream_t s) {
  const int T = b->n_tokens, H = cfg->hidden, D = cfg->head_dim;
  const int Hq = cfg->n_q_heads, Hkv = cfg->n_kv_heads, F = cfg->ffn_dim;
  const int Nqkv = (Hq + 2 * Hkv) * D;
  const bool moe = is_moe(cfg);
  BatchDev bd{b->cu_q, b->ctx_len, b->slot, b->pos, b->n_seqs, b->n_tokens, b->max_q_len,
              b->max_ctx_len};
  const KvDev kv = kv_dev(cache);
  int32_t* tok_slot = at<int32_t>(ws, L.tok_slot);
  int32_t* tok_row = at<int32_t>(ws, L.tok_row);
  float2* rope = at<float2>(ws, L.rope);
  float* h = at<float>(ws, L.h);
  float* q = at<float>(ws, L.q);
  float* attn = at<float>(ws, L.attn);
  float* x1 = at<float>(ws, L.x1);
  float* h2 = at<float>(ws, L.h2);
  float* act = at<float>(ws, L.act);
  float* tail = at<float>(ws, L.part);
  void* a3 = at<void>(ws, L.a3);
  auto planes = [&](const void* src, int64_t rows, int cols, int pattern, void* dst) {
    return launch_split3((const float*)src, cols, rows, cols, pattern, dst, s);
  };
  {
    StageTimer t_(ST_PROLOGUE, s, timed);
    TRI_HIP(launch_prologue(bd, kv, D, cfg->rope_base, rope_sections(cfg), tok_slot, tok_row,
                            rope, x_in, w->attn_norm, h, H, cfg->rms_eps, s, true));
  }
  Epi e{};
  e.f32 = 1;
  e.kind = EPI_QKV;
  e.bias = (cfg->flags & TRI_F_QKV_BIAS) ? w->b_qkv : nullptr;
  e.q = q;
  e.kc = cache->k;
  e.vc = cache->v;
  e.tok_slot = tok_slot;
  e.tok_row = tok_row;
  e.rope = rope;
  e.q_norm = (cfg->flags & TRI_F_QK_NORM) ? w->q_norm : nullptr;
  e.k_norm = (cfg->flags & TRI_F_QK_NORM) ? w->k_norm : nullptr;
  e.eps = cfg->rms_eps;
  e.n_q_heads = Hq;
  e.n_kv_heads = Hkv;
  e.head_dim = D;
  e.max_seq = kv.panel_rows();
  {
    StageTimer t_(ST_QKV, s, timed);
    TRI_HIP(planes(h, T, H, 0, a3));
    TRI_HIP(planes(w->w_qkv, Nqkv, H, 1, at<void>(ws, L.w_qkv3)));
    TRI_HIP(launch_gemm(a3, 3 * H, at<void>(ws, L.w_qkv3), 3 * H, T, Nqkv, 3 * H, e, tail, s));
  }
  {
    StageTimer t_(ST_ATTN_PREFILL, s, timed);
    TRI_HIP(launch_attn_prefill(q, cache->k, cache->v, attn, bd, kv, Hq, Hkv, D, 1, nullptr, s,
                                true));
  }
  e = Epi{};
  e.f32 = 1;
  e.kind = EPI_RESID;
  e.out = x1;
  e.ldo = H;
  e.resid = x_in;
  e.ldr = H;
  {
    StageTimer t_(ST_OPROJ, s, timed);
    TRI_HIP(planes(attn, T, Hq * D, 0, a3));
    TRI_HIP(planes(w->w_o, H, Hq * D, 1, at<void>(ws, L.w_o3)));
    TRI_HIP(launch_gemm(a3, 3 * Hq * D, at<void>(ws, L.w_o3), 3 * Hq * D, T, H, 3 * Hq * D, e,
                        tail, s));
  }
  {
    StageTimer t_(ST_NORM2, s, timed);
    TRI_HIP(launch_rmsnorm(x1, w->mlp_norm, h2, nullptr, T, H, cfg->rms_eps, s, true));
  }
  void* wgu3 = at<void>(ws, L.w_gu3);
  void* wd3 = at<void>(ws, L.w_d3);
  if (!moe) {
    e = Epi{};
    e.f32 = 1;
    e.kind = EPI_SWIGLU;
    e.out = act;
    e.ldo = F;
    e.ffn = F;
    {
      StageTimer t_(ST_GATEUP, s, timed);
      TRI_HIP(planes(h2, T, H, 0, a3));
      TRI_HIP(planes(w->w_gate_up, 2 * F, H, 1, wgu3));
      TRI_HIP(launch_gemm(a3, 3 * H, wgu3, 3 * H, T, 2 * F, 3 * H, e, tail, s));
    }
    e = Epi{};
    e.f32 = 1;
    e.kind = EPI_RESID;
    e.out = x_out;
    e.ldo = H;
    e.resid = x1;
    e.ldr = H;
    StageTimer t_(ST_DOWN, s, timed);
    TRI_HIP(planes(act, T, F, 0, a3));
    TRI_HIP(planes(w->w_down, H, F, 1, wd3));
    TRI_HIP(launch_gemm(a3, 3 * F, wd3, 3 * F, T, H, 3 * F, e, tail, s));
    return TRI_OK;
  }
  const int E = cfg->n_experts, k = cfg->top_k, Fe = cfg->expert_ffn_dim;
  const int P = T * k;
  int32_t* idx = route_idx ? route_idx : at<int32_t>(ws, L.route_idx);
  float* rw = route_w ? route_w : at<float>(ws, L.route_w);
  int32_t* perm = at<int32_t>(ws, L.perm);
  int32_t* inv = at<int32_t>(ws, L.inv);
  int32_t* seg = at<int32_t>(ws, L.seg);
  int32_t* tile_off = at<int32_t>(ws, L.tile_off);
  float* y = at<float>(ws, L.y);
  {
    StageTimer t_(ST_ROUTER, s, timed);
    TRI_HIP(launch_moe_route_f32(h2, w->w_router, T, H, E, k,
                                 (cfg->flags & TRI_F_MOE_RENORM) ? 1 : 0, idx, rw, s, true));
  }
  {
    StageTimer t_(ST_MOE_PERMUTE, s, timed);
    TRI_HIP(launch_moe_permute(idx, P, E, moe_tile_rows(P, E), at<int32_t>(ws, L.rank),
                               at<int32_t>(ws, L.counts), perm, inv, seg, tile_off, s));
  }
  e = Epi{};
  e.f32 = 1;
  e.kind = EPI_SWIGLU;
  e.out = act;
  e.ldo = Fe;
  e.ffn = Fe;
  {
    StageTimer t_(ST_MOE_GATEUP, s, timed);
    TRI_HIP(planes(h2, T, H, 0, a3));
    TRI_HIP(planes(w->w_gate_up, (int64_t)E * 2 * Fe, H, 1, wgu3));
    TRI_HIP(launch_gemm_grouped(a3, 3 * H, T, perm, k, wgu3, (int64_t)2 * Fe * 3 * H, 2 * Fe,
                                3 * H, seg, tile_off, E, P, e, s));
  }
  e = Epi{};
  e.f32 = 1;
  e.kind = EPI_STORE_F32;
  e.out = y;
  e.ldo = H;
  {
    StageTimer t_(ST_MOE_DOWN, s, timed);
    TRI_HIP(planes(act, P, Fe, 0, a3));
    TRI_HIP(planes(w->w_down, (int64_t)E * H, Fe, 1, wd3));
    TRI_HIP(launch_gemm_grouped(a3, 3 * Fe, P, nullptr, k, wd3, (int64_t)H * 3 * Fe, H, 3 * Fe,
                                seg, tile_off, E, P, e, s));
  }
  {
    StageTimer t_(ST_MOE_COMBINE, s, timed);
    TRI_HIP(launch_moe_combine(x1, y, inv, rw, T, H, k, x_out, s, true));
  }
  return TRI_OK;
}

}  // namespace

// One layer call on the caller's workspace; `timed` = false keeps the call
// free of profiling events (no event is created or recorded).
tri_status tri::layer_call(bool decode, bool timed, const tri_layer_config* cfg,
                           const tri_layer_weights* w, const tri_kv_cache* cache,
                           const tri_batch* b, const void* x_in, void* x_out, int32_t* route_idx,
                           float* route_w, void* ws, size_t ws_bytes, void* stream) {
  tri_status st = check_config(cfg);
  if (st != TRI_OK) return st;
  if (!w || !cache) return TRI_ERR_NULL;
  if ((st = check_batch_scalars(b)) != TRI_OK) return st;
  if (decode && (b->n_tokens != b->n_seqs || b->max_q_len > 1)) return TRI_ERR_SHAPE;
  if (b->n_tokens == 0) return TRI_OK;
  if (!x_in || !x_out || !ws || !b->cu_q || !b->ctx_len || !b->slot || !b->pos) return TRI_ERR_NULL;
  if ((st = check_cache(cache)) != TRI_OK) return st;
  if (!w->attn_norm || !w->w_qkv || !w->w_o || !w->mlp_norm || !w->w_gate_up || !w->w_down)
    return TRI_ERR_NULL;
  const bool moe = is_moe(cfg);
  if (moe && !w->w_router) return TRI_ERR_NULL;
  const bool bias = (cfg->flags & TRI_F_QKV_BIAS) != 0;
  if (bias && !w->b_qkv) return TRI_ERR_NULL;
  const bool qk_norm = (cfg->flags & TRI_F_QK_NORM) != 0;
  if (qk_norm && (!w->q_norm || !w->k_norm)) return TRI_ERR_NULL;
  if (b->max_ctx_len >= cache->max_seq || b->max_q_len > cache->max_seq) return TRI_ERR_RANGE;
  if (decode && (int64_t)b->max_ctx_len + 1 > cache->max_seq) return TRI_ERR_RANGE;
  const void* ptrs[] = {x_in, x_out, ws, cache->k, cache->v, w->attn_norm, w->w_qkv, w->w_o,
                        w->mlp_norm, w->w_gate_up, w->w_down};
  for (const void* p : ptrs)
    if (!aligned16(p)) return TRI_ERR_ALIGN;
  if (bias && !aligned16(w->b_qkv)) return TRI_ERR_ALIGN;
  if (qk_norm && (!aligned16(w->q_norm) || !aligned16(w->k_norm))) return TRI_ERR_ALIGN;
  if (moe && !aligned16(w->w_router)) return TRI_ERR_ALIGN;
  if (((uintptr_t)ws & (kAlign - 1)) != 0) return TRI_ERR_ALIGN;
  const Layout L = layout_of(cfg, b);
  if (ws_bytes < L.total) return TRI_ERR_WORKSPACE;
  const size_t act_bytes = (size_t)b->n_tokens * cfg->hidden * (is_f32(cfg) ? 4 : 2);
  if (overlaps(x_in, act_bytes, x_out, act_bytes)) return TRI_ERR_ALIAS;
  if (overlaps(ws, L.total, x_in, act_bytes) || overlaps(ws, L.total, x_out, act_bytes))
    return TRI_ERR_ALIAS;
  if (is_f32(cfg))
    return layer_f32(cfg, w, cache, b, x_in, x_out, route_idx, route_w, ws, L, timed,
                     (hipStream_t)stream);

  hipStream_t s = (hipStream_t)stream;
  const int T = b->n_tokens, H = cfg->hidden, D = cfg->head_dim;
  const int Hq = cfg->n_q_heads, Hkv = cfg->n_kv_heads, F = cfg->ffn_dim;
  const int Nqkv = (Hq + 2 * Hkv) * D;
  BatchDev bd{b->cu_q, b->ctx_len, b->slot, b->pos, b->n_seqs, b->n_tokens, b->max_q_len,
              b->max_ctx_len};
  const KvDev kv = kv_dev(cache);
  int32_t* tok_slot = at<int32_t>(ws, L.tok_slot);
  int32_t* tok_row = at<int32_t>(ws, L.tok_row);
  float2* rope = at<float2>(ws, L.rope);
  void* h = at<void>(ws, L.h);
  void* q = at<void>(ws, L.q);
  void* attn = at<void>(ws, L.attn);
  void* x1 = at<void>(ws, L.x1);
  void* h2 = at<void>(ws, L.h2);
  void* act = at<void>(ws, L.act);
  float* part = at<float>(ws, L.part);

  {
    // token map + rotary table + pre-attention RMSNorm
    StageTimer t_(ST_PROLOGUE, s, timed);
    TRI_HIP(launch_prologue(bd, kv, D, cfg->rope_base, rope_sections(cfg), tok_slot, tok_row,
                            rope, x_in, w->attn_norm, h, H, cfg->rms_eps, s));
  }
  Epi e{};
  e.kind = EPI_QKV;
  e.bias = bias ? w->b_qkv : nullptr;
  e.q = q;
  e.kc = cache->k;
  e.vc = cache->v;
  e.tok_slot = tok_slot;
  e.tok_row = tok_row;
  e.rope = rope;
  e.q_norm = qk_norm ? w->q_norm : nullptr;
  e.k_norm = qk_norm ? w->k_norm : nullptr;
  e.eps = cfg->rms_eps;
  e.n_q_heads = Hq;
  e.n_kv_heads = Hkv;
  e.head_dim = D;
  e.max_seq = kv.panel_rows();
  {
    StageTimer t_(ST_QKV, s, timed);
    if ((st = run_linear(h, H, w->w_qkv, T, Nqkv, H, e, part, s)) != TRI_OK) return st;
  }
  // Flash attention serves the multi-token sequences, split-KV attention the
  // single-token ones (a batch in which every sequence has max_q_len > 1
  // tokens has none).  When a batch has both, the split-KV kernels run on the
  // side stream, overlapping the compute-bound flash kernel with the
  // memory-bound decode attention.
  const bool flash = !decode && b->max_q_len > 1;
  const bool splitkv =
      decode || b->max_q_len == 1 || (int64_t)b->n_seqs * b->max_q_len != b->n_tokens;
  float* part_dec = (float*)((char*)part + flash_part_bytes(cfg, b));
  hipStream_t sd = s;  // stream of the split-KV attention
  SideStream* side = (flash && splitkv) ? side_stream(s) : nullptr;
  std::unique_lock<std::mutex> side_lock;
  if (side) {
    side_lock = std::unique_lock<std::mutex>(side->mu);
    if (side_ready(*side, s)) {
      TRI_HIP(hipEventRecord(side->fork, s));
      TRI_HIP(hipStreamWaitEvent(side->s, side->fork, 0));
      sd = side->s;
    }
  }
  if (splitkv) {
    {
      StageTimer t_(ST_ATTN_DECODE, sd, timed);
      TRI_HIP(launch_attn_decode_split(q, cache->k, cache->v, part_dec, bd, kv, Hq, Hkv, D, sd));
    }
    StageTimer t_(ST_ATTN_COMBINE, sd, timed);
    TRI_HIP(launch_attn_decode_combine(part_dec, attn, bd, kv, Hq, Hkv, D, sd));
  }
  if (flash) {
    StageTimer t_(ST_ATTN_PREFILL, s, timed);
    TRI_HIP(launch_attn_prefill(q, cache->k, cache->v, attn, bd, kv, Hq, Hkv, D, 0, part, s));
  }
  if (sd != s) {
    TRI_HIP(hipEventRecord(side->join, sd));
    TRI_HIP(hipStreamWaitEvent(s, side->join, 0));
  }
  if (side_lock.owns_lock()) side_lock.unlock();
  e = Epi{};
  e.kind = EPI_RESID;
  e.out = x1;
  e.ldo = H;
  e.resid = x_in;
  e.ldr = H;
  if (skinny_resid_norm_fused(T, H, Hq * D)) {
    // short batch: the O projection's split-K reduction also adds the
    // residual and applies the pre-MLP RMSNorm (no separate norm launch)
    StageTimer t_(ST_OPROJ, s, timed);
    TRI_HIP(launch_skinny_resid_norm(attn, Hq * D, w->w_o, Hq * D, T, H, Hq * D, x_in, H, x1, H,
                                     w->mlp_norm, h2, cfg->rms_eps, part, s));
  } else {
    {
      StageTimer t_(ST_OPROJ, s, timed);
      if ((st = run_linear(attn, Hq * D, w->w_o, T, H, Hq * D, e, part, s)) != TRI_OK) return st;
    }
    StageTimer t_(ST_NORM2, s, timed);
    TRI_HIP(launch_rmsnorm(x1, w->mlp_norm, h2, nullptr, T, H, cfg->rms_eps, s));
  }

  if (!moe) {
    e = Epi{};
    e.kind = EPI_SWIGLU;
    e.out = act;
    e.ldo = F;
    e.ffn = F;
    {
      StageTimer t_(ST_GATEUP, s, timed);
      if ((st = run_linear(h2, H, w->w_gate_up, T, 2 * F, H, e, part, s)) != TRI_OK) return st;
    }
    e = Epi{};
    e.kind = EPI_RESID;
    e.out = x_out;
    e.ldo = H;
    e.resid = x1;
    e.ldr = H;
    {
      StageTimer t_(ST_DOWN, s, timed);
      if ((st = run_linear(act, F, w->w_down, T, H, F, e, part, s)) != TRI_OK) return st;
    }
    return TRI_OK;
  }

  // ---- mixture of experts
  const int E = cfg->n_experts, k = cfg->top_k, Fe = cfg->expert_ffn_dim;
  const int P = T * k;
  int32_t* idx = route_idx ? route_idx : at<int32_t>(ws, L.route_idx);
  float* rw = route_w ? route_w : at<float>(ws, L.route_w);
  int32_t* perm = at<int32_t>(ws, L.perm);
  int32_t* inv = at<int32_t>(ws, L.inv);
  int32_t* seg = at<int32_t>(ws, L.seg);
  int32_t* tile_off = at<int32_t>(ws, L.tile_off);
  float* y = at<float>(ws, L.y);
  {
    StageTimer t_(ST_ROUTER, s, timed);
    TRI_HIP(launch_moe_route_bf16(h2, w->w_router, T, H, E, k,
                                  (cfg->flags & TRI_F_MOE_RENORM) ? 1 : 0,
                                  at<float>(ws, L.logits), idx, rw, s));
  }
  {
    StageTimer t_(ST_MOE_PERMUTE, s, timed);
    TRI_HIP(launch_moe_permute(idx, P, E, moe_tile_rows(P, E), at<int32_t>(ws, L.rank),
                               at<int32_t>(ws, L.counts), perm, inv, seg, tile_off, s));
  }
  e = Epi{};
  e.kind = EPI_SWIGLU;
  e.out = act;
  e.ldo = Fe;
  e.ffn = Fe;
  {
    StageTimer t_(ST_MOE_GATEUP, s, timed);
    TRI_HIP(launch_gemm_grouped(h2, H, T, perm, k, w->w_gate_up, (int64_t)2 * Fe * H, 2 * Fe, H,
                                seg, tile_off, E, P, e, s));
  }
  e = Epi{};
  e.kind = EPI_STORE_F32;
  e.out = y;
  e.ldo = H;
  {
    StageTimer t_(ST_MOE_DOWN, s, timed);
    TRI_HIP(launch_gemm_grouped(act, Fe, P, nullptr, k, w->w_down, (int64_t)H * Fe, H, Fe, seg,
                                tile_off, E, P, e, s));
  }
  {
    StageTimer t_(ST_MOE_COMBINE, s, timed);
    TRI_HIP(launch_moe_combine(x1, y, inv, rw, T, H, k, x_out, s));
  }
  return TRI_OK;
}



extern "C" {

tri_status tri_workspace_size(const tri_layer_config* cfg, const tri_batch* batch, size_t* bytes) {
  if (!bytes) return TRI_ERR_NULL;
  tri_status st = check_config(cfg);
  if (st != TRI_OK) return st;
  if ((st = check_batch_scalars(batch)) != TRI_OK) return st;
  *bytes = layout_of(cfg, batch).total;
  return TRI_OK;
}

tri_status tri_workspace_layout(const tri_layer_config* cfg, const tri_batch* batch,
                                tri_workspace_map* map) {
  if (!map) return TRI_ERR_NULL;
  tri_status st = check_config(cfg);
  if (st != TRI_OK) return st;
  if ((st = check_batch_scalars(batch)) != TRI_OK) return st;
  const Layout l = layout_of(cfg, batch);
  map->h = l.h;
  map->q = l.q;
  map->attn = l.attn;
  map->x1 = l.x1;
  map->h2 = l.h2;
  map->act = l.act;
  map->perm = l.perm;
  map->y = l.y;
  map->total = l.total;
  return TRI_OK;
}

tri_status tri_layer_prefill(const tri_layer_config* cfg, const tri_layer_weights* w,
                             const tri_kv_cache* cache, const tri_batch* batch, const void* x_in,
                             void* x_out, int32_t* route_idx, float* route_w, void* workspace,
                             size_t workspace_bytes, void* stream) {
  return layer_call(false, true, cfg, w, cache, batch, x_in, x_out, route_idx, route_w,
                    workspace, workspace_bytes, stream);
}

tri_status tri_layer_decode(const tri_layer_config* cfg, const tri_layer_weights* w,
                            const tri_kv_cache* cache, const tri_batch* batch, const void* x_in,
                            void* x_out, int32_t* route_idx, float* route_w, void* workspace,
                            size_t workspace_bytes, void* stream) {
  return layer_call(true, true, cfg, w, cache, batch, x_in, x_out, route_idx, route_w,
                    workspace, workspace_bytes, stream);
}

tri_status tri_kvcache_append(const tri_layer_config* cfg, const tri_kv_cache* cache,
                              const tri_batch* b, const void* k_new, const void* v_new,
                              void* stream) {
  if (!cfg) return TRI_ERR_NULL;
  if (cfg->head_dim != 64 && cfg->head_dim != 128) return TRI_ERR_UNSUPPORTED;
  if (cfg->n_kv_heads <= 0) return TRI_ERR_SHAPE;
  if (cfg->dtype != TRI_BF16 && cfg->dtype != TRI_F32) return TRI_ERR_UNSUPPORTED;
  if (!cache) return TRI_ERR_NULL;
  tri_status st = check_batch_scalars(b);
  if (st != TRI_OK) return st;
  if (b->n_tokens == 0) return TRI_OK;
  if (!k_new || !v_new || !b->cu_q || !b->ctx_len || !b->slot) return TRI_ERR_NULL;
  if ((st = check_cache(cache)) != TRI_OK) return st;
  if (b->max_ctx_len >= cache->max_seq || b->max_q_len > cache->max_seq) return TRI_ERR_RANGE;
  const void* ptrs[] = {k_new, v_new, cache->k, cache->v};
  for (const void* p : ptrs)
    if (!aligned16(p)) return TRI_ERR_ALIGN;
  BatchDev bd{b->cu_q, b->ctx_len, b->slot, b->pos, b->n_seqs, b->n_tokens, b->max_q_len,
              b->max_ctx_len};
  StageTimer t_(ST_APPEND, (hipStream_t)stream);
  TRI_HIP(launch_kv_append_direct(bd, kv_dev(cache), cfg->n_kv_heads,
                                  cfg->head_dim, k_new, v_new, cache->k, cache->v,
                                  (hipStream_t)stream, is_f32(cfg)));
  return TRI_OK;
}

tri_status tri_linear_workspace_size(int32_t M, int32_t N, int32_t K, size_t* bytes) {
  if (!bytes) return TRI_ERR_NULL;
  if (M <= 0 || N <= 0 || K <= 0 || K % 64 != 0 || N % 4 != 0) return TRI_ERR_SHAPE;
  *bytes = M <= kSkinnyMaxRows ? skinny_partial_bytes(M, N, K, EPI_STORE) : gemm_tail_bytes();
  return TRI_OK;
}

tri_status tri_linear(const void* A, const void* B, void* C, int32_t M, int32_t N, int32_t K,
                      void* workspace, size_t workspace_bytes, void* stream) {
  size_t need = 0;
  tri_status st = tri_linear_workspace_size(M, N, K, &need);
  if (st != TRI_OK) return st;
  if (!A || !B || !C) return TRI_ERR_NULL;
  if ((int64_t)M * K * 2 >= (int64_t)1 << 31 || (int64_t)N * K * 2 >= (int64_t)1 << 31)
    return TRI_ERR_RANGE;  // 32-bit buffer ranges of the operand loads
  if (!aligned16(A) || !aligned16(B) || !aligned16(C)) return TRI_ERR_ALIGN;
  if (need > 0 && (!workspace || workspace_bytes < need)) return TRI_ERR_WORKSPACE;
  if (need > 0 && ((uintptr_t)workspace % kAlign) != 0) return TRI_ERR_ALIGN;
  if (overlaps(C, (size_t)M * N * 2, A, (size_t)M * K * 2) ||
      overlaps(C, (size_t)M * N * 2, B, (size_t)N * K * 2))
    return TRI_ERR_ALIAS;
  Epi e{};
  e.kind = EPI_STORE;
  e.out = C;
  e.ldo = N;
  return run_linear(A, K, B, M, N, K, e, (float*)workspace, (hipStream_t)stream);
}

tri_status tri_moe_route(const tri_layer_config* cfg, const float* h2, const void* w_router,
                         int32_t n_tokens, int32_t* idx, float* w, void* stream) {
  tri_status st = check_config(cfg);
  if (st != TRI_OK) return st;
  if (!is_moe(cfg)) return TRI_ERR_SHAPE;
  if (n_tokens < 0) return TRI_ERR_SHAPE;
  if (n_tokens == 0) return TRI_OK;
  if (!h2 || !w_router || !idx || !w) return TRI_ERR_NULL;
  if (!aligned16(h2) || !aligned16(w_router)) return TRI_ERR_ALIGN;
  StageTimer t_(ST_ROUTER, (hipStream_t)stream);
  TRI_HIP(launch_moe_route_f32(h2, w_router, n_tokens, cfg->hidden, cfg->n_experts, cfg->top_k,
                               (cfg->flags & TRI_F_MOE_RENORM) ? 1 : 0, idx, w,
                               (hipStream_t)stream, is_f32(cfg)));
  return TRI_OK;
}

tri_status tri_profile_enable(int32_t on) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  for (auto& r : p.pending) {
    hipEventSynchronize(r.b);
    p.pool.push_back(r.a);
    p.pool.push_back(r.b);
  }
  p.pending.clear();
  for (int i = 0; i < ST_COUNT; ++i) { p.launches[i] = 0; p.ms[i] = 0.0; }
  p.on = on != 0;
  return TRI_OK;
}

tri_status tri_profile_read(tri_profile* out) {
  if (!out) return TRI_ERR_NULL;
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  for (auto& r : p.pending) {
    if (hipEventSynchronize(r.b) != hipSuccess) return TRI_ERR_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return TRI_ERR_HIP;
    p.launches[r.stage] += 1;
    p.ms[r.stage] += ms;
    p.pool.push_back(r.a);
    p.pool.push_back(r.b);
  }
  p.pending.clear();
  out->n_stages = ST_COUNT;
  for (int i = 0; i < TRI_MAX_STAGES; ++i) {
    out->name[i] = i < ST_COUNT ? kStageName[i] : nullptr;
    out->launches[i] = i < ST_COUNT ? p.launches[i] : 0;
    out->total_ms[i] = i < ST_COUNT ? p.ms[i] : 0.0;
  }
  return TRI_OK;
}

const char* tri_status_string(tri_status s) {
  switch (s) {
    case TRI_OK: return "ok";
    case TRI_ERR_NULL: return "a required pointer is NULL";
    case TRI_ERR_SHAPE: return "inconsistent sizes";
    case TRI_ERR_UNSUPPORTED: return "unsupported configuration";
    case TRI_ERR_RANGE: return "size exceeds a buffer";
    case TRI_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case TRI_ERR_WORKSPACE: return "workspace too small";
    case TRI_ERR_HIP: return "HIP launch failed";
    case TRI_ERR_ALIAS: return "output overlaps an input";
    case TRI_ERR_SCRATCH: return "batch needs more than the fixed scratch of the no-allocation entry";
  }
  return "unknown status";
}

int32_t tri_version(void) { return 200; }

}  // extern "C"
