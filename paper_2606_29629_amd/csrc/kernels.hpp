// Internal launchers of libtri (host side).  Every launcher enqueues on
// `stream` and returns the hipError_t of its launch.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tri {

struct BatchDev {
  const int32_t* cu_q;
  const int32_t* ctx_len;
  const int32_t* slot;
  const int32_t* pos;
  int n_seqs, n_tokens, max_q_len, max_ctx_len;
};

// KV-cache addressing.  Contiguous (table == nullptr): K and V are
// [n_slots, Hkv, max_seq, D].  Paged: K and V are pools
// [n_blocks, Hkv, block_size, D] and logical row r of slot s lives in block
// table[s * (max_seq / block_size) + r / block_size] at row r % block_size.
// A panel is a slot (contiguous) or a block (paged) of panel_rows() rows;
// element (panel, kv head, row, d) is at ((panel Hkv + head) panel_rows + row) D + d.
struct KvDev {
  int n_slots, max_seq;     // logical: sequences and rows per sequence
  const int32_t* table;     // paged block table (device) or nullptr
  int block_size, n_blocks;
  __host__ __device__ int panel_rows() const { return table ? block_size : max_seq; }
  __host__ __device__ int blocks_per_slot() const { return table ? max_seq / block_size : 1; }
};

// Panel holding logical row `row` of slot `sl` (both in range), and the row
// within it; -1 when the block table entry is not a block of the pool.
__device__ __forceinline__ int kv_panel(const KvDev& kv, int sl, int row, int& prow) {
  if (!kv.table) {
    prow = row;
    return sl;
  }
  const int j = row / kv.block_size;
  prow = row - j * kv.block_size;
  const int blk = kv.table[(int64_t)sl * kv.blocks_per_slot() + j];
  return (blk >= 0 && blk < kv.n_blocks) ? blk : -1;
}

// Epilogue applied to C = A B^T (fp32 accumulators) by the GEMM kernels.
enum EpiKind { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3, EPI_STORE_F32 = 4 };
// Kernel-template epilogue ids: the kind in the low bits, kEpiF32 for fp32
// storage of the epilogue's tensors (output, residual, q, cache, bias, gains).
constexpr int kEpiKindMask = 15;
constexpr int kEpiF32 = 16;

struct Epi {
  int kind;
  int f32;            // 1: out, resid, q, cache, bias and gains are fp32 (fp32 storage mode)
  void* out;          // STORE / RESID / SWIGLU: storage type [M, ldo]; STORE_F32: float
  int ldo;
  const void* resid;  // RESID: storage type [M, ldr]
  int ldr;
  int ffn;            // SWIGLU: F; B rows [0,F) are gate, [F,2F) up; out has F cols
  // QKV: columns are q heads, then k heads, then v heads (head_dim each)
  const void* bias;   // nullable, [(Hq + 2 Hkv) D]
  void* q;            // bf16 [M, Hq, D]
  void* kc;           // cache K panels [*, Hkv, max_seq, D] (max_seq = panel rows)
  void* vc;           // cache V
  const int32_t* tok_slot;  // [M] cache panel of each token, -1 = skip the cache write
  const int32_t* tok_row;   // [M] row of each token within its panel
  const float2* rope;       // [M, D/2] (cos, sin)
  const void* q_norm;       // nullable [D] bf16: per-head RMSNorm gains of q (and k_norm of k)
  const void* k_norm;
  float eps;                // their epsilon
  int n_q_heads, n_kv_heads, head_dim, max_seq;
};

// Rotary frequency sections: frequency i < s0 takes position plane 0
// (pos[t]), i < s01 plane 1 (pos[T + t]), the rest plane 2 (pos[2 T + t]).
struct RopeSections {
  int s0, s01;
};

// Layer prologue: per-token map (cache panel and row within it of every
// token, -1 when out of range), the rotary table rope[t][i] = (cos, sin)(p *
// base^(-2i/D)) with p the token's position in frequency i's section (angle in
// double precision), and y = RMSNorm(x) * g.
// x, g, y are bf16, or fp32 with f32 (the fp32 storage mode).
hipError_t launch_prologue(const BatchDev& b, const KvDev& kv, int head_dim, float rope_base,
                           RopeSections sec, int32_t* tok_slot, int32_t* tok_row, float2* rope,
                           const void* x, const void* g, void* y, int hidden, float eps,
                           hipStream_t s, bool f32 = false);

// y = x / sqrt(mean(x^2) + eps) * g   (bf16 out with an optional fp32 copy, or
// fp32 in and out with f32)
hipError_t launch_rmsnorm(const void* x, const void* g, void* y, float* y32, int rows,
                          int hidden, float eps, hipStream_t s, bool f32 = false);

// bf16 planes of an fp32 matrix [rows, cols] (row stride ld_in) for the
// matrix cores: out [rows, 3 cols] = [hi | lo | hi] (pattern 0, activations)
// or [hi | hi | lo] (pattern 1, weights), hi = bf16(v), lo = bf16(v - hi);
// cols is a multiple of 4.
hipError_t launch_split3(const float* in, int64_t ld_in, int64_t rows, int cols, int pattern,
                         void* out, hipStream_t s);

// KV append for a batch given by its device arrays: cache row ctx_len[s] + i
// of slot slot[s] (through the block table when paged) <- row t of k_new /
// v_new (the sequence of each token is found by binary search over cu_q).
hipError_t launch_kv_append_direct(const BatchDev& b, const KvDev& kv, int n_kv_heads,
                                   int head_dim, const void* k_new, const void* v_new, void* kc,
                                   void* vc, hipStream_t s, bool f32 = false);

// Prefill GEMM (large M): C[M,N] = A[M,K] B[N,K]^T with the fused epilogue.
// `tail` (gemm_tail_bytes, may be null) holds the fp32 partials of the tiles
// of a final partial round, which then run split in K.
size_t gemm_tail_bytes();
hipError_t launch_gemm(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                       const Epi& epi, float* tail, hipStream_t s);

// fp32 C = A B^T as split-K planes [splits][M][N] (the consumer sums them
// in plane order); gemm_planes_splits picks the split count.
int gemm_planes_splits(int M, int N, int K);
hipError_t launch_gemm_planes(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                              float* planes, int splits, hipStream_t s);

// Decode projections (M <= 128): skinny tiles, split-K for narrow N; fp32
// partials in `part` (skinny_partial_bytes) reduced by an epilogue kernel.
int skinny_splits(int M, int N, int K, int kind);
// The O projection of a short batch fused with its residual add and the
// following RMSNorm (split-K planes reduced row by row): used when this
// returns true; out = x1 (bf16), y = RMSNorm(x1; g).
bool skinny_resid_norm_fused(int M, int N, int K);
hipError_t launch_skinny_resid_norm(const void* A, int lda, const void* B, int ldb, int M, int N,
                                    int K, const void* resid, int ldr, void* out, int ldo,
                                    const void* g, void* y, float eps, float* part, hipStream_t s);
size_t skinny_partial_bytes(int M, int N, int K, int kind);
hipError_t launch_skinny(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                         const Epi& epi, float* part, hipStream_t s);

// Causal flash attention for sequences with q_len > 1 (or all when
// include_single != 0).  A batch with few query tiles but long key ranges
// splits each query tile's keys over attn_prefill_splits() workgroups, whose
// fp32 partials (attn_prefill_partial_bytes, in `part`) a second kernel merges.
int attn_prefill_splits(int n_seqs, int n_tokens, int max_q_len, int max_ctx_len,
                        int n_q_heads);
size_t attn_prefill_partial_bytes(int n_seqs, int n_tokens, int max_q_len, int max_ctx_len,
                                  int n_q_heads, int head_dim);
// With f32 (the fp32 storage mode) q, the cache and out are fp32 and the key
// range is not split.
hipError_t launch_attn_prefill(const void* q, const void* kc, const void* vc, void* out,
                               const BatchDev& b, const KvDev& kv, int n_q_heads,
                               int n_kv_heads, int head_dim, int include_single, float* part,
                               hipStream_t s, bool f32 = false);

// Split-KV attention for sequences with q_len == 1, plus the combine.
// Keys per split (a multiple of 32); max_split > 0 caps it.
int attn_decode_split_keys(int n_seqs, int n_kv_heads, int max_kv, int head_dim, int group,
                           int max_split);
// The cap the split-KV kernel needs for this cache (0 = none).
int attn_decode_max_split(const KvDev& kv);
// Compute units of the current device (256 when it cannot be queried).
int cu_count();
size_t attn_decode_partial_bytes(int n_seqs, int n_q_heads, int head_dim, int max_kv);
hipError_t launch_attn_decode_split(const void* q, const void* kc, const void* vc, float* part,
                                    const BatchDev& b, const KvDev& kv, int n_q_heads,
                                    int n_kv_heads, int head_dim, hipStream_t s);
hipError_t launch_attn_decode_combine(const float* part, void* out, const BatchDev& b,
                                      const KvDev& kv, int n_q_heads, int n_kv_heads,
                                      int head_dim, hipStream_t s);

// Mixture of experts.  Grouped GEMM over experts: rows [seg[e], seg[e+1]) of
// the routed order belong to expert e; the gate/up pass gathers A rows
// perm[p] / top_k (perm = routed pair ids), the down pass reads A rows in
// routed order.  Tiles of moe_tile_rows(n_pairs, n_experts) rows.
int moe_tile_rows(int n_pairs, int n_experts);
hipError_t launch_gemm_grouped(const void* A, int lda, int a_rows, const int32_t* perm, int top_k,
                               const void* B, int64_t b_stride, int N, int K, const int32_t* seg,
                               const int32_t* tile_off, int n_experts, int n_pairs,
                               const Epi& epi, hipStream_t s);
// w_router bf16, or fp32 with w_f32 (the fp32 storage mode).
hipError_t launch_moe_route_f32(const float* h32, const void* w_router, int T, int H, int E,
                                int k, int renorm, int32_t* idx, float* w, hipStream_t s,
                                bool w_f32 = false);
size_t moe_route_planes_bytes(int T, int H, int E);
hipError_t launch_moe_route_bf16(const void* h, const void* w_router, int T, int H, int E, int k,
                                 int renorm, float* planes, int32_t* idx, float* w, hipStream_t s);
hipError_t launch_moe_permute(const int32_t* idx, int n_pairs, int E, int bm, int32_t* rank,
                              int32_t* counts, int32_t* perm, int32_t* inv, int32_t* seg,
                              int32_t* tile_off, hipStream_t s);
// x1 and out bf16, or fp32 with f32.
hipError_t launch_moe_combine(const void* x1, const float* y, const int32_t* inv, const float* w,
                              int T, int H, int k, void* out, hipStream_t s, bool f32 = false);

}  // namespace tri
