/*
 * tri.h -- C ABI of libtri: the Thinker decoder-layer forward on one MI355X
 * (gfx950), in the two arithmetic-intensity regimes the paper contrasts.
 *
 * The paper's Thinker stage (Section II-A) consumes its token stream in a
 * compute-bound prefill and then decodes autoregressively over a KV cache;
 * Section II-C (Observation 2) attributes prefill to dense GEMM kernels and
 * decode to GEMV-like operators, and Section III-A1 labels each scheduler step
 * prefill, decode or mixed from its per-request scheduled-token counts.  This
 * library computes one decoder layer for such a step:
 *
 *   h   = RMSNorm(x; attn_norm)                      y = x / sqrt(mean(x^2)+eps) * g
 *   q,k,v = h W_qkv^T (+ b_qkv), optionally each q and k head RMS-normalised
 *         (TRI_F_QK_NORM), rotary embedding on q and k at each token's
 *         position (rotate-half pairs (i, i+D/2), angle pos * base^(-2i/D)
 *         formed in double precision; with TRI_F_MROPE frequency i takes the
 *         temporal, height or width id of the token by its section), k and v
 *         appended to the cache
 *   o   = causal grouped-query softmax attention over the cache (query head j
 *         reads KV head floor(j*Hkv/Hq)), scale 1/sqrt(D)
 *   x1  = x + o W_o^T
 *   h2  = RMSNorm(x1; mlp_norm)
 *   out = x1 + SwiGLU(h2)                             dense
 *   out = x1 + sum_j w_j SwiGLU_{e_j}(h2)             MoE, top-k softmax routing
 *
 * The paper gives no layer equations; the structure is the Qwen2-family
 * pre-norm decoder of the model it serves (Section IV-A), and every
 * convention above is a declared reading.
 *
 * Conventions common to all entry points
 *  - Every pointer named "device" is a device (HBM) address; host structs are
 *    read during the call only.  The caller owns every buffer (weights, cache,
 *    activations, outputs, workspace); the library allocates nothing and keeps
 *    no pointer after returning.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *    stream) and never synchronise with the host.
 *  - Arguments are validated on the host before any launch; a negative status
 *    means nothing was launched and nothing was written.  TRI_ERR_HIP means a
 *    launch failed: outputs and this call's cache rows are then unspecified.
 *  - Device-side index arrays (cu_q, ctx_len, slot, pos) cannot be checked on
 *    the host.  Kernels never read or write outside the buffers described
 *    here: a token whose slot is >= n_slots or whose cache row is >= max_seq
 *    is skipped (its outputs are unspecified).
 *  - Element type ("storage type" below): bfloat16 (TRI_BF16, the serving
 *    path) or float32 (TRI_F32, the tight-parity mode) for the weights, the
 *    activations, the KV cache and the workspace intermediates, as
 *    tri_layer_config.dtype says; arithmetic accumulates in float32 in both.
 *    TRI_F32 runs the same kernels on fp32 storage: every projection on the
 *    matrix cores over bf16 operand planes of the fp32 values (activations
 *    split hi | lo | hi, weights hi | hi | lo, v = hi + lo with hi = bf16(v),
 *    lo = bf16(v - hi)), which keeps each product to ~2^-16 relative, and
 *    attention on the fp32 matrix instruction; it rebuilds the weight planes
 *    in the workspace on every call and is not meant for speed.  Weights are
 *    row-major [out, in].  All device buffers must be 16-byte aligned.
 */
#ifndef TRI_H
#define TRI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TRI_OK = 0,
  TRI_ERR_NULL = -1,        /* a required pointer is NULL                         */
  TRI_ERR_SHAPE = -2,       /* inconsistent sizes                                 */
  TRI_ERR_UNSUPPORTED = -3, /* valid but not implemented (dtype, head_dim, flag)  */
  TRI_ERR_RANGE = -4,       /* a size exceeds a buffer (e.g. ctx + q > max_seq)   */
  TRI_ERR_ALIGN = -5,       /* a device pointer is not 16-byte aligned            */
  TRI_ERR_WORKSPACE = -6,   /* workspace smaller than tri_workspace_size()        */
  TRI_ERR_HIP = -7,         /* a HIP launch failed                                */
  TRI_ERR_ALIAS = -8,       /* an output overlaps an input it must not overlap    */
  TRI_ERR_SCRATCH = -9      /* the call needs more than the library's fixed
                               scratch (tri_layer_decode_noalloc)               */
} tri_status;

typedef enum { TRI_BF16 = 0, TRI_F32 = 1 } tri_dtype;

enum {
  TRI_F_QKV_BIAS = 1,   /* add b_qkv after the q/k/v projection                   */
  TRI_F_MOE = 2,        /* mixture-of-experts FFN instead of the dense SwiGLU      */
  TRI_F_MOE_RENORM = 4, /* renormalise the top-k routing weights to sum to 1       */
  TRI_F_QK_NORM = 8,    /* per-head RMSNorm of q and k (gains q_norm, k_norm, eps
                           rms_eps) after the projection, before the rotation: the
                           Qwen3-family variant of the layer                         */
  TRI_F_MROPE = 16,     /* multi-section rotary positions (the multimodal rotary
                           embedding of the Qwen2-VL / Qwen2.5-Omni family): every
                           token has three position ids (temporal, height, width;
                           tri_batch.pos is then [3][n_tokens]) and rotary
                           frequency i < mrope_section[0] takes the temporal id,
                           i < mrope_section[0] + mrope_section[1] the height id,
                           the rest the width id                                     */
  TRI_F_ALL = 31
};

typedef struct {
  int32_t hidden;         /* H; multiple of 64                                      */
  int32_t n_q_heads;      /* Hq                                                     */
  int32_t n_kv_heads;     /* Hkv; Hq % Hkv == 0, Hq / Hkv <= 32                     */
  int32_t head_dim;       /* D in {64, 128}                                         */
  int32_t ffn_dim;        /* dense SwiGLU width F; multiple of 64 (dense only)      */
  int32_t n_experts;      /* E (MoE only), 1..256                                   */
  int32_t top_k;          /* k (MoE only), 1..min(E, 16)                            */
  int32_t expert_ffn_dim; /* per-expert SwiGLU width (MoE only); multiple of 64     */
  float rms_eps;          /* RMSNorm epsilon (>= 0)                                 */
  float rope_base;        /* rotary base (> 0)                                      */
  int32_t dtype;          /* tri_dtype: storage type of every tensor of the call    */
  int32_t flags;          /* TRI_F_* bits                                           */
  int32_t mrope_section[3]; /* TRI_F_MROPE: frequencies per section (temporal,
                             height, width), each >= 0, summing to D/2
                             (TRI_ERR_SHAPE otherwise); ignored without the flag   */
} tri_layer_config;

/* Device pointers to one layer's weights, row-major [out, in], storage type.   */
typedef struct {
  const void* attn_norm; /* [H]                                                    */
  const void* w_qkv;     /* [(Hq + 2 Hkv) D, H]: q heads, then k heads, then v     */
  const void* b_qkv;     /* [(Hq + 2 Hkv) D]; required iff TRI_F_QKV_BIAS          */
  const void* w_o;       /* [H, Hq D]                                              */
  const void* mlp_norm;  /* [H]                                                    */
  const void* w_gate_up; /* dense [2F, H] (gate rows [0,F), up rows [F,2F));
                            MoE   [E, 2Fe, H] (same split per expert)             */
  const void* w_down;    /* dense [H, F]; MoE [E, H, Fe]                           */
  const void* w_router;  /* MoE [E, H]; NULL for a dense layer                     */
  const void* q_norm;    /* [D]; required iff TRI_F_QK_NORM, else ignored          */
  const void* k_norm;    /* [D]; required iff TRI_F_QK_NORM, else ignored          */
} tri_layer_weights;

/* KV cache (device, storage type).  Keys are stored after the rotary embedding.
 * Row r of a slot holds the token at position r of the sequence occupying
 * that slot.  Two layouts:
 *  - contiguous (block_table == NULL): K and V each [n_slots, Hkv, max_seq, D];
 *  - paged, the fixed-size cache blocks of the PagedAttention memory manager
 *    under the serving framework of Section II-A: K and V are pools
 *    [n_blocks, Hkv, block_size, D], and row r of slot s lives in block
 *    block_table[s * (max_seq / block_size) + r / block_size] at row
 *    r % block_size.  block_size is a multiple of 64 that divides max_seq;
 *    block_table is device int32 [n_slots, max_seq / block_size], 4-byte
 *    aligned, and may leave entries that no row of the batch uses unset.
 *    An entry outside [0, n_blocks) is never dereferenced: its rows read as
 *    zero and writes to it are dropped (the sequence's results are then
 *    unspecified).  The layer reads and writes only the blocks the batch's
 *    rows map to.                                                               */
typedef struct {
  void* k;
  void* v;
  int32_t n_slots;              /* sequences (block-table rows when paged)       */
  int32_t max_seq;              /* logical rows per sequence                     */
  const int32_t* block_table;   /* NULL: contiguous                              */
  int32_t block_size;           /* paged: rows per block; else ignored           */
  int32_t n_blocks;             /* paged: blocks in each pool; else ignored      */
} tri_kv_cache;

/* A ragged batch (one scheduler step).  Host scalars size the launches; the
 * arrays are device int32.  Sequence s owns new tokens cu_q[s] .. cu_q[s+1]-1
 * of x; its new token i is written to cache row ctx_len[s] + i of slot
 * slot[s] and attends to rows 0 .. ctx_len[s] + i.  pos[t] is the rotary
 * position of token t (normally ctx_len + i); with TRI_F_MROPE, pos holds
 * three planes, pos[k * n_tokens + t] being id k (temporal, height, width) of
 * token t (for text tokens all three normally equal ctx_len + i).  The caller guarantees
 * ctx_len[s] + q_len[s] <= max_seq for every sequence; a sequence violating it
 * is skipped on the device (no access outside the cache).                     */
typedef struct {
  int32_t n_seqs;      /* >= 0                                                     */
  int32_t n_tokens;    /* T = cu_q[n_seqs]                                         */
  int32_t max_q_len;   /* >= max_s (cu_q[s+1] - cu_q[s])                           */
  int32_t max_ctx_len; /* >= max_s ctx_len[s]; < max_seq (TRI_ERR_RANGE otherwise) */
  const int32_t* cu_q;    /* [n_seqs + 1], cu_q[0] = 0, non-decreasing             */
  const int32_t* ctx_len; /* [n_seqs]                                              */
  const int32_t* slot;    /* [n_seqs], distinct                                    */
  const int32_t* pos;     /* [n_tokens], or [3][n_tokens] with TRI_F_MROPE         */
} tri_batch;

/* Byte offsets of the layer's intermediates inside the workspace (for
 * inspection after a call; contents are valid once the stream has finished).
 * Element type of h .. act: the storage type.                                 */
typedef struct {
  size_t h;      /* [T, H]   RMSNorm(x)                                             */
  size_t q;      /* [T, Hq, D] rotated queries                                      */
  size_t attn;   /* [T, Hq D] attention output                                      */
  size_t x1;     /* [T, H]   x + attn W_o^T                                         */
  size_t h2;     /* [T, H]   RMSNorm(x1)                                            */
  size_t act;    /* dense: [T, F] SwiGLU activation silu(g)*u;
                    MoE: [T*top_k, Fe], rows in routed order                       */
  size_t perm;   /* MoE: [T*top_k] int32 routed order -> pair id t*top_k + j
                    (pairs grouped by expert, ascending pair id within an expert)   */
  size_t y;      /* MoE: [T*top_k, H] fp32 expert outputs, rows in routed order     */
  size_t total;  /* == tri_workspace_size()                                         */
} tri_workspace_map;

/* Workspace bytes needed by tri_layer_prefill / tri_layer_decode for a batch
 * with these host scalars (device arrays are not read).  For a fixed config the
 * size never decreases as n_tokens grows (other scalars equal), so a workspace
 * sized for the largest batch serves every smaller one.                        */
tri_status tri_workspace_size(const tri_layer_config* cfg, const tri_batch* batch,
                              size_t* bytes);

/* The workspace layout used for this config and batch.                        */
tri_status tri_workspace_layout(const tri_layer_config* cfg, const tri_batch* batch,
                                tri_workspace_map* map);

/* One decoder layer over a ragged batch (prefill, chunked prefill with a
 * cached prefix, decode, or any mix: the mixed step of Section III-A1).
 *  x_in      device [T, H] storage type, token activations in batch order
 *  x_out     device [T, H] storage type, layer output; must not overlap x_in
 *  route_idx device [T, top_k] int32 or NULL (MoE: chosen experts, descending
 *            logit, ties to the lower expert index)
 *  route_w   device [T, top_k] float or NULL (MoE: routing weights)
 *  workspace device, >= tri_workspace_size() bytes, 256-byte aligned
 * Cache rows ctx_len[s] .. ctx_len[s] + q_len - 1 of every sequence are
 * written; no other cache row is touched.                                      */
tri_status tri_layer_prefill(const tri_layer_config* cfg, const tri_layer_weights* w,
                             const tri_kv_cache* cache, const tri_batch* batch,
                             const void* x_in, void* x_out, int32_t* route_idx,
                             float* route_w, void* workspace, size_t workspace_bytes,
                             void* stream);

/* The decode step (every sequence has exactly one new token: n_tokens ==
 * n_seqs, max_q_len == 1), on the memory-bound path: skinny projections that
 * stream each weight once and split-KV attention.  Same arguments and
 * results as tri_layer_prefill.                                                */
tri_status tri_layer_decode(const tri_layer_config* cfg, const tri_layer_weights* w,
                            const tri_kv_cache* cache, const tri_batch* batch,
                            const void* x_in, void* x_out, int32_t* route_idx,
                            float* route_w, void* workspace, size_t workspace_bytes,
                            void* stream);

/* The decode step of tri_layer_decode without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  The scratch lives
 * in a fixed device array of TRI_NOALLOC_SCRATCH_BYTES inside the library,
 * one per GPU, held until the process ends; the call itself allocates
 * nothing (no hipMalloc, no allocating library routine, no profiling events).
 * Same arguments and results as tri_layer_decode, minus the workspace.
 * Errors: those of tri_layer_decode; TRI_ERR_SCRATCH, before any launch, when
 * tri_workspace_size() of the batch exceeds TRI_NOALLOC_SCRATCH_BYTES (64 MiB:
 * the 7B-class decode at batch 64 and KV 4096 needs 34 MiB, the 128-expert
 * MoE decode at batch 128 and KV 2048 60 MiB); TRI_ERR_HIP if the scratch's
 * device address cannot be obtained.  Calls on one GPU share its scratch:
 * calls that overlap in time on one GPU (several streams or host threads)
 * race and must be serialised by the caller.                                */
#define TRI_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
tri_status tri_layer_decode_noalloc(const tri_layer_config* cfg, const tri_layer_weights* w,
                                    const tri_kv_cache* cache, const tri_batch* batch,
                                    const void* x_in, void* x_out, int32_t* route_idx,
                                    float* route_w, void* stream);

/* KV-cache append (the cache write of Section II-A's decode loop, done inside
 * the layer calls as well): for every new token t of sequence s,
 *   k[slot[s]][h][ctx_len[s] + i][:] = k_new[t][h][:]   (same for v).
 *  k_new, v_new  device [T, Hkv, D], storage type.                              */
tri_status tri_kvcache_append(const tri_layer_config* cfg, const tri_kv_cache* cache,
                              const tri_batch* batch, const void* k_new, const void* v_new,
                              void* stream);

/* Plain projection C = A B^T on the layer's GEMM kernels: the matrix
 * multiply of the Thinker's projections (Section II-A) and the synthetic
 * kernel of the paper's roofline benchmark over arithmetic intensity
 * (Section II-C, frequency-locked roofline benchmarking).
 *  A [M, K], B [N, K] (the nn.Linear weight layout), C [M, N]: bf16,
 *    row-major, device memory, 16-byte aligned; fp32 accumulation, C rounded
 *    to nearest even.  M, N, K >= 1, K a multiple of 64, N a multiple of 4,
 *    A and B each under 2 GiB; C overlaps neither operand.
 *  workspace: device scratch of tri_linear_workspace_size bytes (split
 *    partials; 256-byte aligned), or NULL when that size is 0.
 *  stream: hipStream_t (NULL = default stream).
 * Errors (before any launch): TRI_ERR_NULL, TRI_ERR_SHAPE, TRI_ERR_RANGE,
 * TRI_ERR_ALIGN, TRI_ERR_WORKSPACE, TRI_ERR_ALIAS; TRI_ERR_HIP if a launch
 * fails. */
tri_status tri_linear_workspace_size(int32_t M, int32_t N, int32_t K, size_t* bytes);
tri_status tri_linear(const void* A, const void* B, void* C, int32_t M, int32_t N, int32_t K,
                      void* workspace, size_t workspace_bytes, void* stream);

/* MoE routing alone (test hook for bit-exact routing): logits = h2 W_r^T in
 * float32 (one fixed summation order per logit), softmax over all experts,
 * top_k by logit (descending, ties to the lower index), weights p[idx]
 * (renormalised if TRI_F_MOE_RENORM).  Inside the layer the router reads h2
 * in the storage type (bf16 widened exactly to float32, or float32).
 *  h2        device [n_tokens, H] float32
 *  w_router  device [E, H] storage type
 *  idx, w    device [n_tokens, top_k] int32 / float32                          */
tri_status tri_moe_route(const tri_layer_config* cfg, const float* h2, const void* w_router,
                         int32_t n_tokens, int32_t* idx, float* w, void* stream);

/* Per-stage timing for benchmarks.  While enabled, the layer entry points
 * record a HIP event pair on the caller's stream around every stage (the
 * stage names are listed in tri_profile.name).  tri_profile_enable(1) resets
 * the counters; tri_profile_read waits for the recorded events and returns
 * launches and total milliseconds per stage.  Not thread-safe with
 * concurrent layer calls from several host threads.                          */
#define TRI_MAX_STAGES 16
typedef struct {
  int32_t n_stages;
  const char* name[TRI_MAX_STAGES];
  int32_t launches[TRI_MAX_STAGES];
  double total_ms[TRI_MAX_STAGES];
} tri_profile;

tri_status tri_profile_enable(int32_t on);
tri_status tri_profile_read(tri_profile* out);

/* Algorithmic work of one layer call, stage by stage: the per-kernel
 * arithmetic intensity from which Section III-C forms the time-weighted
 * intensity of a phase (Eq. 5).  Index i and name[i] are the stage of
 * tri_profile with the same index.  The counts follow the operations'
 * definitions, not the kernels' internals:
 *  flops  2 per multiply-add of every matrix product (the projections, the
 *         two attention products over the causally visible keys, the router,
 *         the experts); a stage without a product counts its multiply-adds
 *         (RMSNorm 4 per element, split merge 2 per partial element, MoE
 *         combine 2 per routed element).  Rotary, softmax and SwiGLU
 *         transcendentals are not counted.
 *  bytes  compulsory HBM traffic in the storage type: every input a stage
 *         reads and every output it writes, once (weights, activations, the
 *         K/V rows attended, once per KV head, cache rows written, the
 *         split-KV partials passed from attn_decode to attn_combine).
 *         On-chip re-reads are not counted.  (The model follows the bf16
 *         launch sequence; the fp32 mode's operand planes are not counted.)
 * Arguments (host memory):
 *  decode         1 for tri_layer_decode's launch sequence, 0 for
 *                 tri_layer_prefill's
 *  q_len, ctx_len [n_seqs] new tokens and cached prefix of each sequence
 *  expert_rows    MoE: [n_experts] routed rows per expert (summing to
 *                 n_tokens * top_k), or NULL, in which case min(E, T * top_k)
 *                 experts are taken as touched
 *  out            every stage filled; runs[i] = 1 iff the call launches stage i
 * Errors: TRI_ERR_NULL; the config's status; TRI_ERR_SHAPE for a negative
 * length, a decode sequence with q_len != 1 or expert_rows of the wrong sum.  */
typedef struct {
  int32_t n_stages;
  const char* name[TRI_MAX_STAGES];
  int32_t runs[TRI_MAX_STAGES];
  double flops[TRI_MAX_STAGES];
  double bytes[TRI_MAX_STAGES];
} tri_work;

tri_status tri_layer_work(const tri_layer_config* cfg, int32_t decode, int32_t n_seqs,
                          const int32_t* q_len, const int32_t* ctx_len,
                          const int32_t* expert_rows, tri_work* out);

/* Time-weighted arithmetic intensity of a phase (Section III-C, Eq. 5):
 *   ai = sum_i d_i (flops_i / bytes_i) / sum_i d_i
 * over the stages i with work->runs[i] set, d_i = prof->total_ms[i]; stages
 * with d_i = 0, or with no work (flops and bytes both 0), drop out.  The work of several calls may be summed stage by
 * stage first; a stage then stands for all its launches.  Host only.
 * Errors: TRI_ERR_NULL; TRI_ERR_SHAPE if the stage counts differ or no stage
 * has time; TRI_ERR_RANGE for a negative time or a timed stage with no bytes. */
tri_status tri_phase_intensity(const tri_work* work, const tri_profile* prof, double* ai);

/* Static description of a status code.                                         */
const char* tri_status_string(tri_status s);

/* Library version: major * 10000 + minor * 100 + patch.                         */
int32_t tri_version(void);

#ifdef __cplusplus
}
#endif
#endif /* TRI_H */
