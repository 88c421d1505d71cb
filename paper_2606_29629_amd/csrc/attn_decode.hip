// Split-KV decode attention for sequences with one new token.
//
// Decode attention reads the whole KV cache of every sequence once per step
// and does ~1 flop per byte, so it is HBM-bound.  The key range of each
// (sequence, KV head) is split into chunks of kSplitKeys so the grid holds
// enough workgroups to keep every CU streaming; one workgroup serves all query
// heads of its KV head (grouped-query reuse: K and V are read once for the
// whole group).
//
// Thread layout: D/8 lanes per key row, 8 dims (one 16-byte load) per lane.
// All K and V loads of the chunk are issued up front.  q.k uses bf16 dot2
// instructions; the per-head partial dots of the D/8 lanes of a key are
// reduced with a transposing butterfly (each exchange halves the number of
// heads a lane carries), so 8 heads cost 8 exchanges instead of 32.  Softmax
// statistics are per chunk (max in the log2 domain, sum); the combine kernel
// merges the chunks: M = max m_s, L = sum l_s 2^(m_s - M),
// o = sum acc_s 2^(m_s - M) / L.
#include "common.hpp"
#include "kernels.hpp"

namespace tri {

constexpr int kSplitKeys = 128;
constexpr int kMaxGroup = 8;  // query heads per KV head

int attn_decode_splits(int max_kv) { return cdiv(max_kv < 1 ? 1 : max_kv, kSplitKeys); }

size_t attn_decode_partial_bytes(int n_tokens, int n_q_heads, int head_dim, int max_kv) {
  return (size_t)n_tokens * n_q_heads * attn_decode_splits(max_kv) * (head_dim + 2) * sizeof(float);
}

template <int D>
__global__ __launch_bounds__(256) void attn_decode_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ Kc, const bf16* __restrict__ Vc,
    float* __restrict__ part, const int32_t* __restrict__ cu_q,
    const int32_t* __restrict__ ctx_len, const int32_t* __restrict__ slot, int n_slots,
    int max_seq, int Hq, int Hkv, int nsplit, float scale_log2e, int n_tokens) {
  constexpr int LPK = D / 8;          // lanes per key row
  constexpr int KPR = 256 / LPK;      // keys per round (workgroup)
  constexpr int ROUNDS = kSplitKeys / KPR;
  constexpr int G = kMaxGroup;
  __shared__ __align__(16) float sc[kSplitKeys][G];  // scores, then probabilities
  __shared__ __align__(16) float red[4][G][D];       // cross-wave reduction of P V
  __shared__ float stat[2][G];                       // chunk max (log2 domain), sum

  const int s = blockIdx.z, kvh = blockIdx.y, sp = blockIdx.x;
  const int t = cu_q[s];
  if (cu_q[s + 1] - t != 1 || t < 0 || t >= n_tokens) return;
  const int c = ctx_len[s], sl = slot[s];
  if (sl < 0 || sl >= n_slots || c < 0 || c + 1 > max_seq) return;
  const int L = c + 1;
  const int k_begin = sp * kSplitKeys;
  if (k_begin >= L) return;
  const int k_end = min(L, k_begin + kSplitKeys);
  const int grp = Hq / Hkv;
  const int qh0 = kvh * grp;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kl = tid / LPK, dc = tid % LPK;
  const int64_t cache_off = ((int64_t)sl * Hkv + kvh) * max_seq * D + dc * 8;

  u32x4 kr[ROUNDS], vr[ROUNDS];
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int key = min(k_begin + r * KPR + kl, k_end - 1);
    kr[r] = ldg16(Kc + cache_off + (int64_t)key * D);
  }
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    const int key = min(k_begin + r * KPR + kl, k_end - 1);
    vr[r] = ldg16(Vc + cache_off + (int64_t)key * D);
  }
  Pack8 qv[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    if (h < grp) qv[h].u = ldg16(Q + ((int64_t)t * Hq + qh0 + h) * D + dc * 8);
    else qv[h].u = u32x4{0u, 0u, 0u, 0u};
  }

  // ---- scores
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    Pack8 kk;
    kk.u = kr[r];
    float v[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float a = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2 qa = {qv[h].e[2 * e], qv[h].e[2 * e + 1]};
        const bf16x2 ka = {kk.e[2 * e], kk.e[2 * e + 1]};
        a = __builtin_amdgcn_fdot2_f32_bf16(qa, ka, a, false);
      }
      v[h] = a;
    }
    // Transposing butterfly over the LPK lanes of this key.
    int nv = G, head = 0;
#pragma unroll
    for (int m = LPK / 2; m >= 1; m >>= 1) {
      if (nv > 1) {
        const bool up = (dc & m) != 0;
        const int hv = nv / 2;
#pragma unroll
        for (int i = 0; i < G / 2; ++i) {
          if (i < hv) {
            const float send = up ? v[i] : v[i + hv];
            const float keep = up ? v[i + hv] : v[i];
            v[i] = keep + __shfl_xor(send, m, 64);
          }
        }
        if (up) head += hv;
        nv = hv;
      } else {
        v[0] += __shfl_xor(v[0], m, 64);
      }
    }
    // After the butterfly every lane holds the full dot of head `head`;
    // lanes of a key carry each head at least once.
    const int key_local = r * KPR + kl;
    const bool first = (dc & ((LPK / G > 1) ? (LPK / G - 1) : 0)) == 0;
    if (first) {
      const int key = k_begin + key_local;
      sc[key_local][head] = key < k_end ? v[0] * scale_log2e : -INFINITY;
    }
  }
  __syncthreads();

  // ---- chunk softmax statistics: wave w handles heads w and w + 4
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int h = wave + 4 * hh;
    float mx = -INFINITY;
    for (int k = lane; k < kSplitKeys; k += 64) mx = fmaxf(mx, sc[k][h]);
    mx = wave_max(mx);
    float sum = 0.f;
    for (int k = lane; k < kSplitKeys; k += 64) {
      const float p = exp2f(sc[k][h] - mx);
      sc[k][h] = p;
      sum += p;
    }
    sum = wave_sum(sum);
    if (lane == 0) {
      stat[0][h] = mx;
      stat[1][h] = sum;
    }
  }
  __syncthreads();

  // ---- P V
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
#pragma unroll
  for (int r = 0; r < ROUNDS; ++r) {
    Pack8 vv;
    vv.u = vr[r];
    const int key_local = r * KPR + kl;
    const f32x4 p0 = *(const f32x4*)&sc[key_local][0];
    const f32x4 p1 = *(const f32x4*)&sc[key_local][4];
    const float p[G] = {p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], p1[2], p1[3]};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = bf2f(vv.e[e]);
#pragma unroll
      for (int h = 0; h < G; ++h) acc[h][e] += p[h] * x;
    }
  }
  // lanes of a wave with the same dc: dc + LPK * j
#pragma unroll
  for (int m = LPK; m < 64; m <<= 1)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] += __shfl_xor(acc[h][e], m, 64);
  if (lane < LPK) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) red[wave][h][dc * 8 + e] = acc[h][e];
  }
  __syncthreads();
  for (int i = tid; i < G * D; i += 256) {
    const int h = i / D, d = i % D;
    if (h >= grp) continue;
    const float o = red[0][h][d] + red[1][h][d] + red[2][h][d] + red[3][h][d];
    float* pp = part + (((int64_t)t * Hq + qh0 + h) * nsplit + sp) * (D + 2);
    pp[d] = o;
    if (d == 0) {
      pp[D] = stat[0][h];
      pp[D + 1] = stat[1][h];
    }
  }
}

// One workgroup of D threads per (sequence, query head).
template <int D>
__global__ __launch_bounds__(128) void attn_combine_kernel(
    const float* __restrict__ part, bf16* __restrict__ O, const int32_t* __restrict__ cu_q,
    const int32_t* __restrict__ ctx_len, const int32_t* __restrict__ slot, int n_slots,
    int max_seq, int Hq, int nsplit, int n_tokens) {
  const int s = blockIdx.x, qh = blockIdx.y, d = threadIdx.x;
  const int t = cu_q[s];
  if (cu_q[s + 1] - t != 1 || t < 0 || t >= n_tokens) return;
  const int c = ctx_len[s], sl = slot[s];
  if (sl < 0 || sl >= n_slots || c < 0 || c + 1 > max_seq) return;
  const int ns = min(cdiv(c + 1, kSplitKeys), nsplit);  // never past the launched splits
  const float* pp = part + ((int64_t)t * Hq + qh) * nsplit * (D + 2);
  float M = -INFINITY;
  for (int i = 0; i < ns; ++i) M = fmaxf(M, pp[i * (D + 2) + D]);
  float Lsum = 0.f, o = 0.f;
  for (int i = 0; i < ns; ++i) {
    const float w = exp2f(pp[i * (D + 2) + D] - M);
    Lsum += pp[i * (D + 2) + D + 1] * w;
    o += pp[i * (D + 2) + d] * w;
  }
  O[((int64_t)t * Hq + qh) * D + d] = f2bf(o / Lsum);
}

hipError_t launch_attn_decode_split(const void* q, const void* kc, const void* vc, float* part,
                                    const BatchDev& b, int n_slots, int max_seq, int n_q_heads,
                                    int n_kv_heads, int head_dim, hipStream_t s) {
  if (b.n_seqs == 0) return hipSuccess;
  const int nsplit = attn_decode_splits(b.max_ctx_len + 1);
  const float scale_log2e = (float)(1.4426950408889634 / __builtin_sqrt((double)head_dim));
  dim3 grid(nsplit, n_kv_heads, b.n_seqs);
  if (head_dim == 128)
    attn_decode_kernel<128><<<grid, 256, 0, s>>>((const bf16*)q, (const bf16*)kc, (const bf16*)vc,
                                                 part, b.cu_q, b.ctx_len, b.slot, n_slots, max_seq,
                                                 n_q_heads, n_kv_heads, nsplit, scale_log2e, b.n_tokens);
  else
    attn_decode_kernel<64><<<grid, 256, 0, s>>>((const bf16*)q, (const bf16*)kc, (const bf16*)vc,
                                                part, b.cu_q, b.ctx_len, b.slot, n_slots, max_seq,
                                                n_q_heads, n_kv_heads, nsplit, scale_log2e, b.n_tokens);
  return hipGetLastError();
}

hipError_t launch_attn_decode_combine(const float* part, void* out, const BatchDev& b,
                                      int n_slots, int max_seq, int n_q_heads, int head_dim,
                                      hipStream_t s) {
  if (b.n_seqs == 0) return hipSuccess;
  const int nsplit = attn_decode_splits(b.max_ctx_len + 1);
  dim3 cgrid(b.n_seqs, n_q_heads);
  if (head_dim == 128)
    attn_combine_kernel<128><<<cgrid, 128, 0, s>>>(part, (bf16*)out, b.cu_q, b.ctx_len, b.slot,
                                                   n_slots, max_seq, n_q_heads, nsplit, b.n_tokens);
  else
    attn_combine_kernel<64><<<cgrid, 64, 0, s>>>(part, (bf16*)out, b.cu_q, b.ctx_len, b.slot,
                                                 n_slots, max_seq, n_q_heads, nsplit, b.n_tokens);
  return hipGetLastError();
}

}  // namespace tri
