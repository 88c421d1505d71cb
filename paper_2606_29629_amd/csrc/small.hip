// Bandwidth-bound helper kernels: layer prologue (token map + rotary table +
// RMSNorm), RMSNorm, KV append.
#include "common.hpp"
#include "kernels.hpp"

namespace tri {

// RMSNorm: one wave per row, 8 bf16 per lane per pass, fp32 sum of squares.
constexpr int kNormMaxChunks = 16;  // hidden <= 64 lanes * 8 * 16 = 8192

__global__ __launch_bounds__(256) void rmsnorm_kernel(const bf16* __restrict__ x,
                                                      const bf16* __restrict__ g,
                                                      bf16* __restrict__ y,
                                                      float* __restrict__ y32, int rows,
                                                      int hidden, float eps) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const bf16* xr = x + (int64_t)row * hidden;
  const int nchunk = hidden / 8;
  Pack8 v[kNormMaxChunks], gv[kNormMaxChunks];
  float ss = 0.f;
  // x and g both loaded up front: one memory round trip before the reduction.
#pragma unroll
  for (int c = 0; c < kNormMaxChunks; ++c) {
    const int ch = lane + c * 64;
    if (ch < nchunk) {
      v[c].u = ldg16(xr + ch * 8);
      gv[c].u = ldg16(g + ch * 8);
    }
  }
#pragma unroll
  for (int c = 0; c < kNormMaxChunks; ++c) {
    const int ch = lane + c * 64;
    if (ch < nchunk) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float f = bf2f(v[c].e[e]);
        ss += f * f;
      }
    }
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)hidden + eps);
#pragma unroll
  for (int c = 0; c < kNormMaxChunks; ++c) {
    const int ch = lane + c * 64;
    if (ch < nchunk) {
      Pack8 o;
      float f[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        f[e] = bf2f(v[c].e[e]) * r * bf2f(gv[c].e[e]);
        o.e[e] = f2bf(f[e]);
      }
      stg16(y + (int64_t)row * hidden + ch * 8, o.u);
      if (y32) {
        float* d = y32 + (int64_t)row * hidden + ch * 8;
        *(f32x4*)d = f32x4{f[0], f[1], f[2], f[3]};
        *(f32x4*)(d + 4) = f32x4{f[4], f[5], f[6], f[7]};
      }
    }
  }
}

hipError_t launch_rmsnorm(const void* x, const void* g, void* y, float* y32, int rows, int hidden,
                          float eps, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  rmsnorm_kernel<<<cdiv(rows, 4), 256, 0, s>>>((const bf16*)x, (const bf16*)g, (bf16*)y, y32,
                                               rows, hidden, eps);
  return hipGetLastError();
}

// Layer prologue, one wave per token t:
//  * token map: the sequence holding t is the number of sequence ends
//    cu_q[1 .. n_seqs] at or below t; the wave loads the ends 64 per lane
//    group at once and counts them with ballots, so the map costs two memory
//    round trips (ends, then the sequence's slot / prefix / start) however
//    many sequences there are, instead of one per bisection step;
//  * rotary table rope[t][i] = (cos, sin)(p * base^(-2i/D)), the angle
//    formed in double precision, lane i < D/2, p = pos[k T + t] for the
//    section k of frequency i (k = 0 for a one-plane position array);
//  * RMSNorm of x[t] into y[t] (as rmsnorm_kernel).
constexpr int kMapChunks = 4;  // sequence ends loaded per lane and round trip

__global__ __launch_bounds__(256) void prologue_kernel(BatchDev b, KvDev kv, int half,
                                                       double base, RopeSections sec,
                                                       int32_t* __restrict__ tok_slot,
                                                       int32_t* __restrict__ tok_row,
                                                       float2* __restrict__ rope,
                                                       const bf16* __restrict__ x,
                                                       const bf16* __restrict__ g,
                                                       bf16* __restrict__ y, int hidden,
                                                       float eps) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= b.n_tokens) return;
  // x, g and the position first: their latency overlaps the map.
  const bf16* xr = x + (int64_t)t * hidden;
  const int nchunk = hidden / 8;
  Pack8 v[kNormMaxChunks], gv[kNormMaxChunks];
#pragma unroll
  for (int c = 0; c < kNormMaxChunks; ++c) {
    const int ch = lane + c * 64;
    if (ch < nchunk) {
      v[c].u = ldg16(xr + ch * 8);
      gv[c].u = ldg16(g + ch * 8);
    }
  }
  const int plane = lane < sec.s0 ? 0 : (lane < sec.s01 ? 1 : 2);
  const int pos = b.pos[(int64_t)(lane < half ? plane : 0) * b.n_tokens + t];
  int sq = 0;
  for (int j0 = 0; j0 < b.n_seqs; j0 += 64 * kMapChunks) {
    int end[kMapChunks];
#pragma unroll
    for (int c = 0; c < kMapChunks; ++c) {
      const int j = j0 + 64 * c + lane;
      const int e = b.cu_q[min(j, b.n_seqs - 1) + 1];  // clamped: no branch around the load
      end[c] = j < b.n_seqs ? e : INT32_MAX;
    }
#pragma unroll
    for (int c = 0; c < kMapChunks; ++c)
      sq += __builtin_popcountll(__builtin_amdgcn_ballot_w64(end[c] <= t));
  }
  if (lane == 0) {
    bool ok = sq < b.n_seqs;
    const int sc = ok ? sq : 0;
    const int q0 = b.cu_q[sc], q1 = b.cu_q[sc + 1], sl = b.slot[sc], c0 = b.ctx_len[sc];
    const int row = c0 + (t - q0);
    ok = ok && sl >= 0 && sl < kv.n_slots && row >= 0 && row < kv.max_seq && t >= q0 && t < q1;
    int prow = -1;
    const int panel = ok ? kv_panel(kv, sl, row, prow) : -1;
    tok_slot[t] = panel;
    tok_row[t] = panel >= 0 ? prow : -1;
  }
  if (lane < half) {
    const double inv_freq = pow(base, -2.0 * (double)lane / (double)(2 * half));
    const double ang = (double)pos * inv_freq;
    double sn, cs;
    sincos(ang, &sn, &cs);
    rope[(int64_t)t * half + lane] = make_float2((float)cs, (float)sn);
  }
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < kNormMaxChunks; ++c) {
    const int ch = lane + c * 64;
    if (ch < nchunk) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float f = bf2f(v[c].e[e]);
        ss += f * f;
      }
    }
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)hidden + eps);
#pragma unroll
  for (int c = 0; c < kNormMaxChunks; ++c) {
    const int ch = lane + c * 64;
    if (ch < nchunk) {
      Pack8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o.e[e] = f2bf(bf2f(v[c].e[e]) * r * bf2f(gv[c].e[e]));
      stg16(y + (int64_t)t * hidden + ch * 8, o.u);
    }
  }
}

hipError_t launch_prologue(const BatchDev& b, const KvDev& kv, int head_dim, float rope_base,
                           RopeSections sec, int32_t* tok_slot, int32_t* tok_row, float2* rope,
                           const void* x, const void* g, void* y, int hidden, float eps,
                           hipStream_t s) {
  if (b.n_tokens == 0) return hipSuccess;
  prologue_kernel<<<cdiv(b.n_tokens, 4), 256, 0, s>>>(
      b, kv, head_dim / 2, (double)rope_base, sec, tok_slot, tok_row, rope,
      (const bf16*)x, (const bf16*)g, (bf16*)y, hidden, eps);
  return hipGetLastError();
}

// One thread per 16-byte chunk of a new K/V row.
__global__ void kv_append_direct_kernel(BatchDev b, KvDev kv, int hkv, int d,
                                        const bf16* __restrict__ kn, const bf16* __restrict__ vn,
                                        bf16* __restrict__ kc, bf16* __restrict__ vc) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int cpr = d / 8;
  if (gid >= (int64_t)b.n_tokens * hkv * cpr) return;
  const int t = (int)(gid / (hkv * cpr));
  const int rem = (int)(gid - (int64_t)t * hkv * cpr);
  const int h = rem / cpr, c = rem - h * cpr;
  int lo = 0, hi = b.n_seqs;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (b.cu_q[mid] <= t) lo = mid; else hi = mid;
  }
  const int sl = b.slot[lo];
  const int row = b.ctx_len[lo] + (t - b.cu_q[lo]);
  if (sl < 0 || sl >= kv.n_slots || row < 0 || row >= kv.max_seq || t >= b.cu_q[lo + 1]) return;
  int prow;
  const int panel = kv_panel(kv, sl, row, prow);
  if (panel < 0) return;
  const int64_t dst = (((int64_t)panel * hkv + h) * kv.panel_rows() + prow) * d + c * 8;
  const int64_t src = ((int64_t)t * hkv + h) * d + c * 8;
  stg16(kc + dst, ldg16(kn + src));
  stg16(vc + dst, ldg16(vn + src));
}

hipError_t launch_kv_append_direct(const BatchDev& b, const KvDev& kv, int n_kv_heads,
                                   int head_dim, const void* k_new, const void* v_new, void* kc,
                                   void* vc, hipStream_t s) {
  const int64_t n = (int64_t)b.n_tokens * n_kv_heads * (head_dim / 8);
  if (n == 0 || b.n_seqs == 0) return hipSuccess;
  kv_append_direct_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(
      b, kv, n_kv_heads, head_dim, (const bf16*)k_new, (const bf16*)v_new, (bf16*)kc,
      (bf16*)vc);
  return hipGetLastError();
}

}  // namespace tri
