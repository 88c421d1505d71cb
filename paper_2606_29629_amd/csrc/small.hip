// Bandwidth-bound helper kernels: layer prologue (token map + rotary table +
// RMSNorm), RMSNorm, KV append, and the bf16 operand planes of the fp32
// storage mode.  Kernels templated on F32 are instantiated for bf16 storage
// (the product path) and fp32 storage (the tight-parity mode).
#include "common.hpp"
#include "kernels.hpp"

namespace tri {

// RMSNorm: one wave per row, 8 bf16 per lane per pass, fp32 sum of squares.
constexpr int kNormMaxChunks = 16;  // hidden <= 64 lanes * 8 * 16 = 8192

// fp32 storage: y = x / sqrt(mean(x^2) + eps) * g over one row, a wave per
// row in two passes (sum of squares, then the scaled product).
__device__ __forceinline__ void rmsnorm_row_f32(const float* __restrict__ xr,
                                                const float* __restrict__ g,
                                                float* __restrict__ yr, int hidden, float eps,
                                                int lane) {
  float ss = 0.f;
  for (int i = 4 * lane; i < hidden; i += 256) {
    const f32x4 v = *(const f32x4*)(xr + i);
    ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)hidden + eps);
  for (int i = 4 * lane; i < hidden; i += 256) {
    const f32x4 v = *(const f32x4*)(xr + i), gv = *(const f32x4*)(g + i);
    *(f32x4*)(yr + i) = f32x4{v[0] * r * gv[0], v[1] * r * gv[1], v[2] * r * gv[2],
                              v[3] * r * gv[3]};
  }
}

template <bool F32>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const void* __restrict__ xv,
                                                      const void* __restrict__ gv_,
                                                      void* __restrict__ yv,
                                                      float* __restrict__ y32, int rows,
                                                      int hidden, float eps) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  if constexpr (F32) {
    rmsnorm_row_f32((const float*)xv + (int64_t)row * hidden, (const float*)gv_,
                    (float*)yv + (int64_t)row * hidden, hidden, eps, lane);
    return;
  }
  const bf16* __restrict__ x = (const bf16*)xv;
  const bf16* __restrict__ g = (const bf16*)gv_;
  bf16* __restrict__ y = (bf16*)yv;
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
                          float eps, hipStream_t s, bool f32) {
  if (rows == 0) return hipSuccess;
  if (f32)
    rmsnorm_kernel<true><<<cdiv(rows, 4), 256, 0, s>>>(x, g, y, nullptr, rows, hidden, eps);
  else
    rmsnorm_kernel<false><<<cdiv(rows, 4), 256, 0, s>>>(x, g, y, y32, rows, hidden, eps);
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

template <bool F32>
__global__ __launch_bounds__(256) void prologue_kernel(BatchDev b, KvDev kv, int half,
                                                       double base, RopeSections sec,
                                                       int32_t* __restrict__ tok_slot,
                                                       int32_t* __restrict__ tok_row,
                                                       float2* __restrict__ rope,
                                                       const void* __restrict__ xv,
                                                       const void* __restrict__ gv_,
                                                       void* __restrict__ yv, int hidden,
                                                       float eps) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= b.n_tokens) return;
  const bf16* __restrict__ x = (const bf16*)xv;
  const bf16* __restrict__ g = (const bf16*)gv_;
  bf16* __restrict__ y = (bf16*)yv;
  // x, g and the position first: their latency overlaps the map.
  const bf16* xr = x + (int64_t)t * hidden;
  const int nchunk = hidden / 8;
  Pack8 v[kNormMaxChunks], gv[kNormMaxChunks];
  if constexpr (!F32) {
#pragma unroll
    for (int c = 0; c < kNormMaxChunks; ++c) {
      const int ch = lane + c * 64;
      if (ch < nchunk) {
        v[c].u = ldg16(xr + ch * 8);
        gv[c].u = ldg16(g + ch * 8);
      }
    }
  }
  const int plane = lane < sec.s0 ? 0 : (lane < sec.s01 ? 1 : 2);
  const int pos = b.pos[(int64_t)(lane < half ? plane : 0) * b.n_tokens + t];
  // The frequency needs no memory: it is formed while the loads are in flight.
  const double inv_freq = lane < half ? pow(base, -2.0 * (double)lane / (double)(2 * half)) : 0.0;
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
  // The sequence's descriptors (the same for the whole wave) are loaded here
  // and used last, so their latency overlaps the rotary table and the norm.
  const bool in_batch = sq < b.n_seqs;
  const int sc = in_batch ? sq : 0;
  const int q0 = b.cu_q[sc], q1 = b.cu_q[sc + 1], sl = b.slot[sc], c0 = b.ctx_len[sc];
  if (lane < half) {
    const double ang = (double)pos * inv_freq;
    double sn, cs;
    sincos(ang, &sn, &cs);
    rope[(int64_t)t * half + lane] = make_float2((float)cs, (float)sn);
  }
  if constexpr (F32) {
    rmsnorm_row_f32((const float*)xv + (int64_t)t * hidden, (const float*)gv_,
                    (float*)yv + (int64_t)t * hidden, hidden, eps, lane);
  } else {
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
  if (lane == 0) {
    const int row = c0 + (t - q0);
    const bool ok = in_batch && sl >= 0 && sl < kv.n_slots && row >= 0 && row < kv.max_seq &&
                    t >= q0 && t < q1;
    int prow = -1;
    const int panel = ok ? kv_panel(kv, sl, row, prow) : -1;
    tok_slot[t] = panel;
    tok_row[t] = panel >= 0 ? prow : -1;
  }
}

hipError_t launch_prologue(const BatchDev& b, const KvDev& kv, int head_dim, float rope_base,
                           RopeSections sec, int32_t* tok_slot, int32_t* tok_row, float2* rope,
                           const void* x, const void* g, void* y, int hidden, float eps,
                           hipStream_t s, bool f32) {
  if (b.n_tokens == 0) return hipSuccess;
  if (f32)
    prologue_kernel<true><<<cdiv(b.n_tokens, 4), 256, 0, s>>>(
        b, kv, head_dim / 2, (double)rope_base, sec, tok_slot, tok_row, rope, x, g, y, hidden,
        eps);
  else
    prologue_kernel<false><<<cdiv(b.n_tokens, 4), 256, 0, s>>>(
        b, kv, head_dim / 2, (double)rope_base, sec, tok_slot, tok_row, rope, x, g, y, hidden,
        eps);
  return hipGetLastError();
}

// One thread per 16-byte chunk of a new K/V row (8 bf16 or 4 fp32 values).
template <typename T>
__global__ void kv_append_direct_kernel(BatchDev b, KvDev kv, int hkv, int d,
                                        const T* __restrict__ kn, const T* __restrict__ vn,
                                        T* __restrict__ kc, T* __restrict__ vc) {
  constexpr int EPC = 16 / sizeof(T);  // elements per chunk
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int cpr = d / EPC;
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
  const int64_t dst = (((int64_t)panel * hkv + h) * kv.panel_rows() + prow) * d + c * EPC;
  const int64_t src = ((int64_t)t * hkv + h) * d + c * EPC;
  stg16(kc + dst, ldg16(kn + src));
  stg16(vc + dst, ldg16(vn + src));
}

hipError_t launch_kv_append_direct(const BatchDev& b, const KvDev& kv, int n_kv_heads,
                                   int head_dim, const void* k_new, const void* v_new, void* kc,
                                   void* vc, hipStream_t s, bool f32) {
  const int64_t n = (int64_t)b.n_tokens * n_kv_heads * (head_dim / (f32 ? 4 : 8));
  if (n == 0 || b.n_seqs == 0) return hipSuccess;
  if (f32)
    kv_append_direct_kernel<float><<<(unsigned)((n + 255) / 256), 256, 0, s>>>(
        b, kv, n_kv_heads, head_dim, (const float*)k_new, (const float*)v_new, (float*)kc,
        (float*)vc);
  else
    kv_append_direct_kernel<bf16><<<(unsigned)((n + 255) / 256), 256, 0, s>>>(
        b, kv, n_kv_heads, head_dim, (const bf16*)k_new, (const bf16*)v_new, (bf16*)kc,
        (bf16*)vc);
  return hipGetLastError();
}

// bf16 operand planes of an fp32 matrix for the matrix cores (fp32 storage
// mode): each value v splits into hi = bf16(v) and lo = bf16(v - hi) (the
// difference exact in fp32; hi + lo keeps ~16 significant bits of v), and
// row r of the output [rows, 3 cols] holds three planes of the row: pattern
// 0 [hi | lo | hi], pattern 1 [hi | hi | lo].  A product of a pattern-0 row
// and a pattern-1 row over 3 cols is a_hi b_hi + a_lo b_hi + a_hi b_lo: the
// fp32 product up to the a_lo b_lo term and the splits' rounding (2^-16
// relative).  One thread per 4 values; cols is a multiple of 4, ld_in the
// input row stride.
__global__ __launch_bounds__(256) void split3_kernel(const float* __restrict__ in, int64_t ld_in,
                                                     int64_t rows, int cols, int pattern,
                                                     bf16* __restrict__ out) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int q = cols / 4;
  if (gid >= rows * q) return;
  const int64_t r = gid / q;
  const int c = (int)(gid - r * q) * 4;
  const f32x4 v = *(const f32x4*)(in + r * ld_in + c);
  bf16x4 hi, lo;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    hi[e] = f2bf(v[e]);
    lo[e] = f2bf(v[e] - bf2f(hi[e]));
  }
  bf16* o = out + r * 3 * (int64_t)cols + c;
  *(bf16x4*)o = hi;
  *(bf16x4*)(o + cols) = pattern == 0 ? lo : hi;
  *(bf16x4*)(o + 2 * cols) = pattern == 0 ? hi : lo;
}

hipError_t launch_split3(const float* in, int64_t ld_in, int64_t rows, int cols, int pattern,
                         void* out, hipStream_t s) {
  const int64_t n = rows * (cols / 4);
  if (n == 0) return hipSuccess;
  split3_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(in, ld_in, rows, cols, pattern,
                                                            (bf16*)out);
  return hipGetLastError();
}

}  // namespace tri
