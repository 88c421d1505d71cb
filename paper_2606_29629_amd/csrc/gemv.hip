// Decode projections: C[M,N] = X[M,K] W[N,K]^T with small M (one row per
// sequence in the batch).  Arithmetic intensity is ~M flop/byte, far below
// the MI355X ridge (~315 flop/B), so the kernel is built to stream W from HBM
// exactly once at full bandwidth; X (<= 128 rows) stays in L2.
//
// Each wave owns 32 rows of W (32 output columns) and a K range, and uses
// v_mfma_f32_32x32x16_bf16 with X as the A operand (rows = tokens) and W as
// the B operand.  Per 64-wide k step, lane (n = l%32, g = l/32) loads 64
// contiguous bytes of W row n at k + 32g; MFMA j consumes the lane's j-th
// 8-element slice.  X fragments use the same k assignment, so the product is
// the plain dot product over k.  Two k steps are in flight per wave.
//
// K is split across the grid's y dimension so that enough waves stream W to
// saturate HBM; fp32 partials [split][M][N] are reduced in a fixed order by the
// epilogue kernel, which also applies the fused epilogue (deterministic).
#include "common.hpp"
#include "kernels.hpp"

namespace tri {

constexpr int kGvCols = 128;   // columns per workgroup (4 waves x 32)
constexpr int kGvStep = 64;    // k per step

int gemv_splits(int M, int N, int K) {
  (void)M;
  const int waves = cdiv(N, 32);
  const int target = 2048;  // ~8 waves per CU on 256 CUs
  int splits = cdiv(target, waves);
  const int max_splits = K / 256;  // at least 256 k per split
  if (splits > max_splits) splits = max_splits;
  if (splits < 1) splits = 1;
  // Split boundaries fall on kGvStep multiples.
  const int steps = K / kGvStep;
  const int per = cdiv(steps, splits);
  return cdiv(steps, per);
}

size_t gemv_partial_bytes(int M, int N, int K) {
  return (size_t)gemv_splits(M, N, K) * M * N * sizeof(float);
}

template <int MB>
__global__ __launch_bounds__(256) void gemv_kernel(const bf16* __restrict__ X, int ldx,
                                                   const bf16* __restrict__ W, int ldw, int M,
                                                   int N, int K, int kper,
                                                   float* __restrict__ part) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * kGvCols + wave * 32;
  if (n0 >= N) return;
  const int lr = lane & 31, lg = lane >> 5;
  const int ks = blockIdx.y * kper;
  const int ke = min(K, ks + kper);
  const bf16* wp = W + (int64_t)min(n0 + lr, N - 1) * ldw + 32 * lg;
  const bf16* xp[MB];
#pragma unroll
  for (int b = 0; b < MB; ++b) xp[b] = X + (int64_t)min(32 * b + lr, M - 1) * ldx + 32 * lg;

  f32x16 acc[MB];
#pragma unroll
  for (int b = 0; b < MB; ++b) acc[b] = f32x16{0.f};

  bf16x8 wc[4], xc[MB][4], wn[4], xn[MB][4];
  auto load = [&](int k, bf16x8 (&w4)[4], bf16x8 (&x4)[MB][4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) w4[j] = *(const bf16x8*)(wp + k + 8 * j);
#pragma unroll
    for (int b = 0; b < MB; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) x4[b][j] = *(const bf16x8*)(xp[b] + k + 8 * j);
  };
  auto mma = [&](bf16x8 (&w4)[4], bf16x8 (&x4)[MB][4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int b = 0; b < MB; ++b)
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x4[b][j], w4[j], acc[b], 0, 0, 0);
  };

  int k = ks;
  if (k < ke) load(k, wc, xc);
  for (; k < ke; k += 2 * kGvStep) {
    const bool has1 = k + kGvStep < ke;
    if (has1) load(k + kGvStep, wn, xn);
    mma(wc, xc);
    if (!has1) break;
    if (k + 2 * kGvStep < ke) load(k + 2 * kGvStep, wc, xc);
    mma(wn, xn);
  }

  const int col = n0 + lr;
  if (col >= N) return;
  float* pp = part + (int64_t)blockIdx.y * M * N;
#pragma unroll
  for (int b = 0; b < MB; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 32 * b + 8 * (r >> 2) + 4 * lg + (r & 3);
      if (row < M) pp[(int64_t)row * N + col] = acc[b][r];
    }
}

// Reduce the split partials in order and apply the epilogue.
__global__ __launch_bounds__(256) void gemv_epi_kernel(const float* __restrict__ part,
                                                       int splits, int M, int N, Epi epi) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t MN = (int64_t)M * N;
  auto sum = [&](int row, int col) {
    float v = 0.f;
    for (int s = 0; s < splits; ++s) v += part[s * MN + (int64_t)row * N + col];
    return v;
  };
  if (epi.kind == EPI_STORE || epi.kind == EPI_RESID) {
    if (gid >= MN) return;
    const int row = (int)(gid / N), col = (int)(gid % N);
    float v = sum(row, col);
    if (epi.kind == EPI_RESID) v += bf2f(((const bf16*)epi.resid)[(int64_t)row * epi.ldr + col]);
    ((bf16*)epi.out)[(int64_t)row * epi.ldo + col] = f2bf(v);
  } else if (epi.kind == EPI_SWIGLU) {
    const int F = epi.ffn;
    if (gid >= (int64_t)M * F) return;
    const int row = (int)(gid / F), f = (int)(gid % F);
    const float g = sum(row, f), u = sum(row, F + f);
    ((bf16*)epi.out)[(int64_t)row * epi.ldo + f] = f2bf(silu(g) * u);
  } else {  // EPI_QKV: one thread per rotary pair
    const int D = epi.head_dim, half = D / 2;
    const int Hq = epi.n_q_heads, Hkv = epi.n_kv_heads;
    const int pairs = (Hq + 2 * Hkv) * half;
    if (gid >= (int64_t)M * pairs) return;
    const int row = (int)(gid / pairs), p = (int)(gid % pairs);
    const int head = p / half, d = p % half;
    const int col = head * D + d;
    float x1 = sum(row, col), x2 = sum(row, col + half);
    if (epi.bias) {
      x1 += bf2f(((const bf16*)epi.bias)[col]);
      x2 += bf2f(((const bf16*)epi.bias)[col + half]);
    }
    if (head < Hq + Hkv) {
      const float2 cs = epi.rope[(int64_t)row * half + d];
      const float y1 = x1 * cs.x - x2 * cs.y;
      const float y2 = x2 * cs.x + x1 * cs.y;
      x1 = y1;
      x2 = y2;
    }
    if (head < Hq) {
      bf16* qp = (bf16*)epi.q + ((int64_t)row * Hq + head) * D + d;
      qp[0] = f2bf(x1);
      qp[half] = f2bf(x2);
    } else {
      const int sl = epi.tok_slot[row];
      if (sl < 0) return;
      const int kvh = head < Hq + Hkv ? head - Hq : head - Hq - Hkv;
      bf16* cache = (bf16*)(head < Hq + Hkv ? epi.kc : epi.vc);
      bf16* cp = cache + (((int64_t)sl * Hkv + kvh) * epi.max_seq + epi.tok_row[row]) * D + d;
      cp[0] = f2bf(x1);
      cp[half] = f2bf(x2);
    }
  }
}

hipError_t launch_gemv(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                       const Epi& epi, float* part, hipStream_t s) {
  if (M == 0) return hipSuccess;
  const int splits = gemv_splits(M, N, K);
  const int steps = K / kGvStep;
  const int kper = cdiv(steps, splits) * kGvStep;
  dim3 grid(cdiv(N, kGvCols), splits);
  if (M <= 32)
    gemv_kernel<1><<<grid, 256, 0, s>>>((const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, kper, part);
  else if (M <= 64)
    gemv_kernel<2><<<grid, 256, 0, s>>>((const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, kper, part);
  else
    gemv_kernel<4><<<grid, 256, 0, s>>>((const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, kper, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int64_t n_out;
  if (epi.kind == EPI_SWIGLU) n_out = (int64_t)M * epi.ffn;
  else if (epi.kind == EPI_QKV) n_out = (int64_t)M * (epi.n_q_heads + 2 * epi.n_kv_heads) * (epi.head_dim / 2);
  else n_out = (int64_t)M * N;
  gemv_epi_kernel<<<(unsigned)((n_out + 255) / 256), 256, 0, s>>>(part, splits, M, N, epi);
  return hipGetLastError();
}

}  // namespace tri
