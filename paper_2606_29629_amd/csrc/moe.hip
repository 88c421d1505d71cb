// Mixture-of-experts routing, permutation and combine.
//
// Router: logits = h W_r^T accumulated in fp32, softmax over all experts,
// top-k by logit with ties to the lower expert index, weights p[idx]
// (renormalised over the k chosen when asked).  Inside the layer (bf16 h2) the
// logits come from the matrix cores as split-K planes summed in a fixed order;
// the fp32-input entry point uses a VALU kernel with a fixed summation order.
//
// Permutation (a counting sort, deterministic): for every expert e, one
// workgroup scans the (token, slot) pairs in order and ranks the pairs routed
// to e with wave ballots; a second kernel turns counts into segment offsets
// (routed order = by expert, then by pair index) and per-expert M-tile offsets
// for the grouped GEMM, and scatters perm[pos] = pair, inv[pair] = pos.
//
// Combine: out[t] = bf16(x1[t] + sum_j w[t][j] * y[inv[t k + j]]), j in order.
#include "common.hpp"
#include "kernels.hpp"

namespace tri {

constexpr int kRouteTok = 8;     // tokens per router workgroup
constexpr int kMaxPlanes = 16;   // split-K planes of the router logits, at most
constexpr int kRouteChunk = 1024;  // hidden columns staged per pass

template <typename InT>
__device__ __forceinline__ float to_f32(InT v) { return (float)v; }

// Top-k of one token's logits (lane holds experts lane + 64 q, q < 4; -inf
// past E) with ties to the lower expert index, then the softmax weights of the
// chosen experts (over all experts, or renormalised over the k chosen).
// Selection s is kept by lane s, which writes slot s of idx / w.
__device__ __forceinline__ void route_topk(const float (&vin)[4], int E, int k, int renorm,
                                           int lane, int32_t* __restrict__ idx,
                                           float* __restrict__ w) {
  float v[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) v[q] = vin[q];
  float my_v = -INFINITY;
  int my_i = 0;
  for (int s = 0; s < k; ++s) {
    // this lane's best (highest value, then lowest expert index)
    float bv = v[0];
    int bi = lane;
#pragma unroll
    for (int q = 1; q < 4; ++q) {
      const int e = lane + 64 * q;
      if (v[q] > bv) { bv = v[q]; bi = e; }
    }
    if (bv == -INFINITY) bi = 0x7fffffff;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
    }
    if (lane == s) { my_v = bv; my_i = bi; }
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (lane + 64 * q == bi) v[q] = -INFINITY;
  }
  const float m = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                                __builtin_bit_cast(int, my_v)));
  float z = 0.f;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (lane + 64 * q < E) z += expf(vin[q] - m);
  z = wave_sum(z);
  const float p = expf(my_v - m);
  float zk = 0.f;  // the k chosen weights summed in selection order
  for (int s = 0; s < k; ++s)
    zk += __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, p), s));
  if (lane < k) {
    idx[lane] = my_i;
    w[lane] = renorm ? p / zk : p / z;
  }
}

// Eight router weights of one row as fp32 (bf16 or fp32 storage).
__device__ __forceinline__ void load_w8(const bf16* p, float (&w)[8]) {
  Pack8 v;
  v.u = ldg16(p);
#pragma unroll
  for (int q = 0; q < 8; ++q) w[q] = bf2f(v.e[q]);
}
__device__ __forceinline__ void load_w8(const float* p, float (&w)[8]) {
  const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    w[q] = a[q];
    w[q + 4] = b[q];
  }
}

template <typename InT, typename WT = bf16>
__global__ __launch_bounds__(256) void moe_router_kernel(const InT* __restrict__ h,
                                                         const WT* __restrict__ wr, int T, int H,
                                                         int E, int k, int renorm,
                                                         int32_t* __restrict__ idx_out,
                                                         float* __restrict__ w_out) {
  __shared__ __align__(16) float hs[kRouteTok][kRouteChunk];
  __shared__ float logit[kRouteTok][256];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * kRouteTok;
  const int el = tid & 127, tg = tid >> 7;  // expert within group; tokens 4 tg .. 4 tg + 3
  for (int eb = 0; eb < E; eb += 128) {
    const int e = eb + el;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int hc = 0; hc < H; hc += kRouteChunk) {
      const int hn = min(kRouteChunk, H - hc);
      __syncthreads();
      for (int i = tid; i < kRouteTok * kRouteChunk; i += 256) {
        const int r = i / kRouteChunk, c = i % kRouteChunk;
        hs[r][c] = (t0 + r < T && c < hn) ? to_f32(h[(int64_t)(t0 + r) * H + hc + c]) : 0.f;
      }
      __syncthreads();
      if (e < E) {
        const WT* wrow = wr + (int64_t)e * H + hc;
        for (int j = 0; j < hn; j += 8) {
          float w8[8];
          load_w8(wrow + j, w8);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float* hp = &hs[4 * tg + i][j];
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[i] = fmaf(w8[q], hp[q], acc[i]);
          }
        }
      }
    }
    if (e < E)
#pragma unroll
      for (int i = 0; i < 4; ++i) logit[4 * tg + i][e] = acc[i];
  }
  __syncthreads();

  // Top-k and softmax weights: wave w handles tokens 2w and 2w + 1.
  for (int tt = 0; tt < 2; ++tt) {
    const int r = 2 * wave + tt, t = t0 + r;
    if (t >= T) break;
    float v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + 64 * q;
      v[q] = e < E ? logit[r][e] : -INFINITY;
    }
    route_topk(v, E, k, renorm, lane, idx_out + (int64_t)t * k, w_out + (int64_t)t * k);
  }
}

// Router on the matrix cores: the logits arrive as split-K planes
// [S][T][E] (fp32, from a bf16 GEMM of h2 and W_r with fp32 accumulation);
// they are summed in plane order (deterministic) before top-k.  One wave per
// token.
__global__ __launch_bounds__(256) void moe_topk_kernel(const float* __restrict__ planes, int S,
                                                       int T, int E, int k, int renorm,
                                                       int32_t* __restrict__ idx_out,
                                                       float* __restrict__ w_out) {
  const int lane = threadIdx.x & 63, t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  // Every plane's value is loaded before the ordered sum (S <= kMaxPlanes),
  // so the loads are in flight together; planes past S and experts past E
  // re-read an in-range address and are dropped.
  const float* base = planes + (int64_t)t * E;
  const int64_t plane = (int64_t)T * E;
  float pv[4][kMaxPlanes];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = min(lane + 64 * q, E - 1);
#pragma unroll
    for (int sp = 0; sp < kMaxPlanes; ++sp)
      pv[q][sp] = 64 * q < E ? base[min(sp, S - 1) * plane + e] : 0.f;  // (E is uniform)
  }
  float v[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float a = 0.f;
#pragma unroll
    for (int sp = 0; sp < kMaxPlanes; ++sp)
      if (sp < S) a += pv[q][sp];
    v[q] = lane + 64 * q < E ? a : -INFINITY;
  }
  route_topk(v, E, k, renorm, lane, idx_out + (int64_t)t * k, w_out + (int64_t)t * k);
}

hipError_t launch_moe_route_f32(const float* h32, const void* w_router, int T, int H, int E,
                                int k, int renorm, int32_t* idx, float* w, hipStream_t s,
                                bool w_f32) {
  if (T == 0) return hipSuccess;
  if (w_f32)
    moe_router_kernel<float, float><<<cdiv(T, kRouteTok), 256, 0, s>>>(
        h32, (const float*)w_router, T, H, E, k, renorm, idx, w);
  else
    moe_router_kernel<float><<<cdiv(T, kRouteTok), 256, 0, s>>>(h32, (const bf16*)w_router, T, H,
                                                                 E, k, renorm, idx, w);
  return hipGetLastError();
}

size_t moe_route_planes_bytes(int T, int H, int E) {
  return (size_t)gemm_planes_splits(T, E, H) * T * E * sizeof(float);
}

hipError_t launch_moe_route_bf16(const void* h, const void* w_router, int T, int H, int E, int k,
                                 int renorm, float* planes, int32_t* idx, float* w, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int S = gemm_planes_splits(T, E, H);
  if (S > kMaxPlanes) return hipErrorInvalidValue;
  hipError_t e = launch_gemm_planes(h, H, w_router, H, T, E, H, planes, S, s);
  if (e != hipSuccess) return e;
  moe_topk_kernel<<<cdiv(T, 4), 256, 0, s>>>(planes, S, T, E, k, renorm, idx, w);
  return hipGetLastError();
}

// One workgroup per expert: rank of every pair routed to it, in pair order.
// The pairs are scanned U x (64 NW) at a time: the loads of a batch are
// issued together and one barrier per batch publishes the waves' counts.  A
// workgroup's batches run one after another, so long pair lists (a
// prefill's) take 16 waves per workgroup and short ones (decode) 4; the
// 16-wave form unrolls 8 deep, which keeps its per-wave counts in registers.
constexpr int kCountUnroll = 16;

template <int NW, int U = (NW > 4 ? 8 : kCountUnroll)>
__global__ __launch_bounds__(NW * 64) void moe_count_kernel(const int32_t* __restrict__ idx,
                                                            int n_pairs,
                                                            int32_t* __restrict__ rank,
                                                            int32_t* __restrict__ counts) {
  constexpr int NT = NW * 64;
  __shared__ int wsum[2][U][NW];
  const int e = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const unsigned long long below = (1ull << lane) - 1ull;
  int base = 0, buf = 0;
  for (int p0 = 0; p0 < n_pairs; p0 += NT * U, buf ^= 1) {
    bool f[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int p = p0 + NT * u + tid;
      const int v = idx[min(p, n_pairs - 1)];  // clamped: no branch around the load
      f[u] = p < n_pairs && v == e;
    }
    int within[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const unsigned long long m = __ballot(f[u]);
      within[u] = __popcll(m & below);
      if (lane == 0) wsum[buf][u][wave] = __popcll(m);
    }
    // double-buffered counts: one barrier per batch suffices
    __syncthreads();
    int run = base;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      int pre = 0, tot = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        pre += w < wave ? wsum[buf][u][w] : 0;
        tot += wsum[buf][u][w];
      }
      if (f[u]) rank[p0 + NT * u + tid] = run + pre + within[u];
      run += tot;
    }
    base = run;
  }
  if (tid == 0) counts[e] = base;
}

// Segment offsets, M-tile offsets (tiles of bm rows) and the scatter.
__global__ __launch_bounds__(256) void moe_scatter_kernel(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ rank,
    const int32_t* __restrict__ counts, int n_pairs, int E, int bm, int32_t* __restrict__ perm,
    int32_t* __restrict__ inv, int32_t* __restrict__ seg, int32_t* __restrict__ tile_off) {
  __shared__ int off[257], toff[257];
  const int tid = threadIdx.x;
  // exclusive scans of the counts and tile counts over the E <= 256 experts:
  // one thread per expert, Hillis-Steele in LDS
  const int c = tid < E ? counts[tid] : 0;
  off[tid + 1] = c;
  toff[tid + 1] = cdiv(c, bm);
  if (tid == 0) off[0] = toff[0] = 0;
  __syncthreads();
  for (int d = 1; d < 256; d <<= 1) {
    const int a = tid + 1 - d >= 1 ? off[tid + 1 - d] : 0;
    const int b = tid + 1 - d >= 1 ? toff[tid + 1 - d] : 0;
    __syncthreads();
    off[tid + 1] += a;
    toff[tid + 1] += b;
    __syncthreads();
  }
  if (blockIdx.x == 0)
    for (int i = tid; i <= E; i += 256) {
      seg[i] = off[i];
      tile_off[i] = toff[i];
    }
  const int p = blockIdx.x * 256 + tid;
  if (p < n_pairs) {
    const int pos = off[idx[p]] + rank[p];
    perm[pos] = p;
    inv[p] = pos;
  }
}

hipError_t launch_moe_permute(const int32_t* idx, int n_pairs, int E, int bm, int32_t* rank,
                              int32_t* counts, int32_t* perm, int32_t* inv, int32_t* seg,
                              int32_t* tile_off, hipStream_t s) {
  if (n_pairs == 0) return hipSuccess;
  if (n_pairs > 256 * kCountUnroll)
    moe_count_kernel<16><<<E, 1024, 0, s>>>(idx, n_pairs, rank, counts);
  else
    moe_count_kernel<4><<<E, 256, 0, s>>>(idx, n_pairs, rank, counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  moe_scatter_kernel<<<cdiv(n_pairs, 256), 256, 0, s>>>(idx, rank, counts, n_pairs, E, bm, perm,
                                                        inv, seg, tile_off);
  return hipGetLastError();
}

// out[t] = x1[t] + sum_j w[t][j] y[inv[t k + j]], 8 columns per thread; x1
// and out in the storage type (bf16, or fp32 with F32).
template <bool F32>
__global__ __launch_bounds__(256) void moe_combine_kernel(const void* __restrict__ x1,
                                                          const float* __restrict__ y,
                                                          const int32_t* __restrict__ inv,
                                                          const float* __restrict__ w, int T,
                                                          int H, int k, void* __restrict__ out) {
  const int t = blockIdx.x;
  for (int c = threadIdx.x * 8; c < H; c += 256 * 8) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
      const float wj = w[(int64_t)t * k + j];
      const float* yp = y + (int64_t)inv[(int64_t)t * k + j] * H + c;
      const f32x4 a = *(const f32x4*)yp, b = *(const f32x4*)(yp + 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[q] = fmaf(wj, a[q], acc[q]);
        acc[q + 4] = fmaf(wj, b[q], acc[q + 4]);
      }
    }
    const int64_t at = (int64_t)t * H + c;
    if constexpr (F32) {
      const f32x4 xa = *(const f32x4*)((const float*)x1 + at);
      const f32x4 xb = *(const f32x4*)((const float*)x1 + at + 4);
      *(f32x4*)((float*)out + at) = f32x4{xa[0] + acc[0], xa[1] + acc[1], xa[2] + acc[2],
                                          xa[3] + acc[3]};
      *(f32x4*)((float*)out + at + 4) = f32x4{xb[0] + acc[4], xb[1] + acc[5], xb[2] + acc[6],
                                              xb[3] + acc[7]};
    } else {
      Pack8 xv, o;
      xv.u = ldg16((const bf16*)x1 + at);
#pragma unroll
      for (int q = 0; q < 8; ++q) o.e[q] = f2bf(bf2f(xv.e[q]) + acc[q]);
      stg16((bf16*)out + at, o.u);
    }
  }
}

hipError_t launch_moe_combine(const void* x1, const float* y, const int32_t* inv, const float* w,
                              int T, int H, int k, void* out, hipStream_t s, bool f32) {
  if (T == 0) return hipSuccess;
  if (f32)
    moe_combine_kernel<true><<<T, 256, 0, s>>>(x1, y, inv, w, T, H, k, out);
  else
    moe_combine_kernel<false><<<T, 256, 0, s>>>(x1, y, inv, w, T, H, k, out);
  return hipGetLastError();
}

}  // namespace tri
