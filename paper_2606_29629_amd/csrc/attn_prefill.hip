// Causal grouped-query flash attention for prefill and chunked prefill.
//
// One workgroup = one (sequence, query head, 128-query tile); 4 waves of 32
// queries.  Keys and values come from the KV cache (the q/k/v projection has
// already written this call's rows), 64 keys per tile, staged through LDS and
// double buffered; the next tile's global loads are issued before the current
// tile's MFMAs.
//
// The score block is computed transposed, S^T = K Q^T, with
// v_mfma_f32_32x32x16_bf16 (A = K rows from LDS, B = the wave's queries held in
// registers for the whole loop).  A lane then owns one query column and 32 of
// the tile's 64 keys, so the running max / sum of the online softmax need one
// cross-lane exchange (lane ^ 32) per tile.  The output is also kept
// transposed, O^T += V^T P^T: P^T is taken straight from the score
// accumulators, and V is written to LDS transposed with the keys of every
// 16-key group permuted to the order in which the score accumulator holds
// them, so each lane's 8 V^T values are one ds_read_b128.  The P V product runs
// on the fp16 matrix path (v_mfma_f32_32x32x16_f16, same rate as bf16): V
// converts from bf16 exactly in fp16's normal range, and P is split into
// P_hi = fp16(P) and P_lo = fp16(P - P_hi), two MFMAs into one accumulator,
// so P keeps ~22 significant bits and the weights match the fp32 row sum.
// Scores use exp2 with the 1/sqrt(D) * log2(e) scale folded in.
#include "common.hpp"
#include "kernels.hpp"

namespace tri {

constexpr int kFaBQ = 128;  // queries per workgroup
constexpr int kFaBK = 64;   // keys per tile

// Position inside a 16-key group at which key kk is stored in V^T (the order in
// which a score-accumulator lane holds keys: lane half g, element e <->
// key (e % 4) + 8 (e / 4) + 4 g).
__device__ __forceinline__ int vt_slot(int kk) {
  return 8 * ((kk >> 2) & 1) + (kk & 3) + 4 * (kk >> 3);
}

// Physical 16-byte chunk of logical chunk pc in V^T row d.  The (d % 8) term
// spreads the 8 lanes of a ds_read_b128 phase (consecutive d); the (d / 8)
// term spreads the transposing 2-byte stores (d = 8 ch + e, same e).
__device__ __forceinline__ int vt_chunk(int pc, int d) { return pc ^ (d & 7) ^ ((d >> 3) & 7); }

// K tile rows are D * 2 bytes.  With 64 four-byte banks, 16 lanes reading the
// same chunk of 16 consecutive keys are conflict-free when the chunk is
// XOR-ed with key % 16 (256-byte rows, D = 128) or with (key / 2) % 8
// (128-byte rows, D = 64).
template <int D>
__device__ __forceinline__ int k_chunk_t(int ch, int key) {
  return D == 128 ? (ch ^ (key & 15)) : (ch ^ ((key >> 1) & 7));
}
#define k_chunk(ch, key) k_chunk_t<D>(ch, key)

template <int D>
struct FaSmem {
  bf16 k[2][kFaBK * D];  // [key][d], 16-byte chunks swizzled by k_chunk
  f16 vt[2][D * kFaBK];  // V^T in fp16: [d][key slot], chunks swizzled by vt_chunk
};

template <int D>
__global__ __launch_bounds__(256) void attn_prefill_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ Kc, const bf16* __restrict__ Vc,
    bf16* __restrict__ O, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ ctx_len,
    const int32_t* __restrict__ slot, int n_slots, int max_seq, int Hq, int Hkv,
    float scale_log2e, int include_single, int n_tokens) {
  constexpr int DC = D / 8;             // 16-byte chunks per K row
  constexpr int KLD = kFaBK * DC / 256; // K chunks per thread per tile
  constexpr int DS = D / 16;            // MFMA k-steps over d
  constexpr int DB = D / 32;            // 32-row d blocks of O^T
  extern __shared__ __align__(16) char smem_raw[];
  FaSmem<D>& sm = *reinterpret_cast<FaSmem<D>*>(smem_raw);

  const int s = blockIdx.z, qh = blockIdx.y;
  const int q0 = cu_q[s], n = cu_q[s + 1] - q0;
  if (n <= 0 || (n == 1 && !include_single) || q0 < 0 || q0 + n > n_tokens) return;
  const int qt = (int)gridDim.x - 1 - (int)blockIdx.x;  // heavy (late) tiles first
  if (qt * kFaBQ >= n) return;
  const int c = ctx_len[s], sl = slot[s];
  if (sl < 0 || sl >= n_slots || c < 0 || c + n > max_seq) return;
  const int kvh = (qh * Hkv) / Hq;
  const int64_t cache_off = ((int64_t)sl * Hkv + kvh) * max_seq * D;
  const bf16* Kp = Kc + cache_off;
  const bf16* Vp = Vc + cache_off;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  const int kv_len = c + min(n, (qt + 1) * kFaBQ);
  const int nkt = cdiv(kv_len, kFaBK);

  // This lane's query (clamped to a valid row; rows >= n are not written).
  const int qi = qt * kFaBQ + wave * 32 + lr;
  const int qrow = q0 + min(qi, n - 1);
  const int qpos = c + qi;                 // cache row of this query
  const int wave_qmin = c + qt * kFaBQ + wave * 32;
  bf16x8 qf[DS];
  {
    const bf16* qp = Q + ((int64_t)qrow * Hq + qh) * D + 8 * lg;
#pragma unroll
    for (int t = 0; t < DS; ++t) qf[t] = *(const bf16x8*)(qp + 16 * t);
  }

  // Global -> register staging of one K/V tile.
  u32x4 rk[KLD], rv[KLD];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int id = tid + 256 * i, key = id / DC, ch = id % DC;
      const int kr = min(kt * kFaBK + key, kv_len - 1);
      rk[i] = ldg16(Kp + (int64_t)kr * D + ch * 8);
      rv[i] = ldg16(Vp + (int64_t)kr * D + ch * 8);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KLD; ++i) {
      const int id = tid + 256 * i, key = id / DC, ch = id % DC;
      *(u32x4*)&sm.k[buf][key * D + k_chunk(ch, key) * 8] = rk[i];
      Pack8 v;
      v.u = rv[i];
      const int slotk = (key & ~15) + vt_slot(key & 15);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = ch * 8 + e;
        sm.vt[buf][d * kFaBK + vt_chunk(slotk >> 3, d) * 8 + (slotk & 7)] = bf2h_sat(v.e[e]);
      }
    }
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int b = 0; b < DB; ++b) oacc[b] = f32x16{0.f};
  float m_run = -INFINITY, l_run = 0.f;

  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nkt) gload(kt + 1);
    const int key0 = kt * kFaBK;
    if (key0 <= wave_qmin + 31) {  // some key of this tile is visible to this wave
      // S^T = K Q^T for two 32-key blocks.
      f32x16 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        sacc[kb] = f32x16{0.f};
        const int key = kb * 32 + lr;
#pragma unroll
        for (int t = 0; t < DS; ++t) {
          const int ch = 2 * t + lg;
          const bf16x8 kf = *(const bf16x8*)&sm.k[buf][key * D + k_chunk(ch, key) * 8];
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[t], sacc[kb], 0, 0, 0);
        }
      }
      // Mask + scale; element r of block kb is key key0 + 32kb + (r%4) + 8(r/4) + 4lg.
      const bool diag = key0 + kFaBK - 1 > wave_qmin;
      float mt = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float v = sacc[kb][r] * scale_log2e;
          if (diag) {
            const int key = key0 + 32 * kb + (r & 3) + 8 * (r >> 2) + 4 * lg;
            if (key > qpos) v = -INFINITY;
          }
          sacc[kb][r] = v;
          mt = fmaxf(mt, v);
        }
      mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
      const float m_new = fmaxf(m_run, mt);
      // m_new is finite: key 0 of the first tile is visible to every query.
      const float alpha = exp2f(m_run - m_new);
      m_run = m_new;
      float ls = 0.f;
      f16x8 pf[4], pl[4];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float p = exp2f(sacc[kb][8 * h + e] - m_new);
            ls += p;
            const f16 hi = (f16)p;
            pf[2 * kb + h][e] = hi;
            pl[2 * kb + h][e] = (f16)(p - (float)hi);
          }
      l_run = l_run * alpha + ls;
#pragma unroll
      for (int b = 0; b < DB; ++b) oacc[b] *= alpha;
      // O^T += V^T P^T over four 16-key groups.
#pragma unroll
      for (int g16 = 0; g16 < 4; ++g16) {
        const int pc = 2 * g16 + lg;  // chunk of the key slots this lane feeds
#pragma unroll
        for (int b = 0; b < DB; ++b) {
          const int d = 32 * b + lr;
          const f16x8 vf = *(const f16x8*)&sm.vt[buf][d * kFaBK + vt_chunk(pc, d) * 8];
          oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pf[g16], oacc[b], 0, 0, 0);
          oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pl[g16], oacc[b], 0, 0, 0);
        }
      }
    }
    if (kt + 1 < nkt) sstore(buf ^ 1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (qi >= n) return;
  const float inv = 1.0f / l_tot;
  bf16* op = O + ((int64_t)(q0 + qi) * Hq + qh) * D;
  // oacc[b] element r: d = 32b + 8(r/4) + 4lg + r%4  -> 4 consecutive d per (r/4).
#pragma unroll
  for (int b = 0; b < DB; ++b)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      bf16x4 o4;
#pragma unroll
      for (int e = 0; e < 4; ++e) o4[e] = f2bf(oacc[b][4 * r4 + e] * inv);
      *(bf16x4*)(op + 32 * b + 8 * r4 + 4 * lg) = o4;
    }
}

template <int D>
static hipError_t run_fa(const void* q, const void* kc, const void* vc, void* out,
                         const BatchDev& b, int n_slots, int max_seq, int Hq, int Hkv,
                         int include_single, hipStream_t s) {
  const size_t smem = sizeof(FaSmem<D>);
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)attn_prefill_kernel<D>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    attr = true;
  }
  dim3 grid(cdiv(b.max_q_len, kFaBQ), Hq, b.n_seqs);
  const float scale_log2e = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  attn_prefill_kernel<D><<<grid, 256, smem, s>>>((const bf16*)q, (const bf16*)kc, (const bf16*)vc,
                                                 (bf16*)out, b.cu_q, b.ctx_len, b.slot, n_slots,
                                                 max_seq, Hq, Hkv, scale_log2e, include_single, b.n_tokens);
  return hipGetLastError();
}

hipError_t launch_attn_prefill(const void* q, const void* kc, const void* vc, void* out,
                               const BatchDev& b, int n_slots, int max_seq, int n_q_heads,
                               int n_kv_heads, int head_dim, int include_single, hipStream_t s) {
  if (b.n_seqs == 0 || b.max_q_len == 0) return hipSuccess;
  if (head_dim == 128)
    return run_fa<128>(q, kc, vc, out, b, n_slots, max_seq, n_q_heads, n_kv_heads,
                       include_single, s);
  return run_fa<64>(q, kc, vc, out, b, n_slots, max_seq, n_q_heads, n_kv_heads, include_single,
                    s);
}

}  // namespace tri
