// Split-KV decode attention for sequences with one new token.
//
// Decode attention reads the whole KV cache of every sequence once per step
// and does ~1 flop per byte, so it is HBM-bound: the kernel is a stream of the
// cache through LDS with the arithmetic on the matrix cores.
//
// Grid: (key split, KV head, sequence); one wave per workgroup.  The key
// range [0, ctx + 1) of a (sequence, KV head) is cut into splits of
// `split_keys` so that the grid holds enough waves to keep every CU
// streaming; the wave serves all query heads of its KV head (grouped-query
// reuse: K and V are read once for the whole group).
//
// The split's keys move in tiles of 32 rows (K and V, contiguous in the cache)
// from HBM to a wave-private 3-stage LDS ring with buffer_load_dwordx4 ... lds;
// two tiles are in flight while one is consumed, and only the wave's own
// vmcnt orders them (no barrier).  Key rows past the sequence read as zero.
//
// Per tile, as in the prefill kernel with the group's heads as the query
// columns: S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (A = K rows from LDS,
// B = Q of the group's heads, lane column = head); online softmax per head in
// the log2 domain with a lazily raised max; O^T += V^T P^T with V^T read by
// ds_read_b64_tr_b16 and P split into bf16 hi + lo parts (16 significant
// bits).
//
// Output per (token, head, split): the unnormalised accumulator, the running
// max m (log2 domain) and sum l; the combine kernel merges the splits:
// M = max m_s, L = sum l_s 2^(m_s - M), o = sum acc_s 2^(m_s - M) / L.
#include "common.hpp"
#include "kernels.hpp"

namespace tri {

constexpr int kDecTile = 32;     // keys per tile
constexpr int kDecStages = 3;    // LDS ring depth
constexpr int kDecMinSplit = 128;

// Keys per split: the longest context cut into equal pieces of at most 512
// keys (a multiple of the 32-key tile), or of at most 128 when the grid would
// otherwise be small.
int attn_decode_split_keys(int n_seqs, int n_kv_heads, int max_kv) {
  if (max_kv < 1) max_kv = 1;
  const int64_t wgs = (int64_t)n_seqs * n_kv_heads * cdiv(max_kv, 512);
  const int cap = wgs >= 768 ? 512 : kDecMinSplit;
  const int ns = cdiv(max_kv, cap);
  return cdiv(cdiv(max_kv, ns), kDecTile) * kDecTile;
}

size_t attn_decode_partial_bytes(int n_tokens, int n_q_heads, int head_dim, int max_kv) {
  const int ns = cdiv(max_kv < 1 ? 1 : max_kv, kDecMinSplit);  // bound for every split size
  return (size_t)n_tokens * n_q_heads * ns * (head_dim + 2) * sizeof(float);
}

template <int D>
struct DecSmem {
  bf16 k[kDecStages][kDecTile * D];  // [key][d], chunks swizzled by kv_chunk
  bf16 v[kDecStages][kDecTile * D];
};

template <int D>
__global__ __launch_bounds__(64) void attn_decode_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ Kc, const bf16* __restrict__ Vc,
    float* __restrict__ part, const int32_t* __restrict__ cu_q,
    const int32_t* __restrict__ ctx_len, const int32_t* __restrict__ slot, int n_slots,
    int max_seq, int Hq, int Hkv, int nsplit, int split_keys, float scale_log2e, int n_tokens) {
  constexpr int DC = D / 8;                  // 16-byte chunks per row
  constexpr int TB = kDecTile * D * 2;       // bytes per K (or V) tile
  constexpr int BLK = TB / 1024;             // 1 KB loads per tile and operand
  constexpr int LPI = 2 * BLK;               // loads per tile
  constexpr int DS = D / 16, DB = D / 32;
  extern __shared__ __align__(16) char smem_raw[];
  DecSmem<D>& sm = *reinterpret_cast<DecSmem<D>*>(smem_raw);

  const int s = blockIdx.z, kvh = blockIdx.y, sp = blockIdx.x;
  const int t = cu_q[s];
  if (cu_q[s + 1] - t != 1 || t < 0 || t >= n_tokens) return;
  const int c = ctx_len[s], sl = slot[s];
  if (sl < 0 || sl >= n_slots || c < 0 || c + 1 > max_seq) return;
  const int k_begin = sp * split_keys;
  const int k_end = min(c + 1, k_begin + split_keys);
  if (k_begin >= k_end) return;
  const int nt = cdiv(k_end - k_begin, kDecTile);
  const int grp = Hq / Hkv;
  const int qh0 = kvh * grp;

  const int lane = threadIdx.x;
  const int r = lane & 31, g = lane >> 5;
  const int64_t cache_off = ((int64_t)sl * Hkv + kvh) * max_seq * D;
  // Rows at or past k_end read as zero.
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(Kc + cache_off), (short)0, k_end * D * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(Vc + cache_off), (short)0, k_end * D * 2, 0x00020000);
  // Lane l of 1 KB block b fills tile row b (64 / DC) + l / DC, physical
  // chunk l % DC = logical chunk kv_chunk(l % DC, row) (an involution).
  uint32_t ld_off[BLK];
#pragma unroll
  for (int j = 0; j < BLK; ++j) {
    const int row = j * (64 / DC) + lane / DC;
    ld_off[j] = (uint32_t)((row * D + kv_chunk<D>(lane % DC, row) * 8) * 2);
  }
  // Tile i (keys k_begin + 32 i ...) into stage i % 3; tiles past the split
  // are issued out of range (zero fill, no traffic) to keep the count uniform.
  auto issue = [&](int i) {
    const uint32_t kill = i < nt ? 0u : 0x80000000u;
    const uint32_t kb = (uint32_t)(k_begin + kDecTile * (i < nt ? i : 0)) * D * 2;
    const int st = i % kDecStages;
#pragma unroll
    for (int j = 0; j < BLK; ++j) {
      buffer_load_lds16(rk, &sm.k[st][j * 512], (ld_off[j] | kill) + kb, 0);
      buffer_load_lds16(rv, &sm.v[st][j * 512], (ld_off[j] | kill) + kb, 0);
    }
  };
  // Q of head column r, loaded before the tiles so the first wait covers it
  // too (heads past the group repeat the last one; their results are not
  // written).
  bf16x8 qf[DS];
  {
    const bf16* qp = Q + ((int64_t)t * Hq + qh0 + min(r, grp - 1)) * D + 8 * g;
#pragma unroll
    for (int k = 0; k < DS; ++k) qf[k] = *(const bf16x8*)(qp + 16 * k);
  }
  issue(0);
  issue(1);

  const int tr_key = 4 * g + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  f32x16 oacc[DB];
#pragma unroll
  for (int b = 0; b < DB; ++b) oacc[b] = f32x16{0.f};
  float m_run = -INFINITY, l_run = 0.f;  // running max in raw score units
  const float slack_raw = kSoftmaxSlack / scale_log2e;

  for (int i = 0; i < nt; ++i) {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPI) : "memory");  // tile i landed
    issue(i + 2);  // into the stage of tile i - 1, whose reads fed issued MFMAs
    const int st = i % kDecStages;
    const int key0 = k_begin + kDecTile * i;
    // S^T = K Q^T; element e: key key0 + 8 (e / 4) + 4 g + e % 4, head r.
    f32x16 sacc = f32x16{0.f};
#pragma unroll
    for (int k = 0; k < DS; ++k) {
      const bf16x8 kf = *(const bf16x8*)&sm.k[st][r * D + kv_chunk<D>(2 * k + g, r) * 8];
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[k], sacc, 0, 0, 0);
    }
    float mt = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = key0 + 8 * (e >> 2) + 4 * g + (e & 3);
      if (key >= k_end) sacc[e] = -INFINITY;
      mt = fmaxf(mt, sacc[e]);
    }
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    // Running max in raw score units, raised only past the slack (every tile
    // has a valid key, so m_run is finite after the first).
    const bool raise = mt > m_run + slack_raw;
    if (__builtin_amdgcn_ballot_w64(raise)) {
      const float m_new = raise ? mt : m_run;
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * scale_log2e);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int b = 0; b < DB; ++b) oacc[b] *= alpha;
    }
    const float mc = m_run * scale_log2e;
    bf16x8 pf[2], pl[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float p8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p8[e] = __builtin_amdgcn_exp2f(fmaf(sacc[8 * h + e], scale_log2e, -mc));
        l_run += p8[e];
      }
      split_hilo8(p8, pf[h], pl[h]);
    }
    // O^T += V^T P^T over the two 16-key groups of the tile.
    const bf16* vb = sm.v[st];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k1 = 16 * h + tr_key, k2 = k1 + 8;
#pragma unroll
      for (int b = 0; b < DB; ++b) {
        const int col = 32 * b + tr_col;
        union {
          s16x4 s[2];
          bf16x8 v;
        } vf;
        vf.s[0] = lds_read_tr16(vb + k1 * D + kv_chunk<D>(col >> 3, k1) * 8 + (col & 7));
        vf.s[1] = lds_read_tr16(vb + k2 * D + kv_chunk<D>(col >> 3, k2) * 8 + (col & 7));
        oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf.v, pf[h], oacc[b], 0, 0, 0);
        oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf.v, pl[h], oacc[b], 0, 0, 0);
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // no load may land in LDS after exit

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (r >= grp) return;
  float* pp = part + (((int64_t)t * Hq + qh0 + r) * nsplit + sp) * (D + 2);
  // oacc[b] element e: d = 32 b + 8 (e / 4) + 4 g + e % 4.
#pragma unroll
  for (int b = 0; b < DB; ++b)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
#pragma unroll
      for (int e = 0; e < 4; ++e) pp[32 * b + 8 * r4 + 4 * g + e] = oacc[b][4 * r4 + e];
    }
  if (g == 0) {
    pp[D] = m_run * scale_log2e;  // log2 domain for the combine
    pp[D + 1] = l_tot;
  }
}

// One workgroup of D threads per (sequence, query head).
template <int D>
__global__ __launch_bounds__(128) void attn_combine_kernel(
    const float* __restrict__ part, bf16* __restrict__ O, const int32_t* __restrict__ cu_q,
    const int32_t* __restrict__ ctx_len, const int32_t* __restrict__ slot, int n_slots,
    int max_seq, int Hq, int nsplit, int split_keys, int n_tokens) {
  const int s = blockIdx.x, qh = blockIdx.y, d = threadIdx.x;
  const int t = cu_q[s];
  if (cu_q[s + 1] - t != 1 || t < 0 || t >= n_tokens) return;
  const int c = ctx_len[s], sl = slot[s];
  if (sl < 0 || sl >= n_slots || c < 0 || c + 1 > max_seq) return;
  const int ns = min(cdiv(c + 1, split_keys), nsplit);  // never past the launched splits
  const float* pp = part + ((int64_t)t * Hq + qh) * nsplit * (D + 2);
  // Splits in groups of 8: the group's (m, l, acc) loads are issued together,
  // then folded in split order into a running (M, L, o).
  float M = -INFINITY, Lsum = 0.f, o = 0.f;
  for (int i0 = 0; i0 < ns; i0 += 8) {
    float m[8], l[8], a[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool ok = i0 + j < ns;
      const float* q = pp + (ok ? i0 + j : 0) * (D + 2);
      m[j] = ok ? q[D] : -INFINITY;
      l[j] = ok ? q[D + 1] : 0.f;
      a[j] = ok ? q[d] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (i0 + j >= ns) break;
      const float Mn = fmaxf(M, m[j]);
      const float sc = exp2f(M - Mn), w = exp2f(m[j] - Mn);
      Lsum = Lsum * sc + l[j] * w;
      o = o * sc + a[j] * w;
      M = Mn;
    }
  }
  O[((int64_t)t * Hq + qh) * D + d] = f2bf(o / Lsum);
}

template <int D>
static hipError_t run_decode(const void* q, const void* kc, const void* vc, float* part,
                             const BatchDev& b, int n_slots, int max_seq, int Hq, int Hkv,
                             hipStream_t s) {
  const int max_kv = b.max_ctx_len + 1;
  const int split = attn_decode_split_keys(b.n_seqs, Hkv, max_kv);
  const int nsplit = cdiv(max_kv, split);
  const float scale_log2e = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  dim3 grid(nsplit, Hkv, b.n_seqs);
  attn_decode_kernel<D><<<grid, 64, sizeof(DecSmem<D>), s>>>(
      (const bf16*)q, (const bf16*)kc, (const bf16*)vc, part, b.cu_q, b.ctx_len, b.slot, n_slots,
      max_seq, Hq, Hkv, nsplit, split, scale_log2e, b.n_tokens);
  return hipGetLastError();
}

hipError_t launch_attn_decode_split(const void* q, const void* kc, const void* vc, float* part,
                                    const BatchDev& b, int n_slots, int max_seq, int n_q_heads,
                                    int n_kv_heads, int head_dim, hipStream_t s) {
  if (b.n_seqs == 0) return hipSuccess;
  if (head_dim == 128)
    return run_decode<128>(q, kc, vc, part, b, n_slots, max_seq, n_q_heads, n_kv_heads, s);
  return run_decode<64>(q, kc, vc, part, b, n_slots, max_seq, n_q_heads, n_kv_heads, s);
}

hipError_t launch_attn_decode_combine(const float* part, void* out, const BatchDev& b,
                                      int n_slots, int max_seq, int n_q_heads, int n_kv_heads,
                                      int head_dim, hipStream_t s) {
  if (b.n_seqs == 0) return hipSuccess;
  const int max_kv = b.max_ctx_len + 1;
  const int split = attn_decode_split_keys(b.n_seqs, n_kv_heads, max_kv);
  const int nsplit = cdiv(max_kv, split);
  dim3 cgrid(b.n_seqs, n_q_heads);
  if (head_dim == 128)
    attn_combine_kernel<128><<<cgrid, 128, 0, s>>>(part, (bf16*)out, b.cu_q, b.ctx_len, b.slot,
                                                   n_slots, max_seq, n_q_heads, nsplit, split,
                                                   b.n_tokens);
  else
    attn_combine_kernel<64><<<cgrid, 64, 0, s>>>(part, (bf16*)out, b.cu_q, b.ctx_len, b.slot,
                                                 n_slots, max_seq, n_q_heads, nsplit, split,
                                                 b.n_tokens);
  return hipGetLastError();
}

}  // namespace tri
