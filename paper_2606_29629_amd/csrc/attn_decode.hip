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
// The split's keys move in tiles of 32 rows (K and V, contiguous in the
// cache), two tiles in flight while one is consumed, ordered only by the
// wave's own vmcnt (no barrier).  K goes straight from HBM to registers, in
// the MFMA operand layout (lane: key l % 32, 8 head-dim values of slice
// l / 32); V goes to a wave-private 3-stage LDS ring with buffer_load_dwordx4
// ... lds, because its operand must be transposed.  Keeping K out of LDS
// halves the LDS per wave, so twice the waves -- and twice the bytes in
// flight -- fit on a CU.  Key rows past the sequence read as zero.
//
// Per tile, as in the prefill kernel with the group's heads as the query
// columns: S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (A = K rows, B = Q of
// the group's heads, lane column = head); online softmax per head in
// the log2 domain with a lazily raised max; O^T += V^T P^T with V^T read by
// ds_read_b64_tr_b16 and P split into bf16 hi + lo parts (16 significant
// bits).
//
// Output per (sequence, head, split): the unnormalised accumulator, the running
// max m (log2 domain) and sum l; the combine kernel merges the splits:
// M = max m_s, L = sum l_s 2^(m_s - M), o = sum acc_s 2^(m_s - M) / L.
#include "common.hpp"
#include "kernels.hpp"

namespace tri {

constexpr int kDecTile = 32;     // keys per tile
constexpr int kDecStages = 3;    // LDS ring depth
constexpr int kDecMinSplit = 128;

// Waves of this kernel resident on one CU: the LDS (V ring + staged Q) and
// the register file (two waves per SIMD for D = 128, three for D = 64) bound it.
static int decode_waves_per_cu(int head_dim, int group) {
  const int smem = (head_dim == 128 ? kDecStages * kDecTile * 128 * 2 : kDecStages * kDecTile * 64 * 2) +
                   cdiv(group, 512 / head_dim) * 1024;
  const int by_lds = (160 * 1024) / smem;
  const int by_regs = head_dim == 128 ? 8 : 12;
  return by_lds < by_regs ? by_lds : by_regs;
}

// Keys per split: every (sequence, KV head) is cut into the same number of
// splits, as many as make the grid one full round of resident waves (each
// wave then streams from launch to finish with no second round), but no
// split shorter than kDecMinSplit keys; the split is a multiple of the
// 32-key tile.
int attn_decode_split_keys(int n_seqs, int n_kv_heads, int max_kv, int head_dim, int group,
                           int max_split) {
  if (max_kv < 1) max_kv = 1;
  const int64_t pairs = (int64_t)(n_seqs > 0 ? n_seqs : 1) * (n_kv_heads > 0 ? n_kv_heads : 1);
  const int64_t resident = (int64_t)decode_waves_per_cu(head_dim, group) * cu_count();
  int64_t ns = resident / pairs;
  if (ns < 1) ns = 1;
  if (ns > cdiv(max_kv, kDecMinSplit)) ns = cdiv(max_kv, kDecMinSplit);
  int split = cdiv(cdiv(max_kv, (int)ns), kDecTile) * kDecTile;
  if (max_split > 0 && split > max_split) split = max_split / kDecTile * kDecTile;
  return split;
}

// A split of a paged cache spans at most 64 blocks (one per lane of its
// block-id register): splits of up to 62 blocks.
int attn_decode_max_split(const KvDev& kv) { return kv.table ? 62 * kv.block_size : 0; }

// Partials of one (sequence, query head, split): D accumulators, max and sum.
// Indexed by sequence, so only the batch's sequences (not its tokens) count.
size_t attn_decode_partial_bytes(int n_seqs, int n_q_heads, int head_dim, int max_kv) {
  const int ns = cdiv(max_kv < 1 ? 1 : max_kv, kDecMinSplit);  // bound for every split size
  return (size_t)n_seqs * n_q_heads * ns * (head_dim + 2) * sizeof(float);
}

template <int D>
struct DecSmem {
  bf16 v[kDecStages][kDecTile * D];  // [key][d], chunks swizzled by kv_chunk
};

template <int N>
struct IntC {
  static constexpr int value = N;
};

__device__ __forceinline__ uint32_t lds_addr(const bf16* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) bf16*)p;
}

// Four 16-byte LDS reads, then an LDS wait, in one asm block (outside the
// compiler's LDS-fill tracking; the caller orders them after the fill).
__device__ __forceinline__ void lds_read_b128_x4(const uint32_t* a, bf16x8 (&v)[4]) {
  asm volatile(
      "ds_read_b128 %0, %4\n\t"
      "ds_read_b128 %1, %5\n\t"
      "ds_read_b128 %2, %6\n\t"
      "ds_read_b128 %3, %7\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3])
      : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]));
}

// 2 * DB transposing reads (ds_read_b64_tr_b16, see lds_read_tr16) into DB
// MFMA operands (reads 2b and 2b + 1 form operand b), then an LDS wait.
template <int DB>
__device__ __forceinline__ void lds_read_tr16_group(const uint32_t (&a)[2 * DB], bf16x8 (&v)[DB]) {
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
  u32x2 o[2 * DB];
  if constexpr (DB == 4) {
    asm volatile(
        "ds_read_b64_tr_b16 %0, %8\n\t"
        "ds_read_b64_tr_b16 %1, %9\n\t"
        "ds_read_b64_tr_b16 %2, %10\n\t"
        "ds_read_b64_tr_b16 %3, %11\n\t"
        "ds_read_b64_tr_b16 %4, %12\n\t"
        "ds_read_b64_tr_b16 %5, %13\n\t"
        "ds_read_b64_tr_b16 %6, %14\n\t"
        "ds_read_b64_tr_b16 %7, %15\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]),
          "=&v"(o[6]), "=&v"(o[7])
        : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]),
          "v"(a[7]));
  } else {
    static_assert(DB == 2, "head_dim 64 or 128");
    asm volatile(
        "ds_read_b64_tr_b16 %0, %4\n\t"
        "ds_read_b64_tr_b16 %1, %5\n\t"
        "ds_read_b64_tr_b16 %2, %6\n\t"
        "ds_read_b64_tr_b16 %3, %7\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3])
        : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]));
  }
#pragma unroll
  for (int b = 0; b < DB; ++b) {
    union {
      u32x2 s[2];
      bf16x8 v;
    } u;
    u.s[0] = o[2 * b];
    u.s[1] = o[2 * b + 1];
    v[b] = u.v;
  }
}

template <int D, bool PAGED>
__global__ __launch_bounds__(64, 2) void attn_decode_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ Kc, const bf16* __restrict__ Vc,
    float* __restrict__ part, const int32_t* __restrict__ cu_q,
    const int32_t* __restrict__ ctx_len, const int32_t* __restrict__ slot, KvDev kv, int Hq,
    int Hkv, int nsplit, int split_keys, float scale_log2e, int n_tokens) {
  constexpr int DC = D / 8;                  // 16-byte chunks per row
  constexpr int TB = kDecTile * D * 2;       // bytes per K (or V) tile
  constexpr int BLK = TB / 1024;             // 1 KB loads per V tile
  constexpr int DS = D / 16, DB = D / 32;
  constexpr int LPI = BLK + DS;              // loads per tile (V to LDS, K to registers)
  extern __shared__ __align__(16) char smem_raw[];
  DecSmem<D>& sm = *reinterpret_cast<DecSmem<D>*>(smem_raw);

  const int s = blockIdx.z, kvh = blockIdx.y, sp = blockIdx.x;
  // The sequence's scalars in one round trip (s < n_seqs by the grid).
  const int t = cu_q[s], t1 = cu_q[s + 1], c = ctx_len[s], sl = slot[s];
  if (t1 - t != 1 || t < 0 || t >= n_tokens) return;
  if (sl < 0 || sl >= kv.n_slots || c < 0 || c + 1 > kv.max_seq) return;
  const int k_begin = sp * split_keys;
  const int k_end = min(c + 1, k_begin + split_keys);
  if (k_begin >= k_end) return;
  const int nt = cdiv(k_end - k_begin, kDecTile);
  const int grp = Hq / Hkv;
  const int qh0 = kvh * grp;

  const int lane = threadIdx.x;
  const int r = lane & 31, g = lane >> 5;
  // Paged cache: lane j holds the pool block of the split's j-th block (the
  // split spans at most 64 blocks), -1 for an entry outside the pool.
  const int prows = PAGED ? kv.block_size : kv.max_seq;
  const int jb0 = PAGED ? k_begin / kv.block_size : 0;
  int tbl = -1;
  if (PAGED) {
    const int nblk = (k_end - 1) / kv.block_size - jb0 + 1;
    if (lane < nblk) {
      const int blk = kv.table[(int64_t)sl * kv.blocks_per_slot() + jb0 + lane];
      tbl = (blk >= 0 && blk < kv.n_blocks) ? blk : -1;
    }
  }
  // The loop's tile i is the split's tile (i + rot) mod nt: the waves of one
  // split index start at different tiles, so the grid does not read every
  // (sequence, head) region at the same offset at once.  Tiles past the
  // split stay past it (empty).
  const int rot = (int)(((unsigned)s * 7u + (unsigned)kvh * 3u) % (unsigned)nt);
  auto phys = [&](int i) {
    const int j = i + rot;
    return i < nt ? (j >= nt ? j - nt : j) : i;
  };
  // Buffer descriptor of tile i's rows of one cache operand: keys past the
  // sequence, tiles past the split and blocks outside the pool read as zero.
  auto tile_rsrc = [&](const bf16* base, int i) {
    const int key0 = k_begin + kDecTile * phys(i);
    int panel = sl, prow = key0, rows = 0;
    if (i < nt) {
      rows = min(kDecTile, k_end - key0);
      if (PAGED) {
        const int j = key0 / kv.block_size;
        panel = __builtin_amdgcn_readlane(tbl, j - jb0);
        prow = key0 - j * kv.block_size;
        if (panel < 0) rows = 0;
      }
    }
    if (rows == 0) panel = prow = 0;
    return __builtin_amdgcn_make_buffer_rsrc(
        (void*)(base + (((int64_t)panel * Hkv + kvh) * prows + prow) * D), (short)0,
        rows * D * 2, 0x00020000);
  };
  // V: lane l of 1 KB block b fills tile row b (64 / DC) + l / DC, physical
  // chunk l % DC = logical chunk kv_chunk(l % DC, row) (an involution).
  uint32_t ld_off[BLK];
#pragma unroll
  for (int j = 0; j < BLK; ++j) {
    const int row = j * (64 / DC) + lane / DC;
    ld_off[j] = (uint32_t)((row * D + kv_chunk<D>(lane % DC, row) * 8) * 2);
  }
  // K: k-step k of lane (r, g) is key r, logical chunk 2 k + g.
  uint32_t k_off[DS];
#pragma unroll
  for (int k = 0; k < DS; ++k) k_off[k] = (uint32_t)((r * D + (2 * k + g) * 8) * 2);
  // Tile i = keys k_begin + 32 i ...; tiles past the split are issued with an
  // empty descriptor (zero fill, no traffic) to keep the load count uniform.
  auto issue_v = [&](int i) {
    const __amdgpu_buffer_rsrc_t rv = tile_rsrc(Vc, i);
    const int st = i % kDecStages;
#pragma unroll
    for (int j = 0; j < BLK; ++j) buffer_load_lds16(rv, &sm.v[st][j * 512], ld_off[j], 0);
  };
  bf16x8 kreg[2][DS];  // K of tile i in slot i % 2
  auto issue_k = [&](auto slot, int i) {
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(Kc, i);
#pragma unroll
    for (int k = 0; k < DS; ++k)
      kreg[decltype(slot)::value][k] =
          __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rk, k_off[k], 0, 0));
  };
  // Q of the group's heads, staged once in LDS after the V ring ([grp][D],
  // chunks swizzled like the K/V tiles so the per-tile fragment reads are
  // conflict-free) by direct loads issued ahead of the tiles, so the first
  // tile wait covers them; head column r >= grp repeats the last head (its
  // results are not written).
  constexpr int RPB = 64 / DC;  // rows per 1 KB load
  bf16* qs = reinterpret_cast<bf16*>(smem_raw + sizeof(DecSmem<D>));
  {
    const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(Q + ((int64_t)t * Hq + qh0) * D), (short)0, grp * D * 2, 0x00020000);
    for (int j = 0; j < cdiv(grp, RPB); ++j) {
      const int row = j * RPB + lane / DC;
      buffer_load_lds16(rq, &qs[j * 512],
                        (uint32_t)((row * D + kv_chunk<D>(lane % DC, row) * 8) * 2), 0);
    }
  }
  const int qrow = min(r, grp - 1);
  uint32_t q_addr[DS];
#pragma unroll
  for (int k = 0; k < DS; ++k) q_addr[k] = lds_addr(&qs[qrow * D + kv_chunk<D>(2 * k + g, qrow) * 8]);
  // Issue order per tile: V (to LDS), then K (to registers); both of tile i
  // have landed once at most the LPI loads of tile i + 1 are outstanding.
  issue_v(0);
  issue_k(IntC<0>{}, 0);
  issue_v(1);
  issue_k(IntC<1>{}, 1);

  const int tr_key = 4 * g + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  f32x16 oacc[DB];
#pragma unroll
  for (int b = 0; b < DB; ++b) oacc[b] = f32x16{0.f};
  float m_run = -INFINITY, l_run = 0.f;  // running max in raw score units
  const float slack_raw = kSoftmaxSlack / scale_log2e;

  auto step = [&](auto slot, int i) {
    constexpr int ks = decltype(slot)::value;
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPI) : "memory");  // tile i landed
    issue_v(i + 2);  // into the stage of tile i - 1, whose reads fed issued MFMAs
    const int st = i % kDecStages;
    const int key0 = k_begin + kDecTile * phys(i);
    // S^T = K Q^T; element e: key key0 + 8 (e / 4) + 4 g + e % 4, head r.
    f32x16 sacc = f32x16{0.f};
#pragma unroll
    for (int k0 = 0; k0 < DS; k0 += 4) {
      bf16x8 qf[4];
      lds_read_b128_x4(&q_addr[k0], qf);
#pragma unroll
      for (int k = 0; k < 4; ++k)
        sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kreg[ks][k0 + k], qf[k], sacc, 0, 0, 0);
    }
    issue_k(slot, i + 2);  // the slot's K has been read by the MFMAs above
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
    // O^T += V^T P^T over the two 16-key groups of the tile.  The
    // transposing reads of a group are issued together and waited for in one
    // asm block: the wave's own top-of-step vmcnt wait already orders them
    // after the tile's LDS fill, and keeping them out of the compiler's view
    // stops it from also waiting for the fills of later tiles.
    const bf16* vb = sm.v[st];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k1 = 16 * h + tr_key, k2 = k1 + 8;
      uint32_t a[2 * DB];
#pragma unroll
      for (int b = 0; b < DB; ++b) {
        const int col = 32 * b + tr_col;
        a[2 * b] = lds_addr(vb + k1 * D + kv_chunk<D>(col >> 3, k1) * 8 + (col & 7));
        a[2 * b + 1] = lds_addr(vb + k2 * D + kv_chunk<D>(col >> 3, k2) * 8 + (col & 7));
      }
      bf16x8 vf[DB];
      lds_read_tr16_group<DB>(a, vf);
#pragma unroll
      for (int b = 0; b < DB; ++b) {
        oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[b], pf[h], oacc[b], 0, 0, 0);
        oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[b], pl[h], oacc[b], 0, 0, 0);
      }
    }
  };
  // Both steps of the loop body are unconditional, so the compiler's own
  // waits for the K registers see exactly two tiles of loads after them.
  int i = 0;
  for (; i + 1 < nt; i += 2) {
    step(IntC<0>{}, i);
    step(IntC<1>{}, i + 1);
  }
  if (i < nt) step(IntC<0>{}, i);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // no load may land after exit

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (r >= grp) return;
  float* pp = part + (((int64_t)s * Hq + qh0 + r) * nsplit + sp) * (D + 2);
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
  const int t = cu_q[s], t1 = cu_q[s + 1], c = ctx_len[s], sl = slot[s];  // s < n_seqs
  if (t1 - t != 1 || t < 0 || t >= n_tokens) return;
  if (sl < 0 || sl >= n_slots || c < 0 || c + 1 > max_seq) return;
  const int ns = min(cdiv(c + 1, split_keys), nsplit);  // never past the launched splits
  const float* pp = part + ((int64_t)s * Hq + qh) * nsplit * (D + 2);
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

template <int D, bool PAGED>
static hipError_t run_decode(const void* q, const void* kc, const void* vc, float* part,
                             const BatchDev& b, const KvDev& kv, int Hq, int Hkv,
                             hipStream_t s) {
  const int max_kv = b.max_ctx_len + 1;
  const int split =
      attn_decode_split_keys(b.n_seqs, Hkv, max_kv, D, Hq / Hkv, attn_decode_max_split(kv));
  const int nsplit = cdiv(max_kv, split);
  const float scale_log2e = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  dim3 grid(nsplit, Hkv, b.n_seqs);
  const size_t smem = sizeof(DecSmem<D>) + (size_t)cdiv(Hq / Hkv, 512 / D) * 1024;
  attn_decode_kernel<D, PAGED><<<grid, 64, smem, s>>>(
      (const bf16*)q, (const bf16*)kc, (const bf16*)vc, part, b.cu_q, b.ctx_len, b.slot, kv, Hq,
      Hkv, nsplit, split, scale_log2e, b.n_tokens);
  return hipGetLastError();
}

hipError_t launch_attn_decode_split(const void* q, const void* kc, const void* vc, float* part,
                                    const BatchDev& b, const KvDev& kv, int n_q_heads,
                                    int n_kv_heads, int head_dim, hipStream_t s) {
  if (b.n_seqs == 0) return hipSuccess;
  const bool paged = kv.table != nullptr;
  if (head_dim == 128)
    return paged ? run_decode<128, true>(q, kc, vc, part, b, kv, n_q_heads, n_kv_heads, s)
                 : run_decode<128, false>(q, kc, vc, part, b, kv, n_q_heads, n_kv_heads, s);
  return paged ? run_decode<64, true>(q, kc, vc, part, b, kv, n_q_heads, n_kv_heads, s)
               : run_decode<64, false>(q, kc, vc, part, b, kv, n_q_heads, n_kv_heads, s);
}

hipError_t launch_attn_decode_combine(const float* part, void* out, const BatchDev& b,
                                      const KvDev& kv, int n_q_heads, int n_kv_heads,
                                      int head_dim, hipStream_t s) {
  if (b.n_seqs == 0) return hipSuccess;
  const int n_slots = kv.n_slots, max_seq = kv.max_seq;
  const int max_kv = b.max_ctx_len + 1;
  const int split = attn_decode_split_keys(b.n_seqs, n_kv_heads, max_kv, head_dim,
                                           n_q_heads / n_kv_heads, attn_decode_max_split(kv));
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
