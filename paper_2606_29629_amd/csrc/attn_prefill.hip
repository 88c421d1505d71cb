// Causal grouped-query flash attention for prefill and chunked prefill.
//
// One workgroup = one (sequence, query head, 128-query tile); 4 waves of 32
// queries.  Keys and values come from the KV cache (the q/k/v projection has
// already written this call's rows), 64 keys per tile.  K and V tiles go from
// HBM straight into LDS with buffer_load_dwordx4 ... lds, double buffered: the
// loads of tile k+1 are in flight while tile k is processed.  Key rows past
// the visible range read as zero (buffer range check) and are masked.
//
// Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16
// (A = K rows from LDS, B = the wave's queries held in registers for the whole
// loop).  A lane then owns one query column and 32 of the tile's 64 keys, so
// the running max / sum of the online softmax need one cross-lane exchange
// (lane ^ 32) per tile.  The output is kept transposed too, O^T += V^T P^T.
// P^T comes straight from the score accumulators.  V stays in its natural
// [key][d] layout and its MFMA operand is read with ds_read_b64_tr_b16: within
// each 16-lane group, the lanes of quad j point at key row j (4 dims each) and
// the instruction hands lane i the value at dim d0 + i of those four keys; two
// such reads give a lane its 8 keys in the order in which the score
// accumulator holds them.  P is split into P_hi = bf16(P) and
// P_lo = bf16(P - P_hi), two MFMAs into one accumulator, so the weights keep
// 16 significant bits.  Softmax in the log2 domain: one FMA (scale and max)
// and one v_exp_f32 per score; the running max is raised lazily (only past a
// slack of 8), so the accumulators are rescaled on few tiles.
//
// fp32 storage (F32, the tight-parity mode): q, the cache and the output are
// fp32, tiles hold fp32 rows, and both products run on the fp32 matrix
// instruction v_mfma_f32_32x32x2_f32 with the same tiling, mask and online
// softmax.  Its k-step t pairs head-dim values t (lanes 0..31) and
// D/2 + t (lanes 32..63) for S^T = K Q^T, and keys 8 j + i and 8 j + 4 + i
// for O^T = V^T P^T, the keys each lane's score accumulator holds, so P is
// used in fp32 where it was computed.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace tri {

constexpr int kFaBQ = 128;  // queries per workgroup
constexpr int kFaBK = 64;   // keys per tile
constexpr int kMaxFaSplit = 8;  // key-range splits of a query tile, at most
constexpr int kCombQ = 32;      // queries per workgroup of the split merge

// K/V tiles: four separate LDS arrays (K and V of buffers 0 and 1), [key][d]
// with chunks swizzled by kv_chunk (common.hpp).  Separate arrays, and a loop
// body instantiated per buffer, let the compiler see that reading one buffer
// never aliases the direct-to-LDS fill of the other, so it waits for no fill
// before a read.

// fp32 tiles: physical 16-byte chunk of logical chunk c in row r (rows of 16
// or 32 chunks): 16 consecutive rows read one logical chunk conflict-free.
__device__ __forceinline__ int kv_chunk_f32(int c, int r) { return c ^ (r & 15); }

// SPLIT: the key tiles of a query tile are dealt to `nsplit` workgroups
// (blockIdx.z = sequence * nsplit + split), each writing its unnormalised
// output with its running max (log2 units) and sum to `part`
// [nsplit][n_tokens][Hq][D + 2]; attn_prefill_combine_kernel merges them.
// Used when the batch has too few query tiles to fill the GPU (a chunk over
// a long cached prefix).
template <int D, bool PAGED, bool SPLIT, bool F32 = false>
__global__ __launch_bounds__(256, F32 ? 1 : 2) void attn_prefill_kernel(
    const void* __restrict__ Qv, const void* __restrict__ Kcv, const void* __restrict__ Vcv,
    void* __restrict__ Ov, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ ctx_len,
    const int32_t* __restrict__ slot, KvDev kv, int Hq, int Hkv, float scale_log2e,
    int include_single, int n_tokens, int nsplit, float* __restrict__ part) {
  using E = typename Store<F32>::T;             // storage element of q, cache, output
  constexpr int DC = D * (int)sizeof(E) / 16;   // 16-byte chunks per row
  constexpr int EPC = 16 / (int)sizeof(E);      // elements per chunk
  constexpr int ROWS_PER_KB = 64 / DC;          // tile rows filled by one 1 KB wave load
  constexpr int BLK = kFaBK / ROWS_PER_KB / 4;  // 1 KB loads per wave per operand and tile
  constexpr int DS = D / 16;                    // MFMA k-steps over d
  constexpr int DB = D / 32;                    // 32-row d blocks of O^T
  const E* __restrict__ Q = (const E*)Qv;
  const E* __restrict__ Kc = (const E*)Kcv;
  const E* __restrict__ Vc = (const E*)Vcv;
  E* __restrict__ O = (E*)Ov;
  __shared__ __align__(16) E sk0[kFaBK * D], sk1[kFaBK * D], sv0[kFaBK * D], sv1[kFaBK * D];
  auto chunk_of = [](int c, int r) {
    if constexpr (F32) return kv_chunk_f32(c, r);
    else return kv_chunk<D>(c, r);
  };

  const int s = SPLIT ? (int)blockIdx.z / nsplit : (int)blockIdx.z, qh = blockIdx.y;
  const int sp = SPLIT ? (int)blockIdx.z - s * nsplit : 0;
  // The sequence's scalars in one round trip (s < n_seqs by the grid).
  const int q0 = cu_q[s], n = cu_q[s + 1] - q0, c = ctx_len[s], sl = slot[s];
  if (n <= 0 || (n == 1 && !include_single) || q0 < 0 || q0 + n > n_tokens) return;
  const int qt = (int)gridDim.x - 1 - (int)blockIdx.x;  // heavy (late) tiles first
  if (qt * kFaBQ >= n) return;
  if (sl < 0 || sl >= kv.n_slots || c < 0 || c + n > kv.max_seq) return;
  const int kvh = (qh * Hkv) / Hq;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 31, lg = lane >> 5;
  const int kv_len = c + min(n, (qt + 1) * kFaBQ);
  const int nkt = cdiv(kv_len, kFaBK);
  // This workgroup's key tiles [kt_lo, kt_hi): all of them, or split sp's share.
  const int tps = SPLIT ? cdiv(nkt, nsplit) : nkt;
  const int kt_lo = sp * tps, kt_hi = min(nkt, kt_lo + tps);
  if (kt_lo >= kt_hi) return;  // an empty split (the combine skips it)

  // Tile kt's rows live in one cache panel (the slot, or a pool block of a
  // multiple of 64 rows); the block ids come from the table one tile ahead.
  const int prows = PAGED ? kv.block_size : kv.max_seq;
  auto panel_of = [&](int kt) {
    if (!PAGED || kt >= nkt) return sl;
    const int blk = kv.table[(int64_t)sl * kv.blocks_per_slot() + kt * kFaBK / kv.block_size];
    return (blk >= 0 && blk < kv.n_blocks) ? blk : -1;
  };
  // Descriptor of tile kt's rows of one operand: rows past the visible range
  // (and a block outside the pool) read as zero through the range check.
  auto tile_rsrc = [&](const E* base, int kt, int panel) {
    const int key0 = kt * kFaBK;
    int rows = min(kFaBK, kv_len - key0), prow = key0;
    if (PAGED) prow = key0 - (key0 / kv.block_size) * kv.block_size;
    if (panel < 0) rows = panel = prow = 0;
    return __builtin_amdgcn_make_buffer_rsrc(
        (void*)(base + (((int64_t)panel * Hkv + kvh) * prows + prow) * D), (short)0,
        rows * D * (int)sizeof(E), 0x00020000);
  };
  // Lane l of a 1 KB wave load fills physical chunk l % DC of tile row
  // l / DC of its block, i.e. logical chunk kv_chunk(l % DC, row) (the
  // swizzle is an involution).
  uint32_t ld_off[BLK];
#pragma unroll
  for (int j = 0; j < BLK; ++j) {
    const int row = (wave + 4 * j) * ROWS_PER_KB + lane / DC;
    ld_off[j] = (uint32_t)((row * D + chunk_of(lane % DC, row) * EPC) * (int)sizeof(E));
  }
  auto gload = [&](int kt, auto buf, int panel) {
    E* kd = buf ? sk1 : sk0;
    E* vd = buf ? sv1 : sv0;
    const __amdgpu_buffer_rsrc_t rk = tile_rsrc(Kc, kt, panel);
    const __amdgpu_buffer_rsrc_t rv = tile_rsrc(Vc, kt, panel);
#pragma unroll
    for (int j = 0; j < BLK; ++j) {
      const int blk = (wave + 4 * j) * ROWS_PER_KB * D;
      buffer_load_lds16(rk, kd + blk, ld_off[j], 0);
      buffer_load_lds16(rv, vd + blk, ld_off[j], 0);
    }
  };
  using Buf0 = std::integral_constant<int, 0>;
  using Buf1 = std::integral_constant<int, 1>;

  // This lane's query (clamped to a valid row; rows >= n are not written).
  const int qi = qt * kFaBQ + wave * 32 + lr;
  const int qrow = q0 + min(qi, n - 1);
  const int qpos = c + qi;                 // cache row of this query
  const int wave_qmin = c + qt * kFaBQ + wave * 32;
  // bf16: k-step t of lane (r, g) holds q values 16 t + 8 g .. + 7;
  // fp32: q values g D/2 .. g D/2 + D/2 - 1, one per k-step.
  bf16x8 qf[F32 ? 1 : DS];
  float q32[F32 ? D / 2 : 1];
  if constexpr (F32) {
    const float* qp = (const float*)Q + ((int64_t)qrow * Hq + qh) * D + lg * (D / 2);
#pragma unroll
    for (int t = 0; t < D / 8; ++t) {
      const f32x4 v = *(const f32x4*)(qp + 4 * t);
#pragma unroll
      for (int e = 0; e < 4; ++e) q32[4 * t + e] = v[e];
    }
  } else {
    const bf16* qp = (const bf16*)Q + ((int64_t)qrow * Hq + qh) * D + 8 * lg;
#pragma unroll
    for (int t = 0; t < DS; ++t) qf[t] = *(const bf16x8*)(qp + 16 * t);
  }

  // Transposing V reads: in 16-lane group G (lane / 16), lane i = lane % 16
  // points at key row 4 (lane / 32) + i / 4 of a 16-key group (+ 8 for the
  // second read), dims 32 b + 16 (G % 2) + 4 (i % 4) .. + 3.
  const int tr_key = 4 * lg + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  f32x16 oacc[DB];
#pragma unroll
  for (int b = 0; b < DB; ++b) oacc[b] = f32x16{0.f};
  float m_run = -INFINITY, l_run = 0.f;  // running max in raw score units
  const float slack_raw = kSoftmaxSlack / scale_log2e;

  gload(kt_lo, Buf0{}, panel_of(kt_lo));
  int next_panel = panel_of(kt_lo + 1);
  // Key tile kt from buffer `buf` (tiles alternate between the buffers,
  // the first in buffer 0).
  // Causal mask, tile max and the lazily raised running max of one key tile's
  // raw scores (both storage modes); returns the log2-domain offset of the
  // exponent.  Element r of block kb is key key0 + 32 kb + (r % 4) + 8 (r / 4)
  // + 4 lg.
  auto softmax_update = [&](f32x16 (&sacc)[2], int key0) {
    // Mask (raw scores; the scale is applied inside the exponent); element r
    // of block kb is key key0 + 32kb + (r%4) + 8(r/4) + 4lg.
    // The mask is a wave-uniform branch: only the tiles crossing the
    // diagonal pay for it.
    if (key0 + kFaBK - 1 > wave_qmin) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + 32 * kb + (r & 3) + 8 * (r >> 2) + 4 * lg;
          if (key > qpos) sacc[kb][r] = -INFINITY;
        }
    }
    // Raise the running max (raw units) only past the slack; rescale when
    // any lane of the wave did.  m_run is finite after the first tile (key 0
    // is visible to every query).  A query's scores sit in two lanes (lg = 0,
    // 1): when neither half of any row passes the threshold, no row's max
    // does, and the cross-lane exchange is skipped (the common case once
    // the max has settled).
    const float thr = m_run + slack_raw;
    const float mh = tree_max32(sacc);
    if (__builtin_amdgcn_ballot_w64(mh > thr)) {
      const float mt = fmaxf(mh, __shfl_xor(mh, 32, 64));
      const bool raise = mt > thr;
      const float m_new = raise ? mt : m_run;
      // (SPLIT: a lane that still has no finite max must not form -inf - -inf)
      const float alpha = (SPLIT && !raise) ? 1.f
                                            : __builtin_amdgcn_exp2f((m_run - m_new) * scale_log2e);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int b = 0; b < DB; ++b) oacc[b] *= alpha;
    }
    // (SPLIT: a lane whose query precedes every key seen so far in this
    // split still has no finite max; its weights are exp2(-inf) = 0.)
    const float mc = (SPLIT && m_run == -INFINITY) ? 0.f : m_run * scale_log2e;
    return mc;
  };
  // fp32 storage: one key tile on the fp32 matrix instruction.  S^T = K Q^T
  // (k-step t: head-dim values t and D/2 + t, K fragments four steps per
  // 16-byte read), then O^T += V^T P^T over keys 8 j + 4 lg + i, whose
  // weights are the lane's own score elements 4 j + i.
  // (always inlined: called out of line, its captures, the accumulators
  // among them, would live in private memory)
  auto step_f32 = [&](const E* k_lds, const E* v_lds, int key0) __attribute__((always_inline)) {
    if constexpr (F32) {
      constexpr int QC = D / 8;  // 16-byte chunks of a half row
      f32x16 sacc[2] = {f32x16{0.f}, f32x16{0.f}};
#pragma unroll
      for (int u = 0; u < QC; ++u) {
        f32x4 kf[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const int key = kb * 32 + lr;
          kf[kb] = *(const f32x4*)&k_lds[key * D + kv_chunk_f32(lg * QC + u, key) * 4];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
            sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(kf[kb][e], q32[4 * u + e], sacc[kb],
                                                            0, 0, 0);
      }
      const float mc = softmax_update(sacc, key0);
      float p[2][16];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          p[kb][r] = __builtin_amdgcn_exp2f(fmaf(sacc[kb][r], scale_log2e, -mc));
      float ls[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v8[e] = p[g >> 1][8 * (g & 1) + e];
        ls[g] = tree_sum8(v8);
      }
      l_run += (ls[0] + ls[1]) + (ls[2] + ls[3]);
      // V element (key, d), key = 32 kb + 8 j + 4 lg + i, d = 32 bb + lr: as
      // key % 16 = 8 (j % 2) + 4 lg + i, its swizzled chunk (d / 4) ^ (key % 16)
      // is 8 (bb ^ (j % 2)) + ((lr / 4) ^ (4 lg + i)), so four lane offsets
      // (one per i) plus compile-time constants address every read.
      int v_off[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        v_off[i] = (4 * lg + i) * D + (((lr >> 2) ^ (4 * lg + i)) << 2) + (lr & 3);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int bb = 0; bb < DB; ++bb) {
              const float vv = v_lds[v_off[i] + (32 * kb + 8 * j) * D + 32 * (bb ^ (j & 1))];
              oacc[bb] = __builtin_amdgcn_mfma_f32_32x32x2f32(vv, p[kb][4 * j + i], oacc[bb], 0,
                                                              0, 0);
            }
          }
    }
  };
  auto step = [&](int kt, auto buf) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();  // tile kt is in LDS; every wave is done with tile kt - 1
    if (kt + 1 < kt_hi) gload(kt + 1, std::integral_constant<int, 1 - buf>{}, next_panel);
    next_panel = panel_of(kt + 2);
    const E* kb_lds = buf ? sk1 : sk0;
    const E* vb = buf ? sv1 : sv0;
    const int key0 = kt * kFaBK;
    if (key0 > wave_qmin + 31) return;  // no key of this tile is visible to this wave
    if constexpr (F32) {
      step_f32(kb_lds, vb, key0);
    } else {
      // S^T = K Q^T for two 32-key blocks: the two MFMA chains interleaved,
      // K fragments read KLA k-steps ahead (a ring of KLA + 1), so no MFMA
      // waits on the LDS read issued just before it.
      constexpr int KLA = 3;
      f32x16 sacc[2] = {f32x16{0.f}, f32x16{0.f}};
      bf16x8 kf[KLA + 1][2];
      auto kread = [&](int t, bf16x8 (&dst)[2]) {
  #pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const int key = kb * 32 + lr;
          dst[kb] = *(const bf16x8*)&kb_lds[key * D + kv_chunk<D>(2 * t + lg, key) * 8];
        }
      };
  #pragma unroll
      for (int t = 0; t < KLA && t < DS; ++t) kread(t, kf[t]);
      // (the issue order is fenced: left alone, the compiler moves each read
      // next to its MFMA to save registers, and every MFMA waits on LDS)
  #pragma unroll
      for (int t = 0; t < DS; ++t) {
        if (t + KLA < DS) kread(t + KLA, kf[(t + KLA) % (KLA + 1)]);
  #pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[t % (KLA + 1)][kb], qf[t], sacc[kb],
                                                             0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
      // V^T fragments of a 16-key group (two transposing reads per d block),
      // the first group issued before the softmax.
      union VFrag { s16x4 s[2]; bf16x8 h; };
      VFrag vf[2][DB];
      auto vread = [&](int g16, VFrag (&dst)[DB]) {
        const int k1 = 16 * g16 + tr_key, k2 = k1 + 8;
  #pragma unroll
        for (int bb = 0; bb < DB; ++bb) {
          const int col = 32 * bb + tr_col;
          dst[bb].s[0] = lds_read_tr16(vb + k1 * D + kv_chunk<D>(col >> 3, k1) * 8 + (col & 7));
          dst[bb].s[1] = lds_read_tr16(vb + k2 * D + kv_chunk<D>(col >> 3, k2) * 8 + (col & 7));
        }
      };
      vread(0, vf[0]);
      const float mc = softmax_update(sacc, key0);
      bf16x8 pf[4], pl[4];
      float ls[4];  // the tile's row sum in four tree-summed parts
  #pragma unroll
      for (int kb = 0; kb < 2; ++kb)
  #pragma unroll
        for (int h = 0; h < 2; ++h) {
          float p8[8];
  #pragma unroll
          for (int e = 0; e < 8; ++e)
            p8[e] = __builtin_amdgcn_exp2f(fmaf(sacc[kb][8 * h + e], scale_log2e, -mc));
          ls[2 * kb + h] = tree_sum8(p8);
          split_hilo8(p8, pf[2 * kb + h], pl[2 * kb + h]);
        }
      l_run += (ls[0] + ls[1]) + (ls[2] + ls[3]);
      // O^T += V^T P^T over four 16-key groups: the hi MFMAs of the four d
      // blocks, then the lo ones (four independent chains), with the next
      // group's V fragments read meanwhile.
  #pragma unroll
      for (int g16 = 0; g16 < 4; ++g16) {
        if (g16 + 1 < 4) vread(g16 + 1, vf[(g16 + 1) & 1]);
  #pragma unroll
        for (int bb = 0; bb < DB; ++bb)
          oacc[bb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[g16 & 1][bb].h, pf[g16], oacc[bb], 0, 0, 0);
  #pragma unroll
        for (int bb = 0; bb < DB; ++bb)
          oacc[bb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[g16 & 1][bb].h, pl[g16], oacc[bb], 0, 0, 0);
      }
      }
};
  for (int kt = kt_lo; kt < kt_hi; kt += 2) {
    step(kt, Buf0{});
    if (kt + 1 < kt_hi) step(kt + 1, Buf1{});
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (qi >= n) return;
  if constexpr (SPLIT) {
    float* pp = part + (((int64_t)sp * n_tokens + q0 + qi) * Hq + qh) * (D + 2);
#pragma unroll
    for (int b = 0; b < DB; ++b)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
        *(f32x4*)(pp + 32 * b + 8 * r4 + 4 * lg) =
            f32x4{oacc[b][4 * r4], oacc[b][4 * r4 + 1], oacc[b][4 * r4 + 2], oacc[b][4 * r4 + 3]};
    if (lg == 0) {
      pp[D] = m_run == -INFINITY ? -INFINITY : m_run * scale_log2e;
      pp[D + 1] = l_tot;
    }
    return;
  }
  const float inv = 1.0f / l_tot;
  E* op = O + ((int64_t)(q0 + qi) * Hq + qh) * D;
  typedef E E4 __attribute__((ext_vector_type(4)));
  // oacc[b] element r: d = 32b + 8(r/4) + 4lg + r%4  -> 4 consecutive d per (r/4).
#pragma unroll
  for (int b = 0; b < DB; ++b)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      E4 o4;
#pragma unroll
      for (int e = 0; e < 4; ++e) o4[e] = (E)(oacc[b][4 * r4 + e] * inv);
      *(E4*)(op + 32 * b + 8 * r4 + 4 * lg) = o4;
    }
}

// Merge of the split partials of one (query tile, head): per query and
// head, the splits' (max, sum, unnormalised output) folded in split order.
// Same grid as the attention kernel without the split dimension; each thread
// takes four consecutive d of one query per pass.
template <int D>
__global__ __launch_bounds__(256) void attn_prefill_combine_kernel(
    const float* __restrict__ part, bf16* __restrict__ O, const int32_t* __restrict__ cu_q,
    const int32_t* __restrict__ ctx_len, const int32_t* __restrict__ slot, KvDev kv, int Hq,
    int include_single, int n_tokens, int nsplit) {
  const int s = blockIdx.z, qh = blockIdx.y;
  const int q0 = cu_q[s], n = cu_q[s + 1] - q0, c = ctx_len[s], sl = slot[s];
  if (n <= 0 || (n == 1 && !include_single) || q0 < 0 || q0 + n > n_tokens) return;
  const int qc = blockIdx.x;  // kCombQ-query chunk
  if (qc * kCombQ >= n) return;
  if (sl < 0 || sl >= kv.n_slots || c < 0 || c + n > kv.max_seq) return;
  const int qt = qc * kCombQ / kFaBQ;  // the flash query tile of the chunk
  const int nkt = cdiv(c + min(n, (qt + 1) * kFaBQ), kFaBK);
  const int tps = cdiv(nkt, nsplit);
  const int ns = cdiv(nkt, tps);  // non-empty splits (<= kMaxFaSplit)
  constexpr int TPQ = D / 4;      // threads per query
  const int d = 4 * ((int)threadIdx.x % TPQ);
  const int64_t plane = (int64_t)n_tokens * Hq * (D + 2);
  for (int qi = qc * kCombQ + (int)threadIdx.x / TPQ; qi < min(n, (qc + 1) * kCombQ);
       qi += 256 / TPQ) {
    const float* pp = part + ((int64_t)(q0 + qi) * Hq + qh) * (D + 2);
    // every split's partial is loaded before the fold (splits past ns re-read
    // the last one and are dropped), so the loads are in flight together
    float m[kMaxFaSplit], l[kMaxFaSplit];
    f32x4 a[kMaxFaSplit];
#pragma unroll
    for (int j = 0; j < kMaxFaSplit; ++j) {
      const float* pj = pp + min(j, ns - 1) * plane;
      m[j] = pj[D];
      l[j] = pj[D + 1];
      a[j] = *(const f32x4*)(pj + d);
    }
    float M = -INFINITY, L = 0.f;
    f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < kMaxFaSplit; ++j) {
      if (j >= ns || m[j] == -INFINITY) continue;  // no key of split j visible to this query
      const float Mn = fmaxf(M, m[j]);
      const float sc = exp2f(M - Mn), w = exp2f(m[j] - Mn);
      L = L * sc + l[j] * w;
      o = o * sc + a[j] * w;
      M = Mn;
    }
    const float inv = 1.0f / L;
    bf16x4 o4;
#pragma unroll
    for (int e = 0; e < 4; ++e) o4[e] = f2bf(o[e] * inv);
    *(bf16x4*)(O + ((int64_t)(q0 + qi) * Hq + qh) * D + d) = o4;
  }
}

// Key-range splits for a batch of n_tokens tokens: doubled (up to 8) while
// the split workgroups still fit about one per CU (1.25 per CU: the query
// tile count is estimated from n_tokens, which also counts the single-token
// sequences of a mixed step), and every split keeps >= 8 key tiles of the
// longest key range.  (Filling the second workgroup slot of each CU with
// more splits costs more in partials and merge than it gains: a 512-token
// chunk over a 6144-token prefix takes 117 us with 2 splits against 172 us
// with 8.)
int attn_prefill_splits(int n_seqs, int n_tokens, int max_q_len, int max_ctx_len,
                        int n_q_heads) {
  const int64_t wgs = (int64_t)cdiv(n_tokens, kFaBQ) * n_q_heads;  // query tiles of the batch
  const int max_tiles = cdiv(max_ctx_len + max_q_len, kFaBK);
  int sp = 1;
  while (sp < kMaxFaSplit && wgs * sp * 2 * 4 <= (int64_t)cu_count() * 5 &&
         max_tiles >= 16 * sp &&
         (int64_t)n_seqs * sp * 2 <= 65535)  // the grid's z extent
    sp *= 2;
  return sp;
}

size_t attn_prefill_partial_bytes(int n_seqs, int n_tokens, int max_q_len, int max_ctx_len,
                                  int n_q_heads, int head_dim) {
  const int sp = attn_prefill_splits(n_seqs, n_tokens, max_q_len, max_ctx_len, n_q_heads);
  return sp > 1 ? (size_t)sp * n_tokens * n_q_heads * (head_dim + 2) * sizeof(float) : 0;
}

template <int D, bool PAGED, bool SPLIT, bool F32 = false>
static hipError_t run_fa(const void* q, const void* kc, const void* vc, void* out,
                         const BatchDev& b, const KvDev& kv, int Hq, int Hkv,
                         int include_single, int nsplit, float* part, hipStream_t s) {
  dim3 grid(cdiv(b.max_q_len, kFaBQ), Hq, b.n_seqs * nsplit);
  const float scale_log2e = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  attn_prefill_kernel<D, PAGED, SPLIT, F32><<<grid, 256, 0, s>>>(
      q, kc, vc, out, b.cu_q, b.ctx_len, b.slot, kv, Hq, Hkv, scale_log2e, include_single,
      b.n_tokens, nsplit, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !SPLIT) return e;
  dim3 cgrid(cdiv(b.max_q_len, kCombQ), Hq, b.n_seqs);
  attn_prefill_combine_kernel<D><<<cgrid, 256, 0, s>>>(part, (bf16*)out, b.cu_q, b.ctx_len, b.slot,
                                                       kv, Hq, include_single, b.n_tokens, nsplit);
  return hipGetLastError();
}

template <int D, bool PAGED>
static hipError_t run_fa_any(const void* q, const void* kc, const void* vc, void* out,
                             const BatchDev& b, const KvDev& kv, int Hq, int Hkv,
                             int include_single, float* part, hipStream_t s) {
  const int sp = attn_prefill_splits(b.n_seqs, b.n_tokens, b.max_q_len, b.max_ctx_len, Hq);
  if (sp > 1)
    return run_fa<D, PAGED, true>(q, kc, vc, out, b, kv, Hq, Hkv, include_single, sp, part, s);
  return run_fa<D, PAGED, false>(q, kc, vc, out, b, kv, Hq, Hkv, include_single, 1, nullptr, s);
}

hipError_t launch_attn_prefill(const void* q, const void* kc, const void* vc, void* out,
                               const BatchDev& b, const KvDev& kv, int n_q_heads,
                               int n_kv_heads, int head_dim, int include_single, float* part,
                               hipStream_t s, bool f32) {
  if (b.n_seqs == 0 || b.max_q_len == 0) return hipSuccess;
  const bool paged = kv.table != nullptr;
  if (f32) {  // fp32 storage: no key-range split
    const int H = n_q_heads, G = n_kv_heads, I = include_single;
    if (head_dim == 128)
      return paged ? run_fa<128, true, false, true>(q, kc, vc, out, b, kv, H, G, I, 1, nullptr, s)
                   : run_fa<128, false, false, true>(q, kc, vc, out, b, kv, H, G, I, 1, nullptr, s);
    return paged ? run_fa<64, true, false, true>(q, kc, vc, out, b, kv, H, G, I, 1, nullptr, s)
                 : run_fa<64, false, false, true>(q, kc, vc, out, b, kv, H, G, I, 1, nullptr, s);
  }
  if (head_dim == 128)
    return paged ? run_fa_any<128, true>(q, kc, vc, out, b, kv, n_q_heads, n_kv_heads, include_single, part, s)
                 : run_fa_any<128, false>(q, kc, vc, out, b, kv, n_q_heads, n_kv_heads, include_single, part, s);
  return paged ? run_fa_any<64, true>(q, kc, vc, out, b, kv, n_q_heads, n_kv_heads, include_single, part, s)
               : run_fa_any<64, false>(q, kc, vc, out, b, kv, n_q_heads, n_kv_heads, include_single, part, s);
}

}  // namespace tri
