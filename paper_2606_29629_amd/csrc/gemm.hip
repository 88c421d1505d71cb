// Prefill GEMMs on the matrix cores: C[M,N] = A[M,K] B[N,K]^T, bf16 operands,
// fp32 accumulation, with the layer's epilogues fused (residual add, SwiGLU,
// q/k/v split + rotary embedding + KV-cache write, fp32 store).
//
// Both operands are K-contiguous ("nn.Linear" weights [out, in] and row-major
// activations), which is the native operand layout of the bf16 MFMAs with 8
// values per lane: in v_mfma_f32_32x32x16_bf16 lane l supplies row l % 32 and
// k 8 (l / 32) .. + 7, in v_mfma_f32_16x16x32_bf16 row l % 16 and k 8 (l / 16)
// .. + 7.
//
// Tiling: BM x BN x 64 block tile, WGM x WGN waves (two waves per SIMD, so one
// wave's LDS waits overlap the other's MFMAs), each wave a (BM/WGM) x (BN/WGN)
// sub-tile of SH x SH MFMA blocks: 32x32x16 or 16x16x32 instructions (the
// same flops per clock; the 16x16 form moves half the accumulator bytes per
// flop through the register file, which lets the power-capped prefill GEMMs
// hold a higher clock).  A and B tiles are staged through LDS, double
// buffered, with 16-byte chunks XOR-swizzled (see swz) so that fragment reads
// are free of bank conflicts.  Tiles move from HBM to LDS with
// buffer_load_dwordx4 ... lds (no register staging); the loads of tile k+1
// are in flight while the MFMAs of tile k run.
//
// Dense kernel: workgroups are dispatched round-robin over the 8 XCDs; the
// linear block id is remapped so each XCD owns a contiguous range of tiles,
// walked in groups of 8 M-tiles so co-resident tiles share A and B panels in
// that XCD's L2.
//
// Grouped kernel (mixture of experts): the rows of each expert are a
// contiguous segment of the routed (permuted) order; a device-side tile table
// maps every M-tile to its expert, A rows are gathered through the
// permutation, and B is that expert's weight matrix.  The grid is sized from
// an upper bound on the tile count and surplus workgroups exit, so no count is
// read back to the host; the real tiles are dealt to the XCDs in contiguous
// shares so that an expert's M-tiles share its weights in one L2.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace tri {

constexpr int kBK = 64;
constexpr int kGroupM = 8;
constexpr int kXcds = 8;
// Template-only epilogue kind: EPI_QKV with the per-head q/k RMSNorm (the
// Epi still says EPI_QKV; its q_norm pointer selects this instantiation).
constexpr int EPI_QKV_NORM = 5;

// LDS has 64 banks of 4 bytes (a 256-byte window).  A tile row is 128 bytes,
// so rows r and r+1 share a window; a ds_read_b128 phase of 16 lanes reads the
// same logical chunk of 16 consecutive rows.  XOR-ing the chunk with
// (row / 2) % 8 gives the 8 even and the 8 odd rows 8 distinct 16-byte slots
// each, i.e. all 16 slots of the window: no bank conflict.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// XCD-contiguous remap of block id bid among n: the blocks of XCD x (those
// with bid % 8 == x; dispatch is round-robin over the XCDs) take one
// contiguous range of ids.
__device__ __forceinline__ int xcd_id(int bid, int n) {
  const int per = n / kXcds, rem = n % kXcds;
  const int x = bid % kXcds, loc = bid / kXcds;
  return x * per + min(x, rem) + loc;
}

// Tile of grouped-M order id: groups of kGroupM M-tiles, walked column by
// column, so co-resident tiles share A and B panels in L2.
__device__ __forceinline__ void tile_of_id(int id, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int group = id / (kGroupM * tiles_n);
  const int first_m = group * kGroupM;
  const int gm = min(kGroupM, tiles_m - first_m);
  const int in = id - group * kGroupM * tiles_n;
  tm = first_m + in % gm;
  tn = in / gm;
}

__device__ __forceinline__ void tile_of_block(int bid, int tiles_m, int tiles_n, int& tm,
                                              int& tn) {
  tile_of_id(xcd_id(bid, tiles_m * tiles_n), tiles_m, tiles_n, tm, tn);
}

// MFMA shape SH: SH x SH output blocks, KSTEP = 512 / SH of k per
// instruction, the accumulator a 16- or 4-vector per lane.
template <int SH>
struct Mfma;
template <>
struct Mfma<32> {
  using acc_t = f32x16;
  static constexpr int KSTEP = 16;
  __device__ __forceinline__ static acc_t mma(bf16x8 a, bf16x8 b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mfma<16> {
  using acc_t = f32x4;
  static constexpr int KSTEP = 32;
  __device__ __forceinline__ static acc_t mma(bf16x8 a, bf16x8 b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

// Accumulator geometry.  Block (i, j) of a wave holds C^T (the weight rows
// are the MFMA's row operand): lane l owns token row SH i + l % SH and, in
// each block, QN = SH * SH / 256 groups of four consecutive output columns,
// group q at SH j + (256 / SH) q + 4 (l / SH).  The epilogues walk the G =
// NI * QN groups of a row block: group g = QN j + q, column offset col(g)
// (plus the lane's 4 (l / SH)), values grp(acc, i, g).
template <int SH, int MI, int NI>
struct AccGeo {
  using acc_t = typename Mfma<SH>::acc_t;
  static constexpr int QN = SH * SH / 256, G = NI * QN;
  __device__ __forceinline__ static constexpr int col(int g) {
    return SH * (g / QN) + (256 / SH) * (g % QN);
  }
  __device__ __forceinline__ static f32x4 grp(const acc_t (&acc)[MI][NI], int i, int g) {
    if constexpr (SH == 32) {
      const int j = g / 4, q = g % 4;
      return f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                   acc[i][j][4 * q + 3]};
    } else {
      return acc[i][g];
    }
  }
  __device__ __forceinline__ static int lane_row(int lane) { return lane % SH; }
  __device__ __forceinline__ static int lane_col(int lane) { return 4 * (lane / SH); }
};

// MFMA shapes per tile family: the compute-bound prefill tiles (256 x 256,
// the grouped expert tiles of 128 or 256 rows) and the mid-size-M tiles.  The
// weight-streaming decode tiles keep 32 x 32 blocks.
constexpr int kPrefillSH = 16;
constexpr int kMidSH = 16;

template <int BM, int BN, int S = 2>
struct GemmSmem {
  bf16 a[S][BM * kBK];
  bf16 b[S][BN * kBK];
};

// B-tile row -> weight row.  For SwiGLU each wave's N sub-tile holds WN/2 gate
// rows followed by the matching WN/2 up rows, so a lane owns gate and up of
// the same output column in blocks j and j + NI/2.
template <int BN, int WN>
__device__ __forceinline__ int b_row_of(int kind, int tn, int nt, int ffn) {
  if (kind == EPI_SWIGLU) {
    const int wc = nt / WN, w = nt % WN;
    const int f = tn * (BN / 2) + wc * (WN / 2) + (w % (WN / 2));
    return w < WN / 2 ? f : ffn + f;
  }
  return tn * BN + nt;
}

// Residual prefetch for the 256 x 256 residual epilogue.  The loads for the
// two tiles past the last one (zeros otherwise) fetch instead the two 128-row
// halves of the output tile's residual into the buffers they would fill: half
// h into buffer (KT + h) % 2, its rows 0..63 in the A region, 64..127 in the B
// region, row-major with 512-byte rows whose 16-byte chunks are stored at
// chunk ^ (row % 16) (16 consecutive rows read one logical chunk without bank
// conflicts).  Piece j of wave w in a region covers region rows 2 L and 2 L + 1,
// L = w + 8 j; lane l writes position l % 32 of row 2 L + l / 32, so it fetches
// logical chunk (l % 32) ^ ((2 w + l / 32) % 16) (the swizzle is an
// involution).  Rows past M read as zero through the descriptor's range.
struct ResPf {
  __amdgpu_buffer_rsrc_t rsrc;  // residual of the tile's rows (rows past M out of range)
  uint32_t voff;                // lane part: row l / 32 of the piece, source chunk
  int ld_bytes;                 // residual row stride in bytes
  bool on;
};

// The shared K loop.  a_off / b_off: byte offset (within the buffer) of chunk
// swz(row, lane % 8) of this lane's row in each of its 1 KB LDS blocks (at or
// beyond the buffer size for rows that must read as zero).
//
// S LDS stages, tiles loaded S - 1 ahead.  Schedule of k-tile t (KSTEPS
// k-steps of one MFMA's depth): the fragments of k-step s + 1 are read from
// LDS while the MFMAs of step s run.  Before the MFMAs of the last step, each
// wave waits for its loads of tile t + 1 (those of tiles t + 2 .. t + S - 1
// may stay in flight), one barrier makes tile t + 1 visible and retires every
// read of tile t, the loads of tile t + S go into tile t's buffer and the
// first fragments of tile t + 1 are read -- all under the last step's MFMAs,
// so the barrier costs no matrix-core time beyond the skew between waves.
// Compute-bound tiles use S = 2; the decode projections, bound by the weight
// stream, use more stages for more bytes in flight per CU.
template <int BM, int BN, int WGM, int WGN, int S = 2, int SH = 32>
struct Mainloop {
  using MF = Mfma<SH>;
  using acc_t = typename MF::acc_t;
  static constexpr int NT = WGM * WGN * 64;
  static constexpr int NW = NT / 64;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int MI = WM / SH, NI = WN / SH;
  static constexpr int A_BLK = BM / 8 / NW, B_BLK = BN / 8 / NW;  // 1 KB blocks per wave
  static constexpr int KSTEPS = kBK / MF::KSTEP;
  static_assert(WM % SH == 0 && WN % SH == 0, "wave tile of whole MFMA blocks");

  // MA = the wave's row blocks that hold rows of the tile's valid range
  // (compile-time, MA <= MI): blocks past it would only multiply zero rows,
  // so the wave issues neither their MFMAs nor their A fragment reads (with
  // MA = 0, no MFMA and no fragment read at all).  Its share of the tile
  // loads and every barrier stay, so all waves keep the same barrier count.
  template <int MA, bool RPF = false>
  __device__ __forceinline__ static void run_rows(GemmSmem<BM, BN, S>& sm,
                                                  __amdgpu_buffer_rsrc_t ra,
                                                  const uint32_t (&a_off)[A_BLK],
                                                  __amdgpu_buffer_rsrc_t rb,
                                                  const uint32_t (&b_off)[B_BLK], int K, int wv,
                                                  int lane, acc_t (&acc)[MI][NI],
                                                  const ResPf& rp, int kshift) {
    static_assert(MA >= 0 && MA <= MI, "active row blocks");
    static_assert(!RPF || (BM == 256 && BN == 256 && NW == 8 && S == 2),
                  "residual prefetch: two 64-row regions of 32 pieces per buffer");
    const int wm = wv / WGN, wn = wv % WGN;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) acc[i][j] = acc_t{0.f};
    // kill = 0x80000000 pushes every offset past the buffer's range, so the
    // load writes zeros instead of touching memory (used past the last tile,
    // keeping the schedule free of branches).
    // k-tile kt of the loop reads k-tile (kt + kshift) mod KT of the operands
    // (a rotation: the loop still visits every k-tile once, in a fixed order)
    const int KTr = K / kBK;
    auto kbyte = [&](int kt) {
      const int kk = kt + kshift;
      return (kk >= KTr ? kk - KTr : kk) * kBK * 2;
    };
    auto gload = [&](int kt, int buf, uint32_t kill) {
      const int kb = kbyte(kt);
#pragma unroll
      for (int j = 0; j < A_BLK; ++j)
        buffer_load_lds16(ra, &sm.a[buf][(wv + NW * j) * 8 * kBK], a_off[j] | kill, kb);
#pragma unroll
      for (int j = 0; j < B_BLK; ++j)
        buffer_load_lds16(rb, &sm.b[buf][(wv + NW * j) * 8 * kBK], b_off[j] | kill, kb);
    };
    // Fragment reads.  The lane reads row SH i + l % SH of a block and the
    // 16-byte chunk ks * KSTEP / 8 + l / SH of the step.  The swizzle of a row
    // depends on (row / 2) % 8 only, the same for rows r and r + SH i, so one
    // byte address per operand and k-step serves every block and buffer
    // (immediate offsets).
    uint32_t a_base[KSTEPS], b_base[KSTEPS];
    {
      const int lr = lane % SH, lg = lane / SH;
      const int ra0 = wm * WM + lr, rb0 = wn * WN + lr;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        const int ch = ks * (MF::KSTEP / 8) + lg;
        a_base[ks] = (uint32_t)((ra0 * kBK + swz(ra0, ch) * 8) * 2);
        b_base[ks] = (uint32_t)((rb0 * kBK + swz(rb0, ch) * 8) * 2);
      }
    }
    const char* const lds_a = (const char*)&sm.a[0][0];
    const char* const lds_b = (const char*)&sm.b[0][0];
    auto rd_a = [&](int buf, int ks, int i) {
      return *(const bf16x8*)(lds_a + a_base[ks] + (buf * BM * kBK + i * SH * kBK) * 2);
    };
    auto rd_b = [&](int buf, int ks, int j) {
      return *(const bf16x8*)(lds_b + b_base[ks] + (buf * BN * kBK + j * SH * kBK) * 2);
    };
    bf16x8 fa[2][MI], fb[2][NI];
    auto lload = [&](int buf, int ks, int slot) {
      if constexpr (MA == 0) return;
#pragma unroll
      for (int i = 0; i < MA; ++i) fa[slot][i] = rd_a(buf, ks, i);
#pragma unroll
      for (int j = 0; j < NI; ++j) fb[slot][j] = rd_b(buf, ks, j);
    };
    // Fragment f of a k-step: f < MA -> A block f, else B block f - MA.
    auto lread = [&](int buf, int ks, int slot, int f) {
      if (f < MA) fa[slot][f] = rd_a(buf, ks, f);
      else fb[slot][f - MA] = rd_b(buf, ks, f - MA);
    };
    // Load piece p of a tile: p < A_BLK -> A block p, else B block p - A_BLK.
    auto gpiece = [&](int kt, int buf, uint32_t kill, int p) {
      const int kb = kbyte(kt);
      if (p < A_BLK)
        buffer_load_lds16(ra, &sm.a[buf][(wv + NW * p) * 8 * kBK], a_off[p] | kill, kb);
      else
        buffer_load_lds16(rb, &sm.b[buf][(wv + NW * (p - A_BLK)) * 8 * kBK],
                          b_off[p - A_BLK] | kill, kb);
    };
    // Piece p of residual half h (ResPf): the LDS destination of tile piece p.
    auto rpiece = [&](int h, int buf, int p) {
      const int reg = p < A_BLK ? 0 : 1, j = p - reg * A_BLK;
      const int row = 128 * h + 64 * reg + 2 * (wv + NW * j);
      void* dst = reg ? (void*)&sm.b[buf][(wv + NW * j) * 8 * kBK]
                      : (void*)&sm.a[buf][(wv + NW * j) * 8 * kBK];
      buffer_load_lds16(rp.rsrc, dst, rp.voff, row * rp.ld_bytes);
    };
    // B (weight rows) as the MFMA's row operand and A (token rows) as its
    // column operand: accumulator block (i, j) holds C^T, so a lane owns one
    // token row and groups of four consecutive output columns, and the
    // epilogues move 8 or 16 contiguous bytes per lane.
    auto mfma = [&](int slot, int g) {
      const int i = g / NI, j = g % NI;
      acc[i][j] = MF::mma(fb[slot][j], fa[slot][i], acc[i][j]);
    };
    constexpr int NMF = MA * NI, NRD = MA > 0 ? MA + NI : 0, NLD = A_BLK + B_BLK;
    constexpr int NG = NMF > NRD ? NMF : NRD;
    constexpr int NGL = NG > NLD ? NG : NLD;
    const int KT = K / kBK;
    static_assert((S - 1) * NLD < 64, "vmcnt counts up to 63");
#pragma unroll
    for (int t = 0; t < S; ++t) gload(t, t, t < KT ? 0u : 0x80000000u);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"((S - 1) * NLD) : "memory");  // tile 0 landed
    __syncthreads();
    lload(0, 0, 0);
    int buf = 0;
    // The issue order is spelled out: one MFMA, then one LDS read for the next
    // k-step (and on the last step one or more tile loads), fenced so the
    // compiler keeps it.
    auto ktile = [&](int kt, auto res) {
      const int nbuf = buf + 1 == S ? 0 : buf + 1;
#pragma unroll
      for (int ks = 0; ks + 1 < KSTEPS; ++ks) {
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          if (g < NMF) mfma(ks & 1, g);
          if (g < NRD) lread(buf, ks + 1, (ks + 1) & 1, g);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      constexpr int last = (KSTEPS - 1) & 1;
      // this wave's tile t + 1 loads
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"((S - 2) * NLD) : "memory");
      __syncthreads();
      const uint32_t kill = kt + S < KT ? 0u : 0x80000000u;
#pragma unroll
      for (int g = 0; g < NGL; ++g) {
        if (g < NMF) mfma(last, g);
        if (g < NLD) {
          if constexpr (decltype(res)::value) rpiece(kt + S - KT, buf, g);
          else gpiece(kt + S, buf, kill, g);
        }
        if (g < NRD) lread(nbuf, 0, last ^ 1, g);  // stale but in-range on the last tile
        __builtin_amdgcn_sched_barrier(0);
      }
      buf = nbuf;
    };
    // With the residual prefetch, the last S k-tiles (those whose tile + S
    // does not exist) run in a loop of their own that loads residual halves.
    const int kt_main = (RPF && rp.on) ? KT - S : KT;
    int kt = 0;
    for (; kt < kt_main; ++kt) ktile(kt, std::false_type{});
    if constexpr (RPF) {
      for (; kt < KT; ++kt) ktile(kt, std::true_type{});
    }
  }
  // The tile's first `rows` rows are valid: the wave runs the instantiation
  // for its active row blocks (a wave-uniform choice).
  template <int MA = MI, bool RPF = false>
  __device__ __forceinline__ static void run_valid(int rows, GemmSmem<BM, BN, S>& sm,
                                                   __amdgpu_buffer_rsrc_t ra,
                                                   const uint32_t (&a_off)[A_BLK],
                                                   __amdgpu_buffer_rsrc_t rb,
                                                   const uint32_t (&b_off)[B_BLK], int K, int wv,
                                                   int lane, acc_t (&acc)[MI][NI],
                                                   const ResPf& rp = ResPf{}, int kshift = 0) {
    const int wm = wv / WGN;
    const int act = (rows - wm * WM + SH - 1) / SH;  // row blocks holding valid rows
    if constexpr (MA == 0) {
      run_rows<0, RPF>(sm, ra, a_off, rb, b_off, K, wv, lane, acc, rp, kshift);
    } else {
      if (act >= MA) run_rows<MA, RPF>(sm, ra, a_off, rb, b_off, K, wv, lane, acc, rp, kshift);
      else run_valid<MA - 1, RPF>(rows, sm, ra, a_off, rb, b_off, K, wv, lane, acc, rp, kshift);
    }
  }
};

// Epilogues.  The accumulators are read by column group (AccGeo): row0 =
// output row of the lane in row block 0 (including l % SH); col0 = output
// column of the lane's first group (including 4 (l / SH)).  Rows >= row_lim
// and column groups >= N are not written (N is a multiple of 4).  Operands
// of a lane's row (residual) are loaded for a whole row block before any
// store, at clamped addresses, so no load waits behind a store.
template <int SH, int MI, int NI, int EK>
__device__ __forceinline__ void plain_epilogue(
    const typename Mfma<SH>::acc_t (&acc)[MI][NI], const Epi& epi, int row0, int row_lim,
    int col0, int N) {
  using Geo = AccGeo<SH, MI, NI>;
  constexpr int G = Geo::G;
  constexpr int KIND = EK & kEpiKindMask;
  using T = typename Store<(EK & kEpiF32) != 0>::T;
  typedef T T4 __attribute__((ext_vector_type(4)));
  const T* __restrict__ resid = (const T*)epi.resid;
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int row = row0 + SH * i;
    const int rc = min(row, row_lim - 1);
    T4 res[G];
    if constexpr (KIND == EPI_RESID) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int col = min(col0 + Geo::col(g), N - 4);
        res[g] = *(const T4*)(resid + (int64_t)rc * epi.ldr + col);
      }
    }
    if (row >= row_lim) continue;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int col = col0 + Geo::col(g);
      if (col >= N) continue;
      const f32x4 v = Geo::grp(acc, i, g);
      if constexpr (KIND == EPI_STORE_F32) {
        *(f32x4*)((float*)epi.out + (int64_t)row * epi.ldo + col) = v;
      } else {
        T4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float x = v[e];
          if constexpr (KIND == EPI_RESID) x += (float)res[g][e];
          o[e] = (T)x;
        }
        *(T4*)((T*)epi.out + (int64_t)row * epi.ldo + col) = o;
      }
    }
  }
}

// The residual epilogue of a 256 x 256 tile whose residual was prefetched
// into LDS (ResPf): tile-relative row tr / column tc of the lane's first group
// (row0 - tile row0 and col0 - tile col0), kt_par = KT % 2.  The caller has
// waited for the prefetch loads and passed a barrier.
template <int SH, int MI, int NI>
__device__ __forceinline__ void resid_lds_epilogue(
    const typename Mfma<SH>::acc_t (&acc)[MI][NI], const Epi& epi, int row0, int row_lim,
    int col0, int N, const char* smem, int kt_par, int tr, int tc) {
  using Geo = AccGeo<SH, MI, NI>;
  constexpr int G = Geo::G;
  constexpr int kRegion = 256 * kBK * 2;  // bytes of one buffer's A (or B) region
  typedef bf16 T4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int row = row0 + SH * i, r = tr + SH * i;
    const int h = r >> 7, reg = (r >> 6) & 1, rr = r & 63;
    const char* rbase = smem + reg * 2 * kRegion + ((kt_par + h) & 1) * kRegion + rr * 512;
    T4 res[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int c = tc + Geo::col(g);
      res[g] = *(const T4*)(rbase + (((c >> 3) ^ (rr & 15)) << 4) + (c & 7) * 2);
    }
    if (row >= row_lim) continue;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int col = col0 + Geo::col(g);
      if (col >= N) continue;
      const f32x4 v = Geo::grp(acc, i, g);
      T4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = (bf16)(v[e] + (float)res[g][e]);
      *(T4*)((bf16*)epi.out + (int64_t)row * epi.ldo + col) = o;
    }
  }
}

// SwiGLU: the first half of a wave's columns holds gate rows, the second half
// the matching up rows (b_row_of), so group g < G / 2 pairs with g + G / 2;
// f0 = output column (intermediate index) of the lane's first group.
template <int SH, int MI, int NI, bool F32>
__device__ __forceinline__ void swiglu_epilogue(const typename Mfma<SH>::acc_t (&acc)[MI][NI],
                                                const Epi& epi, int row0, int row_lim, int f0) {
  using Geo = AccGeo<SH, MI, NI>;
  constexpr int G = Geo::G;
  using T = typename Store<F32>::T;
  typedef T T4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int row = row0 + SH * i;
    if (row >= row_lim) continue;
#pragma unroll
    for (int g = 0; g < G / 2; ++g) {
      const int f = f0 + Geo::col(g);
      if (f >= epi.ffn) continue;
      const f32x4 gt = Geo::grp(acc, i, g), up = Geo::grp(acc, i, g + G / 2);
      T4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = (T)(silu(gt[e]) * up[e]);
      *(T4*)((T*)epi.out + (int64_t)row * epi.ldo + f) = o;
    }
  }
}

// QB consecutive first-half groups g0 .. g0 + QB - 1 of row block i, all in
// one q (KIND 0), k (1) or v (2) head: the lane's token row, head-dim values
// d + (col(g0 + u) - col(g0)) + e of the first half and the same plus D / 2
// from group g0 + u + GH.
template <int KIND, int SH, int MI, int NI, int GH, int QB, bool F32>
__device__ __forceinline__ void qkv_block(const typename Mfma<SH>::acc_t (&acc)[MI][NI],
                                          const Epi& epi, int i, int g0, int D, int row0, int M,
                                          int head, int d, const float (&b1)[QB][4],
                                          const float (&b2)[QB][4]) {
  using Geo = AccGeo<SH, MI, NI>;
  const int half = D / 2;
  using T = typename Store<F32>::T;
  typedef T T4 __attribute__((ext_vector_type(4)));
  const int Hq = epi.n_q_heads, Hkv = epi.n_kv_heads;
  const int row = row0 + SH * i;
  const int rc = min(row, M - 1);
  f32x4 cs[QB][2];  // (cos, sin) of the group's 4 values: [u][0] = e 0..1, [u][1] = e 2..3
  int sl = 0, tr = 0;
  if constexpr (KIND != 2) {
    const float2* __restrict__ rp = epi.rope + (int64_t)rc * half + d;
#pragma unroll
    for (int u = 0; u < QB; ++u) {
      const int dc = Geo::col(g0 + u) - Geo::col(g0);
      cs[u][0] = *(const f32x4*)(rp + dc);
      cs[u][1] = *(const f32x4*)(rp + dc + 2);
    }
  }
  if constexpr (KIND != 0) {
    sl = epi.tok_slot[rc];
    tr = epi.tok_row[rc];
  }
  if (row >= M) return;
  T* p;
  if constexpr (KIND == 0) {
    p = (T*)epi.q + ((int64_t)row * Hq + head) * D + d;
  } else {
    if (sl < 0) return;
    const int kvh = KIND == 1 ? head - Hq : head - Hq - Hkv;
    p = (T*)(KIND == 1 ? epi.kc : epi.vc) + (((int64_t)sl * Hkv + kvh) * epi.max_seq + tr) * D + d;
  }
#pragma unroll
  for (int u = 0; u < QB; ++u) {
    const int dc = Geo::col(g0 + u) - Geo::col(g0);
    const f32x4 v1 = Geo::grp(acc, i, g0 + u), v2 = Geo::grp(acc, i, g0 + u + GH);
    T4 o1, o2;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float x1 = v1[e] + b1[u][e], x2 = v2[e] + b2[u][e];
      if constexpr (KIND != 2) {
        const float c = cs[u][e >> 1][2 * (e & 1)], sn = cs[u][e >> 1][2 * (e & 1) + 1];
        const float y1 = x1 * c - x2 * sn;
        const float y2 = x2 * c + x1 * sn;
        x1 = y1;
        x2 = y2;
      }
      o1[e] = (T)x1;
      o2[e] = (T)x2;
    }
    *(T4*)(p + dc) = o1;
    *(T4*)(p + dc + half) = o2;
  }
}

// q/k/v split + bias + rotary embedding + KV-cache write on the accumulators.
// HB = D / 64.  A half head is GH = D / 2 / SH * QN groups, so a first-half
// group g pairs with g + GH (same lane, same element).  The groups are taken
// QB at a time (QB <= GH, all in one half head): the rotary factors (four
// (cos, sin) pairs per group, 32 contiguous bytes) and, for k/v heads, the
// token's cache slot and row are loaded before the stores.
template <int SH, int MI, int NI, int HB, bool F32>
__device__ __forceinline__ void qkv_epilogue(const typename Mfma<SH>::acc_t (&acc)[MI][NI],
                                             const Epi& epi, int row0, int col0, int M, int N) {
  using St = Store<F32>;
  using Geo = AccGeo<SH, MI, NI>;
  constexpr int D = HB * 64, half = D / 2;
  constexpr int GH = half / SH * Geo::QN;
  constexpr int QB = GH < 4 ? GH : 4;
  static_assert(GH % QB == 0 && Geo::G % (2 * GH) == 0, "whole heads per wave");
  const int Hq = epi.n_q_heads, Hkv = epi.n_kv_heads;
#pragma unroll
  for (int g0 = 0; g0 < Geo::G; g0 += QB) {
    if ((g0 / GH) & 1) continue;
    const int col = col0 + Geo::col(g0);  // first-half column of the lane's first group
    if (col >= N) continue;
    const int head = col / D, d = col % D;
    float b1[QB][4], b2[QB][4];
#pragma unroll
    for (int u = 0; u < QB; ++u) {
      const int dc = Geo::col(g0 + u) - Geo::col(g0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        b1[u][e] = epi.bias ? St::ld(epi.bias, col + dc + e) : 0.f;
        b2[u][e] = epi.bias ? St::ld(epi.bias, col + dc + e + half) : 0.f;
      }
    }
    // the head, hence its kind, is uniform across the wave
    const int kind = __builtin_amdgcn_readfirstlane(head < Hq ? 0 : (head < Hq + Hkv ? 1 : 2));
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      if (kind == 0)
        qkv_block<0, SH, MI, NI, GH, QB, F32>(acc, epi, i, g0, D, row0, M, head, d, b1, b2);
      else if (kind == 1)
        qkv_block<1, SH, MI, NI, GH, QB, F32>(acc, epi, i, g0, D, row0, M, head, d, b1, b2);
      else
        qkv_block<2, SH, MI, NI, GH, QB, F32>(acc, epi, i, g0, D, row0, M, head, d, b1, b2);
    }
  }
}

// The q/k/v epilogue with the per-head RMSNorm of q and k.  The sum of
// squares over a head needs every value of a (token, head) before any can be
// stored, more registers than the accumulator tile leaves free, so this
// epilogue goes through LDS (free once every wave is past the mainloop and
// its last loads have landed): one row block (SH rows) of the wave's tile at
// a time, each wave in its own SH x WC fp32 region, 16-byte chunks stored at
// chunk c ^ row (conflict-free column writes and row reads).  Then each lane takes
// four consecutive rotary pairs of a row: 16 lanes cover a row's WC / 2 = 64
// pairs, a pass covers 4 rows, and a head's pairs are an aligned group of
// D / 8 lanes, its sum of squares a group sum.  The lane's columns, bias and
// gains stay fixed across rows.
template <int SH, int MI, int NI, bool F32>
__device__ __forceinline__ void qkv_norm_epilogue(const typename Mfma<SH>::acc_t (&acc)[MI][NI],
                                                  const Epi& epi, char* smem, int wv, int lane,
                                                  int wrow0, int wcol0, int M, int N) {
  using St = Store<F32>;
  using T = typename St::T;
  using Geo = AccGeo<SH, MI, NI>;
  typedef T T4 __attribute__((ext_vector_type(4)));
  constexpr int WC = NI * SH;
  static_assert(WC == 128, "16 lanes per row of the wave's columns");
  const int lr = Geo::lane_row(lane), lg = lane / SH;
  const int D = epi.head_dim, half = D / 2;
  const int Hq = epi.n_q_heads, Hkv = epi.n_kv_heads;
  const int rl = lane >> 4;                       // row within a 4-row pass
  const int p0 = 4 * (lane & 15);                 // first of the lane's 4 pairs
  const int hw = p0 / half, d = p0 % half;        // head within the wave's columns
  const int c1 = hw * D + d, c2 = c1 + half;      // wave columns of the 4 first / second values
  const bool col_ok = wcol0 + c1 < N;             // whole heads: N is a multiple of D
  const int col = col_ok ? wcol0 + c1 : 0;
  const int head = col / D;
  const int kind = head < Hq ? 0 : (head < Hq + Hkv ? 1 : 2);
  float b1[4], b2[4], g1[4], g2[4];
  {
    const void* bp = epi.bias;
    const void* gp = kind == 0 ? epi.q_norm : epi.k_norm;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      b1[e] = bp ? St::ld(bp, col + e) : 0.f;
      b2[e] = bp ? St::ld(bp, col + half + e) : 0.f;
      g1[e] = kind == 2 ? 1.f : St::ld(gp, d + e);
      g2[e] = kind == 2 ? 1.f : St::ld(gp, d + half + e);
    }
  }
  const int kvh = kind == 1 ? head - Hq : head - Hq - Hkv;
  T* const cache = (T*)(kind == 1 ? epi.kc : epi.vc);
  const float inv_d = 1.0f / (float)D;

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  float* __restrict__ buf = (float*)smem + wv * SH * WC;
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    // group g of the row block is row lr, columns col(g) + 4 lg .. + 3
#pragma unroll
    for (int g = 0; g < Geo::G; ++g)
      *(f32x4*)&buf[lr * WC + (((Geo::col(g) / 4 + lg) ^ lr) << 2)] = Geo::grp(acc, i, g);
    const int rbase = wrow0 + SH * i;
    // two passes (8 rows) at a time: the rotary factors, cache slots and rows
    // are loaded before the first store (a store could alias a later load)
    for (int t0 = 0; t0 < SH; t0 += 8) {
      if (rbase + t0 >= M) break;  // uniform
      f32x4 cs[2][2];              // (cos, sin) of pairs d .. d + 3: [pass][0] = 0..1, [1] = 2..3
      int sl[2], tr[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int rc = min(rbase + t0 + 4 * u + rl, M - 1);
        const float2* rp = epi.rope + (int64_t)rc * half + d;
        cs[u][0] = *(const f32x4*)rp;
        cs[u][1] = *(const f32x4*)(rp + 2);
        sl[u] = epi.tok_slot[rc];
        tr[u] = epi.tok_row[rc];
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int t = t0 + 4 * u + rl, row = rbase + t;
        const f32x4 v1 = *(const f32x4*)&buf[t * WC + (((c1 >> 2) ^ t) << 2)];
        const f32x4 v2 = *(const f32x4*)&buf[t * WC + (((c2 >> 2) ^ t) << 2)];
        float x1[4], x2[4], ss = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x1[e] = v1[e] + b1[e];
          x2[e] = v2[e] + b2[e];
          ss += x1[e] * x1[e] + x2[e] * x2[e];
        }
        // sum over the head's D / 8 lanes (8 or 16, aligned)
        ss += __shfl_xor(ss, 1, 64);
        ss += __shfl_xor(ss, 2, 64);
        ss += __shfl_xor(ss, 4, 64);
        if (half == 64) ss += __shfl_xor(ss, 8, 64);
        T4 o1, o2;
        const float r = 1.0f / sqrtf(ss * inv_d + epi.eps);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float y1 = x1[e], y2 = x2[e];
          if (kind != 2) {
            y1 *= r * g1[e];
            y2 *= r * g2[e];
            const float c = cs[u][e >> 1][2 * (e & 1)], sn = cs[u][e >> 1][2 * (e & 1) + 1];
            const float z1 = y1 * c - y2 * sn;
            const float z2 = y2 * c + y1 * sn;
            y1 = z1;
            y2 = z2;
          }
          o1[e] = (T)y1;
          o2[e] = (T)y2;
        }
        T* dst = nullptr;
        if (kind == 0)
          dst = (T*)epi.q + ((int64_t)row * Hq + head) * D + d;
        else if (sl[u] >= 0)
          dst = cache + (((int64_t)sl[u] * Hkv + kvh) * epi.max_seq + tr[u]) * D + d;
        if (row < M && col_ok && dst) {
          *(T4*)dst = o1;
          *(T4*)(dst + half) = o2;
        }
      }
    }
  }
}

template <int BM, int BN, int WGM, int WGN, int EK, int S = 2, int SH = 32>
__global__ __launch_bounds__(WGM * WGN * 64, 1) void gemm_kernel(const bf16* __restrict__ A, int lda,
                                                   const bf16* __restrict__ B, int ldb, int M,
                                                   int N, int K, int kc, Epi epi,
                                                   int tiles_m, int tiles_n, int full,
                                                   int tsplit, float* __restrict__ tail) {
  using ML = Mainloop<BM, BN, WGM, WGN, S, SH>;
  using Geo = AccGeo<SH, ML::MI, ML::NI>;
  constexpr int NW = ML::NW, WM = ML::WM, WN = ML::WN, MI = ML::MI, NI = ML::NI;
  constexpr int KIND = EK & kEpiKindMask;
  constexpr bool F32 = (EK & kEpiF32) != 0;
  extern __shared__ __align__(16) char smem_raw[];
  GemmSmem<BM, BN, S>& sm = *reinterpret_cast<GemmSmem<BM, BN, S>*>(smem_raw);

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wv / WGN, wn = wv % WGN;
  // Blocks [0, full) run whole tiles (ids 0 .. full-1 of the grouped order);
  // the ones after it run the last tiles in `tsplit` K-splits each (fp32
  // partials to `tail`), so that a final partial round fills every CU.
  // Half-tile mode (tsplit == 0, 128-row tiles): the grid covers the last
  // tiles of a 256-row grid (tiles_m of 256 rows, ids from `full`) as two
  // 128-row halves each, over the whole K; the two halves of a tile are
  // consecutive ids, so the XCD remap keeps them in one L2.
  int tm, tn, u = -1;
  if (BM == 128 && tsplit == 0) {
    const int id = xcd_id(blockIdx.x, (int)gridDim.x);
    tile_of_id(full + id / 2, tiles_m, tiles_n, tm, tn);
    tm = 2 * tm + (id & 1);
    if (tm * BM >= M) return;  // the empty half of a last M-tile
  } else if ((int)blockIdx.x < full) {
    tile_of_id(xcd_id(blockIdx.x, full), tiles_m, tiles_n, tm, tn);
  } else {
    u = blockIdx.x - full;
    tile_of_id(full + u / tsplit, tiles_m, tiles_n, tm, tn);
    kc = cdiv(K / kBK, tsplit) * kBK;  // the last split takes the remainder
  }
  const int n_rows_b = KIND == EPI_SWIGLU ? 2 * epi.ffn : N;
  // Split-K (fp32 partial output only): split z covers k in [z kc, z kc + kc)
  // and writes plane z of the output.
  const int k0 = (u >= 0 ? u % tsplit : (int)blockIdx.y) * kc;
  K = min(kc, K - k0);
  A += k0;
  B += k0;

  // Buffer descriptors: rows past the end of A or B read as zero.
  const __amdgpu_buffer_rsrc_t rsrc_a = __builtin_amdgcn_make_buffer_rsrc(
      (void*)A, (short)0, (int)((int64_t)M * lda * 2 - (int64_t)k0 * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsrc_b = __builtin_amdgcn_make_buffer_rsrc(
      (void*)B, (short)0, (int)((int64_t)n_rows_b * ldb * 2 - (int64_t)k0 * 2), 0x00020000);
  // Global -> LDS without registers: each buffer_load_dwordx4 ... lds writes the
  // 64 lanes' 16 bytes to 1 KB of LDS in lane order, i.e. 8 tile rows.  Lane l
  // fills physical chunk l % 8 of row 8 b + l / 8 of its block b, so it fetches
  // the logical chunk swz(row, l % 8) of that row (swz is an involution).
  const int lrow = lane >> 3;
  uint32_t a_off[ML::A_BLK], b_off[ML::B_BLK];
#pragma unroll
  for (int j = 0; j < ML::A_BLK; ++j) {
    const int tr = (wv + NW * j) * 8 + lrow;  // tile row
    const int gr = tm * BM + tr;
    a_off[j] = gr < M ? (uint32_t)(((int64_t)gr * lda + swz(tr, lane & 7) * 8) * 2) : 0x80000000u;
  }
#pragma unroll
  for (int j = 0; j < ML::B_BLK; ++j) {
    const int tr = (wv + NW * j) * 8 + lrow;
    const int gr = b_row_of<BN, WN>(KIND, tn, tr, epi.ffn);
    b_off[j] = gr < n_rows_b ? (uint32_t)(((int64_t)gr * ldb + swz(tr, lane & 7) * 8) * 2) : 0x80000000u;
  }
  typename ML::acc_t acc[MI][NI];
  const int lr = Geo::lane_row(lane), lc = Geo::lane_col(lane);
  // bf16 residual epilogue of a whole 256 x 256 tile: prefetch the residual
  // into the LDS buffers freed by the last two k-tiles (ResPf)
  constexpr bool kResPf = KIND == EPI_RESID && !F32 && BM == 256 && BN == 256 && S == 2 &&
                          NW == 8;
  // The descriptor is built unconditionally (only `on` depends on the split):
  // a descriptor assigned under a run-time branch ends up in private memory,
  // and a kernel with a private segment slows every later dispatch on its
  // queue.
  ResPf rp{};
  if constexpr (kResPf) {
    const int ld_bytes = epi.ldr * 2;
    rp = ResPf{__builtin_amdgcn_make_buffer_rsrc(
                   (void*)((const bf16*)epi.resid + (int64_t)tm * BM * epi.ldr + tn * BN),
                   (short)0, (int)((int64_t)(M - tm * BM) * ld_bytes), 0x00020000),
               (uint32_t)((lane >> 5) * ld_bytes +
                          (((lane & 31) ^ ((2 * wv + (lane >> 5)) & 15)) << 4)),
               ld_bytes, u < 0 && K / kBK >= 2};
  }
  ML::template run_valid<MI, kResPf>(M - tm * BM, sm, rsrc_a, a_off, rsrc_b, b_off, K, wv, lane,
                                     acc, rp);

  if (u >= 0) {  // tail split: the tile's fp32 partial sums, [BM][BN]
    Epi e{};
    e.out = tail + (int64_t)u * BM * BN;
    e.ldo = BN;
    plain_epilogue<SH, MI, NI, EPI_STORE_F32>(acc, e, wm * WM + lr, BM, wn * WN + lc, BN);
    return;
  }
  const int row0 = tm * BM + wm * WM + lr;
  if constexpr (KIND == EPI_STORE_F32) {
    Epi e = epi;
    e.out = (float*)epi.out + (int64_t)blockIdx.y * M * epi.ldo;
    plain_epilogue<SH, MI, NI, EK>(acc, e, row0, M, tn * BN + wn * WN + lc, N);
  } else if constexpr (KIND == EPI_STORE || KIND == EPI_RESID) {
    if constexpr (kResPf) {
      if (rp.on) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();  // every wave's residual pieces have landed
        resid_lds_epilogue<SH, MI, NI>(acc, epi, row0, M, tn * BN + wn * WN + lc, N, smem_raw,
                                       (K / kBK) & 1, wm * WM + lr, wn * WN + lc);
        return;
      }
    }
    plain_epilogue<SH, MI, NI, EK>(acc, epi, row0, M, tn * BN + wn * WN + lc, N);
  } else if constexpr (KIND == EPI_SWIGLU) {
    swiglu_epilogue<SH, MI, NI, F32>(acc, epi, row0, M, tn * (BN / 2) + wn * (WN / 2) + lc);
  } else if constexpr (KIND == EPI_QKV_NORM) {
    static_assert(NW * SH * WN * sizeof(float) <= sizeof(GemmSmem<BM, BN>),
                  "the epilogue's row blocks must fit the mainloop's LDS");
    qkv_norm_epilogue<SH, MI, NI, F32>(acc, epi, smem_raw, wv, lane, tm * BM + wm * WM,
                                       tn * BN + wn * WN, M, N);
  } else if (epi.head_dim == 128) {
    qkv_epilogue<SH, MI, NI, 2, F32>(acc, epi, row0, tn * BN + wn * WN + lc, M, N);
  } else {
    qkv_epilogue<SH, MI, NI, 1, F32>(acc, epi, row0, tn * BN + wn * WN + lc, M, N);
  }
}

// Grouped expert GEMM.  Rows [seg[e], seg[e+1]) of the routed order belong to
// expert e; tile_off[e] .. tile_off[e+1]-1 are its M-tiles (BM rows each).  For
// the gate/up pass (EPI_SWIGLU) A row p is token perm[p] / top_k of A; for the
// down pass (EPI_STORE_F32) A row p is row p of A.  B of expert e starts at
// B + e * b_stride elements.  Output row = routed position p.
template <int BM, int BN, int WGM, int WGN, int EK, int SH = 32>
__global__ __launch_bounds__(WGM * WGN * 64) void gemm_grouped_kernel(
    const bf16* __restrict__ A, int lda, int a_rows, const int32_t* __restrict__ perm, int top_k,
    const bf16* __restrict__ B, int64_t b_stride, int N, int K,
    const int32_t* __restrict__ seg, const int32_t* __restrict__ tile_off, int n_experts,
    int tiles_n, Epi epi) {
  using ML = Mainloop<BM, BN, WGM, WGN, 2, SH>;
  using Geo = AccGeo<SH, ML::MI, ML::NI>;
  constexpr int NW = ML::NW, WM = ML::WM, WN = ML::WN, MI = ML::MI, NI = ML::NI;
  constexpr int KIND = EK & kEpiKindMask;
  constexpr bool F32 = (EK & kEpiF32) != 0;
  extern __shared__ __align__(16) char smem_raw[];
  GemmSmem<BM, BN>& sm = *reinterpret_cast<GemmSmem<BM, BN>*>(smem_raw);

  // The real tiles (tile_off[E] M-tiles x tiles_n) are dealt to the XCDs in
  // contiguous shares (block b runs on XCD b % 8), so an expert's M-tiles run
  // side by side on one XCD and share its weight k-slices in that L2;
  // surplus blocks exit.
  const int total = tile_off[n_experts] * tiles_n;
  const int xcd = blockIdx.x % kXcds, loc = blockIdx.x / kXcds;
  const int per = total / kXcds, rem = total % kXcds;
  if (loc >= per + (xcd < rem ? 1 : 0)) return;  // surplus block
  const int id = xcd * per + min(xcd, rem) + loc;
  const int tn = id % tiles_n, mt = id / tiles_n;
  int lo = 0, hi = n_experts;             // expert e with tile_off[e] <= mt < tile_off[e+1]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (tile_off[mid] <= mt) lo = mid; else hi = mid;
  }
  const int e = lo;
  const int p0 = seg[e] + (mt - tile_off[e]) * BM;  // first routed row of this tile
  const int p_end = seg[e + 1];
  const int n_rows_b = KIND == EPI_SWIGLU ? 2 * epi.ffn : N;

  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wv / WGN, wn = wv % WGN;
  const __amdgpu_buffer_rsrc_t rsrc_a =
      __builtin_amdgcn_make_buffer_rsrc((void*)A, (short)0, (int)((int64_t)a_rows * lda * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsrc_b = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(B + (int64_t)e * b_stride), (short)0, (int)((int64_t)n_rows_b * K * 2), 0x00020000);
  const int lrow = lane >> 3;
  uint32_t a_off[ML::A_BLK], b_off[ML::B_BLK];
#pragma unroll
  for (int j = 0; j < ML::A_BLK; ++j) {
    const int tr = (wv + NW * j) * 8 + lrow;
    const int p = p0 + tr;
    int src = -1;
    if (p < p_end) src = perm ? perm[p] / top_k : p;
    a_off[j] = (src >= 0 && src < a_rows)
                   ? (uint32_t)(((int64_t)src * lda + swz(tr, lane & 7) * 8) * 2)
                   : 0x80000000u;
  }
#pragma unroll
  for (int j = 0; j < ML::B_BLK; ++j) {
    const int tr = (wv + NW * j) * 8 + lrow;
    const int gr = b_row_of<BN, WN>(KIND, tn, tr, epi.ffn);
    b_off[j] = gr < n_rows_b ? (uint32_t)(((int64_t)gr * K + swz(tr, lane & 7) * 8) * 2) : 0x80000000u;
  }
  typename ML::acc_t acc[MI][NI];
  // Short-row tiles (decode) stream their weights at HBM rate with every
  // workgroup in flight at once; started at the same k-tile, all of them
  // would read at one offset modulo the weight row (4 KB rows for H = 2048),
  // so each rotates its k-loop by its own amount.  The prefill down
  // projection (fp32 output) gains from it too; the prefill gate/up, whose
  // tiles of one expert share their k-slices in L2, does not.
  const bool rotate = BM <= 32 || KIND == EPI_STORE_F32;
  const int kshift = rotate ? (int)(((unsigned)id * 7u) % (unsigned)(K / kBK)) : 0;
  ML::run_valid(p_end - p0, sm, rsrc_a, a_off, rsrc_b, b_off, K, wv, lane, acc, ResPf{}, kshift);

  const int lr = Geo::lane_row(lane), lc = Geo::lane_col(lane);
  const int row0 = p0 + wm * WM + lr;
  if constexpr (KIND == EPI_SWIGLU)
    swiglu_epilogue<SH, MI, NI, F32>(acc, epi, row0, p_end, tn * (BN / 2) + wn * (WN / 2) + lc);
  else
    plain_epilogue<SH, MI, NI, EK>(acc, epi, row0, p_end, tn * BN + wn * WN + lc, N);
}

template <typename Kern>
static hipError_t opt_in_lds(Kern k, size_t smem, bool& done) {
  if (done) return hipSuccess;  // one-time opt-in to > 64 KB of LDS
  hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)smem);
  if (e == hipSuccess) done = true;
  return e;
}

// splits > 1 only with EPI_STORE_F32 (plane z of epi.out holds split z); K
// must then be a multiple of 64 * splits.
template <int BM, int BN, int WGM, int WGN, int EK, int S = 2, int SH = 32>
static hipError_t run_gemm(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                           const Epi& epi, hipStream_t s, int splits = 1) {
  const int tiles_m = cdiv(M, BM);
  const int tiles_n = (EK & kEpiKindMask) == EPI_SWIGLU ? cdiv(epi.ffn, BN / 2) : cdiv(N, BN);
  const size_t smem = sizeof(GemmSmem<BM, BN, S>);
  static bool attr_set = false;
  hipError_t e = opt_in_lds(gemm_kernel<BM, BN, WGM, WGN, EK, S, SH>, smem, attr_set);
  if (e != hipSuccess) return e;
  const int kc = K / splits;
  gemm_kernel<BM, BN, WGM, WGN, EK, S, SH><<<dim3(tiles_m * tiles_n, splits), WGM * WGN * 64, smem, s>>>(
      (const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, kc, epi, tiles_m, tiles_n,
      tiles_m * tiles_n, 1, nullptr);
  return hipGetLastError();
}

// Tail split of a large GEMM: with 256 x 256 tiles, one workgroup per CU,
// the last (tiles % CUs) tiles -- all of them when there are fewer tiles than
// CUs -- would run as a partial round; split into `tsplit` K-parts they fill
// it.
int cu_count() {
  static int n = 0;
  if (n == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      n = v;
    else
      n = 256;
  }
  return n;
}

// Tiles of the final partial round: total % CUs, or all of them when the
// GEMM has fewer tiles than CUs.
static int tail_tiles(int total) {
  const int G = cu_count();
  return total > G ? total % G : (total == G ? 0 : total);
}

constexpr int kMaxTailSplit = 8;  // K-parts of a tail tile, at most

static int tail_split(int total, int K, int kind) {
  const int G = cu_count();
  const int rem = tail_tiles(total);
  if (kind == EPI_SWIGLU || rem == 0) return 1;
  // Split s covers k-tiles [s c, s c + c) with c = ceil(k-tiles / t), the
  // last one the remainder: every split must keep at least one k-tile.
  const int kt = K / kBK;
  int t = G / rem;
  if (t > kMaxTailSplit) t = kMaxTailSplit;
  while (t > 1 && (t - 1) * cdiv(kt, t) >= kt) --t;
  return t;
}

// Bound for every large GEMM: the tail tiles times their splits never exceed
// one round (the CU count) of 256 x 256 fp32 tiles.
size_t gemm_tail_bytes() { return (size_t)cu_count() * 256 * 256 * sizeof(float); }

// Sum of a tail tile's split partials in split order + the epilogue.
// Workgroup (j, chunk): tail tile j (id full + j of the grouped order),
// elements [chunk * 2048, chunk * 2048 + 2048) of the tile (rotary pairs for
// q/k/v), 8 per thread.  Each thread loads its 8 elements' values of one
// split plane together, then every operand of the epilogue, before any
// store: tsplit + 1 memory round trips instead of one per element.
constexpr int kTailChunk = 2048;
constexpr int kTailPer = kTailChunk / 256;

// QKV: the q/k/v instantiation (its own kernel, so that the plain path's
// registers for every plane's values do not lower its occupancy).
template <int BM, int BN, bool F32, bool QKV>
__global__ __launch_bounds__(256) void tail_epi_kernel(const float* __restrict__ tail, int tsplit,
                                                       int full, int tiles_m, int tiles_n, int M,
                                                       int N, Epi epi) {
  using St = Store<F32>;
  using T = typename St::T;
  const int j = blockIdx.y;
  int tm, tn;
  tile_of_id(full + j, tiles_m, tiles_n, tm, tn);
  const float* __restrict__ tp = tail + (int64_t)j * tsplit * BM * BN;
  const int e0 = blockIdx.x * kTailChunk + threadIdx.x;
  if constexpr (!QKV) {
    int idx[kTailPer];
    float v[kTailPer];
#pragma unroll
    for (int q = 0; q < kTailPer; ++q) {
      idx[q] = min(e0 + 256 * q, BM * BN - 1);
      v[q] = 0.f;
    }
    // every plane's values are loaded before the ordered sum (tsplit <=
    // kMaxTailSplit, a uniform bound), so the loads are in flight together
    float pv[kMaxTailSplit][kTailPer];
#pragma unroll
    for (int sp = 0; sp < kMaxTailSplit; ++sp)
#pragma unroll
      for (int q = 0; q < kTailPer; ++q)
        pv[sp][q] = sp < tsplit ? tp[(int64_t)sp * BM * BN + idx[q]] : 0.f;
#pragma unroll
    for (int sp = 0; sp < kMaxTailSplit; ++sp)
#pragma unroll
      for (int q = 0; q < kTailPer; ++q)
        if (sp < tsplit) v[q] += pv[sp][q];
    float res[kTailPer];
    if (epi.kind == EPI_RESID) {
#pragma unroll
      for (int q = 0; q < kTailPer; ++q) {
        const int row = min(tm * BM + idx[q] / BN, M - 1), col = min(tn * BN + idx[q] % BN, N - 1);
        res[q] = St::ld(epi.resid, (int64_t)row * epi.ldr + col);
      }
    }
#pragma unroll
    for (int q = 0; q < kTailPer; ++q) {
      const int e = e0 + 256 * q;
      const int row = tm * BM + e / BN, col = tn * BN + e % BN;
      if (e >= BM * BN || row >= M || col >= N) continue;
      if (epi.kind == EPI_STORE_F32) {
        ((float*)epi.out)[(int64_t)row * epi.ldo + col] = v[q];
      } else {
        const float o = epi.kind == EPI_RESID ? v[q] + res[q] : v[q];
        St::st(epi.out, (int64_t)row * epi.ldo + col, o);
      }
    }
    return;
  } else {
    // q/k/v + bias + RoPE + cache write: one thread per rotary pair (a head of
    // D columns lies inside one tile since BN is a multiple of D).
    const int Dh = epi.head_dim, half = Dh / 2;
    const int Hq = epi.n_q_heads, Hkv = epi.n_kv_heads;
    int rr[kTailPer], cc[kTailPer];
    float x1[kTailPer], x2[kTailPer];
#pragma unroll
    for (int q = 0; q < kTailPer; ++q) {
      const int e = min(e0 + 256 * q, BM * (BN / 2) - 1);
      const int pc = e % (BN / 2);
      rr[q] = e / (BN / 2);
      cc[q] = (pc / half) * Dh + pc % half;  // first-half column in the tile
      x1[q] = x2[q] = 0.f;
    }
    // (plane by plane: loading every plane's pairs first needs twice the
    // registers of the plain path and was slower)
    for (int sp = 0; sp < tsplit; ++sp)
#pragma unroll
      for (int q = 0; q < kTailPer; ++q) {
        const float* pl = tp + (int64_t)sp * BM * BN + rr[q] * BN + cc[q];
        x1[q] += pl[0];
        x2[q] += pl[half];
      }
    float2 cs[kTailPer];
    int sl[kTailPer], tr[kTailPer];
    float b1[kTailPer], b2[kTailPer], g1[kTailPer], g2[kTailPer];
#pragma unroll
    for (int q = 0; q < kTailPer; ++q) {
      const int row = min(tm * BM + rr[q], M - 1), col = min(tn * BN + cc[q], N - 1);
      const int head = col / Dh, d = col % Dh;
      cs[q] = epi.rope[(int64_t)row * half + d];
      sl[q] = epi.tok_slot[row];
      tr[q] = epi.tok_row[row];
      b1[q] = epi.bias ? St::ld(epi.bias, col) : 0.f;
      b2[q] = epi.bias ? St::ld(epi.bias, col + half) : 0.f;
      const void* gp = head < Hq ? epi.q_norm : epi.k_norm;
      const bool n = epi.q_norm && head < Hq + Hkv;
      g1[q] = n ? St::ld(gp, d) : 1.f;
      g2[q] = n ? St::ld(gp, d + half) : 1.f;
    }
    // Per-head RMSNorm of q and k: a head's rotary pairs are `half` consecutive
    // elements, an aligned group of lanes, so its sum of squares is a group sum.
    float rs[kTailPer];
#pragma unroll
    for (int q = 0; q < kTailPer; ++q) {
      x1[q] += b1[q];
      x2[q] += b2[q];
      rs[q] = 1.f;
      if (epi.q_norm) {
        const float ss = group_sum(x1[q] * x1[q] + x2[q] * x2[q], half);
        rs[q] = 1.0f / sqrtf(ss / (float)Dh + epi.eps);
      }
    }
#pragma unroll
    for (int q = 0; q < kTailPer; ++q) {
      const int row = tm * BM + rr[q], col = tn * BN + cc[q];
      if (e0 + 256 * q >= BM * (BN / 2) || row >= M || col >= N) continue;
      const int head = col / Dh, d = col % Dh;
      float y1 = x1[q], y2 = x2[q];
      if (head < Hq + Hkv) {
        y1 *= rs[q] * g1[q];
        y2 *= rs[q] * g2[q];
        const float r1 = y1 * cs[q].x - y2 * cs[q].y;
        const float r2 = y2 * cs[q].x + y1 * cs[q].y;
        y1 = r1;
        y2 = r2;
      }
      T* dst;
      if (head < Hq) {
        dst = (T*)epi.q + ((int64_t)row * Hq + head) * Dh + d;
      } else {
        if (sl[q] < 0) continue;
        const int kvh = head < Hq + Hkv ? head - Hq : head - Hq - Hkv;
        T* cache = (T*)(head < Hq + Hkv ? epi.kc : epi.vc);
        dst = cache + (((int64_t)sl[q] * Hkv + kvh) * epi.max_seq + tr[q]) * Dh + d;
      }
      dst[0] = (T)y1;
      dst[half] = (T)y2;
    }
  }
}

template <int BM, int BN, int WGM, int WGN, int EK, int SH = 32>
static hipError_t run_gemm_tail(const void* A, int lda, const void* B, int ldb, int M, int N,
                                int K, const Epi& epi, float* tail, hipStream_t s) {
  constexpr int KIND = EK & kEpiKindMask;
  const int tiles_m = cdiv(M, BM);
  const int tiles_n = KIND == EPI_SWIGLU ? cdiv(epi.ffn, BN / 2) : cdiv(N, BN);
  const int total = tiles_m * tiles_n;
  const int t = tail ? tail_split(total, K, KIND) : 1;
  if (t == 1) return run_gemm<BM, BN, WGM, WGN, EK, 2, SH>(A, lda, B, ldb, M, N, K, epi, s);
  const int n_tail = tail_tiles(total);
  const int full = total - n_tail;
  const size_t smem = sizeof(GemmSmem<BM, BN>);
  static bool attr_set = false;
  hipError_t e = opt_in_lds(gemm_kernel<BM, BN, WGM, WGN, EK, 2, SH>, smem, attr_set);
  if (e != hipSuccess) return e;
  // A tail split in two or three (a final round a quarter to a half full), or
  // in four over a short K, of a bf16-output 256 x 256 GEMM runs instead as
  // 128-row halves of the tail tiles over the whole K: the same round of work
  // (or a little more) with no fp32 partials and no reduction kernel.
  constexpr bool kHalfOk = BM == 256 && BN == 256 && !(EK & kEpiF32) &&
                           (KIND == EPI_STORE || KIND == EPI_RESID || KIND == EPI_QKV ||
                            KIND == EPI_QKV_NORM);
  if constexpr (kHalfOk) {
    if (t <= 3 || (t == 4 && K <= 4096)) {
      if (full > 0) {
        gemm_kernel<BM, BN, WGM, WGN, EK, 2, SH><<<full, WGM * WGN * 64, smem, s>>>(
            (const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, K, epi, tiles_m, tiles_n, full, 1,
            nullptr);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
      }
      // q/k/v keep 128 columns per wave (rotary pairs); the others 64 x 64 waves
      constexpr int HM = (KIND == EPI_QKV || KIND == EPI_QKV_NORM) ? 4 : 2;
      const size_t hsmem = sizeof(GemmSmem<128, 256, 3>);
      static bool half_attr = false;
      e = opt_in_lds(gemm_kernel<128, 256, HM, 8 / HM, EK, 3, kMidSH>, hsmem, half_attr);
      if (e != hipSuccess) return e;
      gemm_kernel<128, 256, HM, 8 / HM, EK, 3, kMidSH><<<2 * n_tail, 512, hsmem, s>>>(
          (const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, K, epi, tiles_m, tiles_n, full, 0,
          nullptr);
      return hipGetLastError();
    }
  }
  gemm_kernel<BM, BN, WGM, WGN, EK, 2, SH><<<full + n_tail * t, WGM * WGN * 64, smem, s>>>(
      (const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, K, epi, tiles_m, tiles_n, full, t, tail);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int elems = KIND == EPI_QKV || KIND == EPI_QKV_NORM ? BM * BN / 2 : BM * BN;
  constexpr bool kQkv = KIND == EPI_QKV || KIND == EPI_QKV_NORM;
  tail_epi_kernel<BM, BN, (EK & kEpiF32) != 0, kQkv>
      <<<dim3(cdiv(elems, kTailChunk), n_tail), 256, 0, s>>>(tail, t, full, tiles_m, tiles_n, M,
                                                             N, epi);
  return hipGetLastError();
}

hipError_t launch_gemm(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                       const Epi& epi, float* tail, hipStream_t s) {
  if (M == 0) return hipSuccess;
  if (epi.f32) {
    constexpr int F = kEpiF32;
    switch (epi.kind) {
      case EPI_RESID:
        return run_gemm_tail<256, 256, 4, 2, EPI_RESID | F, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, tail, s);
      case EPI_SWIGLU: return run_gemm<256, 256, 4, 2, EPI_SWIGLU | F, 2, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, s);
      case EPI_STORE_F32:
        return run_gemm_tail<256, 256, 4, 2, EPI_STORE_F32, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, tail, s);
      case EPI_QKV:
        if (epi.q_norm)
          return run_gemm_tail<256, 256, 4, 2, EPI_QKV_NORM | F, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, tail, s);
        return run_gemm_tail<256, 256, 4, 2, EPI_QKV | F, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, tail, s);
      default: return hipErrorInvalidValue;
    }
  }
  // Mid-size M (a chunk of a few hundred tokens, the mixed step): when the
  // 256 x 256 tiles would not fill one round of CUs, 128 x 128 tiles of four
  // 32 x 128 waves with three LDS stages (two k-tiles in flight): a short
  // k-tile of a small tile computes in less time than a load's round trip,
  // so two stages leave such a GEMM bound by load latency.  The waves keep
  // 128 columns (the q/k/v epilogue pairs rotary halves inside a wave).
  // gate/up at M <= 640: 128 x 256 tiles with three stages (its 256-row
  // tiles leave most of a third tile empty).  A long K (the down
  // projection) keeps the 256 x 256 tail split.
  if (epi.kind != EPI_SWIGLU && epi.kind != EPI_STORE_F32 && K <= 8192 &&
      cdiv(M, 256) * cdiv(N, 256) < cu_count()) {
    // Plain and residual stores (no rotary pairs) take 128 x 256 tiles of
    // eight 64 x 64 waves when those fill one round of CUs at least three
    // quarters full: a 4096-token O projection is one round of 256 such tiles
    // instead of two rounds of 128 x 128.
    const int t256 = cdiv(M, 128) * cdiv(N, 256);
    if ((epi.kind == EPI_STORE || epi.kind == EPI_RESID) && t256 <= cu_count() &&
        4 * t256 >= 3 * cu_count()) {
      if (epi.kind == EPI_STORE)
        return run_gemm<128, 256, 2, 4, EPI_STORE, 3, kMidSH>(A, lda, B, ldb, M, N, K, epi, s);
      return run_gemm<128, 256, 2, 4, EPI_RESID, 3, kMidSH>(A, lda, B, ldb, M, N, K, epi, s);
    }
    switch (epi.kind) {
      case EPI_STORE: return run_gemm<128, 128, 4, 1, EPI_STORE, 3, kMidSH>(A, lda, B, ldb, M, N, K, epi, s);
      case EPI_RESID: return run_gemm<128, 128, 4, 1, EPI_RESID, 3, kMidSH>(A, lda, B, ldb, M, N, K, epi, s);
      default:
        if (epi.q_norm)
          return run_gemm<128, 128, 4, 1, EPI_QKV_NORM, 3, kMidSH>(A, lda, B, ldb, M, N, K, epi, s);
        return run_gemm<128, 128, 4, 1, EPI_QKV, 3, kMidSH>(A, lda, B, ldb, M, N, K, epi, s);
    }
  }
  if (epi.kind == EPI_SWIGLU && M <= 640)
    return run_gemm<128, 256, 2, 4, EPI_SWIGLU, 3, kMidSH>(A, lda, B, ldb, M, N, K, epi, s);
  switch (epi.kind) {
    case EPI_STORE: return run_gemm_tail<256, 256, 4, 2, EPI_STORE, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, tail, s);
    case EPI_RESID: return run_gemm_tail<256, 256, 4, 2, EPI_RESID, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, tail, s);
    case EPI_SWIGLU: return run_gemm<256, 256, 4, 2, EPI_SWIGLU, 2, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, s);
    case EPI_STORE_F32: return run_gemm_tail<256, 256, 4, 2, EPI_STORE_F32, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, tail, s);
    default:
      if (epi.q_norm)
        return run_gemm_tail<256, 256, 4, 2, EPI_QKV_NORM, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, tail, s);
      return run_gemm_tail<256, 256, 4, 2, EPI_QKV, kPrefillSH>(A, lda, B, ldb, M, N, K, epi, tail, s);
  }
}

// Rows per grouped-GEMM tile from the mean rows per expert: skinny tiles when
// experts see few rows (decode), the prefill GEMM's 256 x 256 tiles when they
// see ~224 or more (the 4 x 1024-token MoE prefill: gate/up 290 against
// 310-360 us with 128-row tiles, down 208 against 230-245 us).
int moe_tile_rows(int n_pairs, int n_experts) {
  if (n_pairs <= 48 * n_experts) return 32;
  return n_pairs >= 224 * n_experts ? 256 : 128;
}

template <int BM, int BN, int WGM, int WGN, int EK, int SH = 32>
static hipError_t run_grouped(const void* A, int lda, int a_rows, const int32_t* perm, int top_k,
                              const void* B, int64_t b_stride, int N, int K, const int32_t* seg,
                              const int32_t* tile_off, int n_experts, int max_tiles_m,
                              const Epi& epi, hipStream_t s) {
  const int tiles_n = (EK & kEpiKindMask) == EPI_SWIGLU ? cdiv(epi.ffn, BN / 2) : cdiv(N, BN);
  const size_t smem = sizeof(GemmSmem<BM, BN>);
  static bool attr_set = false;
  hipError_t e = opt_in_lds(gemm_grouped_kernel<BM, BN, WGM, WGN, EK, SH>, smem, attr_set);
  if (e != hipSuccess) return e;
  gemm_grouped_kernel<BM, BN, WGM, WGN, EK, SH><<<max_tiles_m * tiles_n, WGM * WGN * 64, smem, s>>>(
      (const bf16*)A, lda, a_rows, perm, top_k, (const bf16*)B, b_stride, N, K, seg, tile_off,
      n_experts, tiles_n, epi);
  return hipGetLastError();
}

hipError_t launch_gemm_grouped(const void* A, int lda, int a_rows, const int32_t* perm, int top_k,
                               const void* B, int64_t b_stride, int N, int K, const int32_t* seg,
                               const int32_t* tile_off, int n_experts, int n_pairs,
                               const Epi& epi, hipStream_t s) {
  if (n_pairs == 0) return hipSuccess;
  const int bm = moe_tile_rows(n_pairs, n_experts);
  const int max_tiles_m = cdiv(n_pairs, bm) + n_experts;  // each expert adds <= 1 partial tile
  if (epi.f32 && epi.kind == EPI_SWIGLU) {
    constexpr int EK = EPI_SWIGLU | kEpiF32;
    if (bm == 32)
      return run_grouped<32, 256, 1, 4, EK>(A, lda, a_rows, perm, top_k, B, b_stride, N, K, seg,
                                            tile_off, n_experts, max_tiles_m, epi, s);
    if (bm == 256)
      return run_grouped<256, 256, 4, 2, EK, kPrefillSH>(A, lda, a_rows, perm, top_k, B, b_stride, N, K, seg,
                                             tile_off, n_experts, max_tiles_m, epi, s);
    return run_grouped<128, 256, 2, 4, EK, kPrefillSH>(A, lda, a_rows, perm, top_k, B, b_stride, N, K, seg,
                                           tile_off, n_experts, max_tiles_m, epi, s);
  }
  if (bm == 32) {
    if (epi.kind == EPI_SWIGLU)
      return run_grouped<32, 256, 1, 4, EPI_SWIGLU>(A, lda, a_rows, perm, top_k, B, b_stride, N, K,
                                                     seg, tile_off, n_experts, max_tiles_m, epi, s);
    return run_grouped<32, 256, 1, 4, EPI_STORE_F32>(A, lda, a_rows, perm, top_k, B, b_stride, N, K,
                                                      seg, tile_off, n_experts, max_tiles_m, epi, s);
  }
  if (bm == 256) {
    if (epi.kind == EPI_SWIGLU)
      return run_grouped<256, 256, 4, 2, EPI_SWIGLU, kPrefillSH>(A, lda, a_rows, perm, top_k, B, b_stride, N, K,
                                                      seg, tile_off, n_experts, max_tiles_m, epi, s);
    return run_grouped<256, 256, 4, 2, EPI_STORE_F32, kPrefillSH>(A, lda, a_rows, perm, top_k, B, b_stride, N,
                                                       K, seg, tile_off, n_experts, max_tiles_m, epi,
                                                       s);
  }
  if (epi.kind == EPI_SWIGLU)
    return run_grouped<128, 256, 2, 4, EPI_SWIGLU, kPrefillSH>(A, lda, a_rows, perm, top_k, B, b_stride, N, K,
                                                    seg, tile_off, n_experts, max_tiles_m, epi, s);
  return run_grouped<128, 256, 2, 4, EPI_STORE_F32, kPrefillSH>(A, lda, a_rows, perm, top_k, B, b_stride, N, K,
                                                     seg, tile_off, n_experts, max_tiles_m, epi, s);
}

// Split-K reduction: sum the fp32 partial planes [splits][M][N] in split
// order (deterministic) and apply the epilogue; one thread per output element
// (per intermediate column for SwiGLU, per rotary pair for q/k/v).
__global__ __launch_bounds__(256) void splitk_epi_kernel(const float* __restrict__ part,
                                                       int splits, int M, int N, Epi epi) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t MN = (int64_t)M * N;
  // All planes' values are loaded before the ordered sum (splits <= 16), so
  // the loads are in flight together.
  auto sum = [&](int row, int col) {
    const float* q = part + (int64_t)row * N + col;
    float t[16];
#pragma unroll
    for (int s = 0; s < 16; ++s) t[s] = s < splits ? q[s * MN] : 0.f;
    float v = 0.f;
#pragma unroll
    for (int s = 0; s < 16; ++s) v += t[s];
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
    // lanes past the end compute on a clamped pair (their group is whole:
    // M pairs is a multiple of half) and store nothing
    const bool live = gid < (int64_t)M * pairs;
    const int64_t g = live ? gid : (int64_t)M * pairs - 1;
    const int row = (int)(g / pairs), p = (int)(g % pairs);
    const int head = p / half, d = p % half;
    const int col = head * D + d;
    float x1 = sum(row, col), x2 = sum(row, col + half);
    if (epi.bias) {
      x1 += bf2f(((const bf16*)epi.bias)[col]);
      x2 += bf2f(((const bf16*)epi.bias)[col + half]);
    }
    if (epi.q_norm) {
      // per-head RMSNorm of q and k: a head's pairs are an aligned group of
      // `half` lanes (D / 2 = 32 or 64)
      const float ss = group_sum(x1 * x1 + x2 * x2, half);
      if (head < Hq + Hkv) {
        const bf16* gp = (const bf16*)(head < Hq ? epi.q_norm : epi.k_norm);
        const float r = 1.0f / sqrtf(ss / (float)D + epi.eps);
        x1 *= r * bf2f(gp[d]);
        x2 *= r * bf2f(gp[d + half]);
      }
    }
    if (!live) return;
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

// Split-K reduction fused with the residual add and the RMSNorm that follows
// it (the O projection of a short batch): one workgroup per row sums the
// planes in split order and adds the residual (x1, stored in bf16), then
// normalises the stored row into y = x1 / sqrt(mean(x1^2) + eps) * g.
constexpr int kNormRowThreads = 256;
constexpr int kNormRowChunks = 8;  // 4-float chunks per thread: N <= 256 * 4 * 8

__global__ __launch_bounds__(kNormRowThreads) void splitk_resid_norm_kernel(
    const float* __restrict__ part, int splits, int M, int N, const bf16* __restrict__ resid,
    int ldr, bf16* __restrict__ out, int ldo, const bf16* __restrict__ g, bf16* __restrict__ y,
    float eps) {
  const int row = blockIdx.x, tid = threadIdx.x;
  const int64_t MN = (int64_t)M * N;
  const int nch = N / 4;
  f32x4 v[kNormRowChunks];
  float res[kNormRowChunks][4], gg[kNormRowChunks][4];
  // Every operand of the row first (chunk indices clamped: no branch around
  // the loads), then the ordered plane sums.
#pragma unroll
  for (int c = 0; c < kNormRowChunks; ++c) {
    const int ch = min(tid + c * kNormRowThreads, nch - 1);
    const bf16* rp = resid + (int64_t)row * ldr + ch * 4;
    const bf16* gp = g + ch * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      res[c][e] = bf2f(rp[e]);
      gg[c][e] = bf2f(gp[e]);
    }
    v[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // planes in groups of four: a group's loads are in flight together, then
  // added in plane order
  for (int sp0 = 0; sp0 < splits; sp0 += 4) {
    f32x4 t[4][kNormRowChunks];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int c = 0; c < kNormRowChunks; ++c) {
        const int ch = min(tid + c * kNormRowThreads, nch - 1);
        const int sp = min(sp0 + j, splits - 1);  // past the last plane: re-read, dropped
        t[j][c] = *(const f32x4*)(part + sp * MN + (int64_t)row * N + ch * 4);
      }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int c = 0; c < kNormRowChunks; ++c)
        if (sp0 + j < splits) v[c] += t[j][c];
  }
  float ss = 0.f;
  bf16 x1[kNormRowChunks][4];
#pragma unroll
  for (int c = 0; c < kNormRowChunks; ++c) {
    const bool ok = tid + c * kNormRowThreads < nch;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x1[c][e] = f2bf(v[c][e] + res[c][e]);
      const float f = bf2f(x1[c][e]);
      if (ok) ss += f * f;
    }
  }
  __shared__ float red[kNormRowThreads / 64];
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  ss = 0.f;
#pragma unroll
  for (int w = 0; w < kNormRowThreads / 64; ++w) ss += red[w];
  const float r = 1.0f / sqrtf(ss / (float)N + eps);
#pragma unroll
  for (int c = 0; c < kNormRowChunks; ++c) {
    const int ch = tid + c * kNormRowThreads;
    if (ch >= nch) continue;
    bf16x4 o, h;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[e] = x1[c][e];
      h[e] = f2bf(bf2f(x1[c][e]) * r * gg[c][e]);
    }
    *(bf16x4*)(out + (int64_t)row * ldo + ch * 4) = o;
    *(bf16x4*)(y + (int64_t)row * N + ch * 4) = h;
  }
}

// Decode projections (M <= 128 rows).  The arithmetic intensity is ~M flop
// per weight byte, so the weight stream from HBM sets the time: skinny
// 64 x 64 tiles (two or four waves) give ~600 workgroups on the large
// projections -- every one resident at once, each a short run of weight rows,
// which keeps the HBM pages streaming -- and split-K multiplies the
// workgroups of the narrow projections until ~200 are in flight.  Without a
// split the epilogue is fused; with one, fp32 partial planes go to the
// workspace and splitk_epi_kernel finishes.
// q/k/v always splits (its fused epilogue needs a whole head per wave).  The
// split runs of up to two workgroups per CU keep four k-tiles in LDS (three
// in flight), the rest two.  For q/k/v at 64 rows, 4 splits with four stages
// beat 8 with two: its partial planes are halved, and so is what they leave
// dirty in the caches just before the attention streams the KV cache.  Over
// 128-row tiles every split run likewise takes half the workgroups (~100)
// with three stages (two workgroups per CU): fewer partial planes ahead of
// the attention and of the weight streams that follow.
constexpr int kSkinnyBN = 64;

static int skinny_bm(int M) { return M <= 64 ? 64 : 128; }

int skinny_splits(int M, int N, int K, int kind) {
  const int tiles = cdiv(M, skinny_bm(M)) * cdiv(N, kSkinnyBN);
  const int target = M > 64 ? 100 : 200;
  int s = 1;
  while ((tiles * s < target || (kind == EPI_QKV && s == 1)) && s < 16 &&
         K % (kBK * 2 * s) == 0)
    s *= 2;
  return s;
}

// fp32 partial planes [splits][M][N] of a short batch.
static hipError_t run_skinny_planes(const void* A, int lda, const void* B, int ldb, int M, int N,
                                    int K, float* part, int splits, int kind, hipStream_t s) {
  Epi pe{};
  pe.kind = EPI_STORE_F32;
  pe.out = part;
  pe.ldo = N;
  if (M > 64) {
    if (cdiv(N, kSkinnyBN) * splits <= 2 * cu_count())
      return run_gemm<128, kSkinnyBN, 4, 1, EPI_STORE_F32, 3>(A, lda, B, ldb, M, N, K, pe, s, splits);
    return run_gemm<128, kSkinnyBN, 4, 1, EPI_STORE_F32>(A, lda, B, ldb, M, N, K, pe, s, splits);
  }
  if (cdiv(N, kSkinnyBN) * splits <= 2 * cu_count())
    return run_gemm<64, kSkinnyBN, 2, 1, EPI_STORE_F32, 4>(A, lda, B, ldb, M, N, K, pe, s, splits);
  return run_gemm<64, kSkinnyBN, 2, 1, EPI_STORE_F32>(A, lda, B, ldb, M, N, K, pe, s, splits);
}

size_t skinny_partial_bytes(int M, int N, int K, int kind) {
  const int s = skinny_splits(M, N, K, kind);
  return s > 1 ? (size_t)s * M * N * sizeof(float) : 0;
}

template <int BM, int WGM>
static hipError_t run_skinny(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                             const Epi& epi, float* part, int splits, hipStream_t s) {
  if (splits == 1) {
    switch (epi.kind) {
      case EPI_STORE: return run_gemm<BM, kSkinnyBN, WGM, 1, EPI_STORE>(A, lda, B, ldb, M, N, K, epi, s);
      case EPI_RESID: return run_gemm<BM, kSkinnyBN, WGM, 1, EPI_RESID>(A, lda, B, ldb, M, N, K, epi, s);
      case EPI_SWIGLU: return run_gemm<BM, kSkinnyBN, WGM, 1, EPI_SWIGLU>(A, lda, B, ldb, M, N, K, epi, s);
      case EPI_STORE_F32:
        return run_gemm<BM, kSkinnyBN, WGM, 1, EPI_STORE_F32>(A, lda, B, ldb, M, N, K, epi, s);
      default: return hipErrorInvalidValue;
    }
  }
  hipError_t e = run_skinny_planes(A, lda, B, ldb, M, N, K, part, splits, epi.kind, s);
  if (e != hipSuccess) return e;
  int64_t n_out;
  if (epi.kind == EPI_SWIGLU) n_out = (int64_t)M * epi.ffn;
  else if (epi.kind == EPI_QKV) n_out = (int64_t)M * (epi.n_q_heads + 2 * epi.n_kv_heads) * (epi.head_dim / 2);
  else n_out = (int64_t)M * N;
  splitk_epi_kernel<<<(unsigned)((n_out + 255) / 256), 256, 0, s>>>(part, splits, M, N, epi);
  return hipGetLastError();
}

hipError_t launch_skinny(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                         const Epi& epi, float* part, hipStream_t s) {
  if (M == 0) return hipSuccess;
  const int splits = skinny_splits(M, N, K, epi.kind);
  if (splits == 1 && epi.kind == EPI_QKV) return launch_gemm(A, lda, B, ldb, M, N, K, epi, nullptr, s);
  if (M <= 64) return run_skinny<64, 2>(A, lda, B, ldb, M, N, K, epi, part, splits, s);
  return run_skinny<128, 4>(A, lda, B, ldb, M, N, K, epi, part, splits, s);
}

bool skinny_resid_norm_fused(int M, int N, int K) {
  return M <= 128 && M > 0 && N % 4 == 0 && N <= kNormRowThreads * 4 * kNormRowChunks &&
         skinny_splits(M, N, K, EPI_RESID) > 1;
}

hipError_t launch_skinny_resid_norm(const void* A, int lda, const void* B, int ldb, int M, int N,
                                    int K, const void* resid, int ldr, void* out, int ldo,
                                    const void* g, void* y, float eps, float* part, hipStream_t s) {
  if (M == 0) return hipSuccess;
  const int splits = skinny_splits(M, N, K, EPI_RESID);
  hipError_t e = run_skinny_planes(A, lda, B, ldb, M, N, K, part, splits, EPI_RESID, s);
  if (e != hipSuccess) return e;
  splitk_resid_norm_kernel<<<M, kNormRowThreads, 0, s>>>(part, splits, M, N, (const bf16*)resid,
                                                        ldr, (bf16*)out, ldo, (const bf16*)g,
                                                        (bf16*)y, eps);
  return hipGetLastError();
}

int gemm_planes_splits(int M, int N, int K) {
  const int tiles = cdiv(M, 64) * cdiv(N, kSkinnyBN);
  int s = 1;
  while (tiles * s < 400 && s < 16 && K % (kBK * 2 * s) == 0) s *= 2;
  return s;
}

hipError_t launch_gemm_planes(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                              float* planes, int splits, hipStream_t s) {
  if (M == 0) return hipSuccess;
  Epi pe{};
  pe.kind = EPI_STORE_F32;
  pe.out = planes;
  pe.ldo = N;
  return run_gemm<64, kSkinnyBN, 2, 1, EPI_STORE_F32>(A, lda, B, ldb, M, N, K, pe, s, splits);
}

}  // namespace tri
