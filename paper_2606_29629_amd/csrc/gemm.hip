// Prefill GEMM on the matrix cores: C[M,N] = A[M,K] B[N,K]^T, bf16 operands,
// fp32 accumulation, with the layer's epilogues fused (residual add, SwiGLU,
// q/k/v split + rotary embedding + KV-cache write).
//
// Both operands are K-contiguous ("nn.Linear" weights [out, in] and row-major
// activations), which is the native operand layout of v_mfma_f32_32x32x16_bf16:
// lane l supplies row (l % 32) and 8 consecutive k of slice (l / 32).
//
// Tiling: BM x BN x 64 block tile, WGM x WGN waves (8 = 4 x 2: two waves per
// SIMD, so one wave's LDS waits overlap the other's MFMAs), each wave a
// (BM/WGM) x (BN/WGN) sub-tile of 32x32 MFMA blocks.  A and B tiles are staged through LDS, double
// buffered, with 16-byte chunks XOR-swizzled (see swz) so that fragment reads
// are free of bank conflicts.  Tiles move from HBM to
// LDS with buffer_load_dwordx4 ... lds (no register staging); the loads of
// tile k+1 are in flight while the MFMAs of tile k run.
//
// Work distribution: workgroups are dispatched round-robin over the 8 XCDs;
// the linear block id is remapped so each XCD owns a contiguous range of
// tiles, walked in groups of 8 M-tiles so co-resident tiles share A and B
// panels in that XCD's L2.
#include "common.hpp"
#include "kernels.hpp"

namespace tri {

constexpr int kBK = 64;
constexpr int kChunks = kBK / 8;  // 16-byte chunks per tile row
constexpr int kGroupM = 8;
constexpr int kXcds = 8;

// LDS has 64 banks of 4 bytes (a 256-byte window).  A tile row is 128 bytes,
// so rows r and r+1 share a window; a ds_read_b128 phase of 16 lanes reads the
// same logical chunk of 16 consecutive rows.  XOR-ing the chunk with
// (row / 2) % 8 gives the 8 even and the 8 odd rows 8 distinct 16-byte slots
// each, i.e. all 16 slots of the window: no bank conflict.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }

// Tile index for this block: XCD-contiguous ranges, then grouped-M order.
__device__ __forceinline__ void tile_of_block(int bid, int tiles_m, int tiles_n, int& tm,
                                              int& tn) {
  const int total = tiles_m * tiles_n;
  const int per = total / kXcds, rem = total % kXcds;
  const int x = bid % kXcds, loc = bid / kXcds;
  const int id = x * per + min(x, rem) + loc;
  const int group = id / (kGroupM * tiles_n);
  const int first_m = group * kGroupM;
  const int gm = min(kGroupM, tiles_m - first_m);
  const int in = id - group * kGroupM * tiles_n;
  tm = first_m + in % gm;
  tn = in / gm;
}

template <int BM, int BN>
struct GemmSmem {
  bf16 a[2][BM * kBK];
  bf16 b[2][BN * kBK];
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

// q/k/v split + bias + rotary embedding + KV-cache write on the accumulators.
// HB = 32-column blocks per half head (D / 64): block j (first half of a head)
// pairs with block j + HB (second half), same lane, same element.
template <int MI, int NI, int HB>
__device__ __forceinline__ void qkv_epilogue(const f32x16 (&acc)[MI][NI], const Epi& epi,
                                             int row0, int col0, int M, int N) {
  constexpr int D = HB * 64, half = D / 2;
  const int Hq = epi.n_q_heads, Hkv = epi.n_kv_heads;
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    if ((j / HB) & 1) continue;
    const int col = col0 + 32 * j;  // first-half column
    if (col >= N) continue;
    const int head = col / D, d = col % D;
    float b1 = 0.f, b2 = 0.f;
    if (epi.bias) {
      b1 = bf2f(((const bf16*)epi.bias)[col]);
      b2 = bf2f(((const bf16*)epi.bias)[col + half]);
    }
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row0 + 32 * i + 8 * (r >> 2) + (r & 3);
        if (row >= M) continue;
        float x1 = acc[i][j][r] + b1, x2 = acc[i][j + HB][r] + b2;
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
          if (sl < 0) continue;
          const int kvh = head < Hq + Hkv ? head - Hq : head - Hq - Hkv;
          bf16* cache = (bf16*)(head < Hq + Hkv ? epi.kc : epi.vc);
          bf16* cp = cache + (((int64_t)sl * Hkv + kvh) * epi.max_seq + epi.tok_row[row]) * D + d;
          cp[0] = f2bf(x1);
          cp[half] = f2bf(x2);
        }
      }
  }
}

template <int BM, int BN, int WGM, int WGN, int EK>
__global__ __launch_bounds__(WGM * WGN * 64) void gemm_kernel(const bf16* __restrict__ A, int lda,
                                                   const bf16* __restrict__ B, int ldb, int M,
                                                   int N, int K, Epi epi, int tiles_m,
                                                   int tiles_n) {
  constexpr int NT = WGM * WGN * 64;        // threads
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int MI = WM / 32, NI = WN / 32;
  extern __shared__ __align__(16) char smem_raw[];
  GemmSmem<BM, BN>& sm = *reinterpret_cast<GemmSmem<BM, BN>*>(smem_raw);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  int tm, tn;
  tile_of_block(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int n_rows_b = EK == EPI_SWIGLU ? 2 * epi.ffn : N;

  // Buffer descriptors: rows past the end of A or B read as zero.
  const __amdgpu_buffer_rsrc_t rsrc_a =
      __builtin_amdgcn_make_buffer_rsrc((void*)A, (short)0, (int)((int64_t)M * lda * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t rsrc_b =
      __builtin_amdgcn_make_buffer_rsrc((void*)B, (short)0, (int)((int64_t)n_rows_b * ldb * 2), 0x00020000);
  // Global -> LDS without registers: each buffer_load_dwordx4 ... lds writes the
  // 64 lanes' 16 bytes to 1 KB of LDS in lane order, i.e. 8 tile rows.  Lane l
  // fills physical chunk l % 8 of row 8 b + l / 8 of its block b, so it fetches
  // the logical chunk swz(row, l % 8) of that row (swz is an involution).
  constexpr int NW = NT / 64;
  constexpr int A_BLK = BM / 8 / NW, B_BLK = BN / 8 / NW;  // 1 KB blocks per wave per tile
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int lrow = lane >> 3;
  uint32_t a_off[A_BLK], b_off[B_BLK];
#pragma unroll
  for (int j = 0; j < A_BLK; ++j) {
    const int tr = (wv + NW * j) * 8 + lrow;  // tile row
    const int gr = tm * BM + tr;
    a_off[j] = gr < M ? (uint32_t)(((int64_t)gr * lda + swz(tr, lane & 7) * 8) * 2) : 0x80000000u;
  }
#pragma unroll
  for (int j = 0; j < B_BLK; ++j) {
    const int tr = (wv + NW * j) * 8 + lrow;
    const int gr = b_row_of<BN, WN>(EK, tn, tr, epi.ffn);
    b_off[j] = gr < n_rows_b ? (uint32_t)(((int64_t)gr * ldb + swz(tr, lane & 7) * 8) * 2) : 0x80000000u;
  }

  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = f32x16{0.f};

  auto gload = [&](int kt, int buf) {
    const int kb = kt * kBK * 2;
#pragma unroll
    for (int j = 0; j < A_BLK; ++j)
      buffer_load_lds16(rsrc_a, &sm.a[buf][(wv + NW * j) * 8 * kBK], a_off[j], kb);
#pragma unroll
    for (int j = 0; j < B_BLK; ++j)
      buffer_load_lds16(rsrc_b, &sm.b[buf][(wv + NW * j) * 8 * kBK], b_off[j], kb);
  };

  const int KT = K / kBK;
  const int lr = lane & 31, lg = lane >> 5;
  gload(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) gload(kt + 1, buf ^ 1);  // lands in the other buffer meanwhile
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int ch = kk * 2 + lg;
      bf16x8 af[MI], bfr[NI];
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int r = wm * WM + i * 32 + lr;
        af[i] = *(const bf16x8*)&sm.a[buf][r * kBK + swz(r, ch) * 8];
      }
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int r = wn * WN + j * 32 + lr;
        bfr[j] = *(const bf16x8*)&sm.b[buf][r * kBK + swz(r, ch) * 8];
      }
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // Accumulator element r of block (i, j): row 32i + 8(r/4) + 4(lane/32) + r%4,
  // column 32j + lane%32 of the wave sub-tile.
  const int row0 = tm * BM + wm * WM + 4 * lg;
  if constexpr (EK == EPI_STORE || EK == EPI_RESID) {
    const int col0 = tn * BN + wn * WN + lr;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int col = col0 + 32 * j;
        if (col >= N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + 32 * i + 8 * (r >> 2) + (r & 3);
          if (row >= M) continue;
          float v = acc[i][j][r];
          if constexpr (EK == EPI_RESID)
            v += bf2f(((const bf16*)epi.resid)[(int64_t)row * epi.ldr + col]);
          ((bf16*)epi.out)[(int64_t)row * epi.ldo + col] = f2bf(v);
        }
      }
  } else if constexpr (EK == EPI_SWIGLU) {
    const int f0 = tn * (BN / 2) + wn * (WN / 2) + lr;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI / 2; ++j) {
        const int f = f0 + 32 * j;
        if (f >= epi.ffn) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = row0 + 32 * i + 8 * (r >> 2) + (r & 3);
          if (row >= M) continue;
          const float gt = acc[i][j][r], up = acc[i][j + NI / 2][r];
          ((bf16*)epi.out)[(int64_t)row * epi.ldo + f] = f2bf(silu(gt) * up);
        }
      }
  } else if (epi.head_dim == 128) {
    qkv_epilogue<MI, NI, 2>(acc, epi, tm * BM + wm * WM + 4 * lg, tn * BN + wn * WN + lr, M, N);
  } else {
    qkv_epilogue<MI, NI, 1>(acc, epi, tm * BM + wm * WM + 4 * lg, tn * BN + wn * WN + lr, M, N);
  }
}

template <int BM, int BN, int WGM, int WGN, int EK>
static hipError_t run_gemm(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                           const Epi& epi, hipStream_t s) {
  const int tiles_m = cdiv(M, BM);
  const int tiles_n = EK == EPI_SWIGLU ? cdiv(epi.ffn, BN / 2) : cdiv(N, BN);
  const size_t smem = sizeof(GemmSmem<BM, BN>);
  static bool attr_set = false;  // one-time opt-in to > 64 KB of LDS
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)gemm_kernel<BM, BN, WGM, WGN, EK>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  gemm_kernel<BM, BN, WGM, WGN, EK><<<tiles_m * tiles_n, WGM * WGN * 64, smem, s>>>(
      (const bf16*)A, lda, (const bf16*)B, ldb, M, N, K, epi, tiles_m, tiles_n);
  return hipGetLastError();
}

hipError_t launch_gemm(const void* A, int lda, const void* B, int ldb, int M, int N, int K,
                       const Epi& epi, hipStream_t s) {
  if (M == 0) return hipSuccess;
  switch (epi.kind) {
    case EPI_STORE: return run_gemm<256, 256, 4, 2, EPI_STORE>(A, lda, B, ldb, M, N, K, epi, s);
    case EPI_RESID: return run_gemm<256, 256, 4, 2, EPI_RESID>(A, lda, B, ldb, M, N, K, epi, s);
    case EPI_SWIGLU: return run_gemm<256, 256, 4, 2, EPI_SWIGLU>(A, lda, B, ldb, M, N, K, epi, s);
    default: return run_gemm<256, 256, 4, 2, EPI_QKV>(A, lda, B, ldb, M, N, K, epi, s);
  }
}

}  // namespace tri
