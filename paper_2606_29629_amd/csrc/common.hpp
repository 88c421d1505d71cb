// Shared device helpers for the gfx950 (CDNA4) kernels of libtri.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tri {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16 v) { return (float)v; }
__device__ __forceinline__ bf16 f2bf(float v) { return (bf16)v; }  // RNE (v_cvt_pk_bf16_f32)
// bf16 -> fp16, saturating at the fp16 range (exact for 2^-14 <= |v| <= 65504).
__device__ __forceinline__ f16 bf2h_sat(bf16 v) {
  return (f16)fminf(fmaxf((float)v, -65504.f), 65504.f);
}

// 16-byte vector of 8 bf16 <-> raw 4 dwords.
union Pack8 {
  u32x4 u;
  bf16x8 h;
  bf16 e[8];
};

__device__ __forceinline__ u32x4 ldg16(const void* p) { return *(const u32x4*)p; }

// 16 bytes per lane from a buffer straight into LDS (buffer_load_dwordx4 ... lds):
// the wave's 64 lanes fill 1 KB at `lds` in lane order; `lds` must be
// wave-uniform.  Offsets at or past the buffer's size read as zero.
__device__ __forceinline__ void buffer_load_lds16(__amdgpu_buffer_rsrc_t r, void* lds,
                                                  uint32_t voffset, int soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16,
                                           voffset, soffset, 0, 0);
}
__device__ __forceinline__ void stg16(void* p, u32x4 v) { *(u32x4*)p = v; }

// Sum over aligned groups of `half` lanes (32 or 64).
__device__ __forceinline__ float group_sum(float v, int half) {
  v += __shfl_xor(v, 1, 64);
  v += __shfl_xor(v, 2, 64);
  v += __shfl_xor(v, 4, 64);
  v += __shfl_xor(v, 8, 64);
  v += __shfl_xor(v, 16, 64);
  if (half == 64) v += __shfl_xor(v, 32, 64);
  return v;
}

// Wave-level reductions (wave64) through cross-lane shuffles.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}
// Sum over aligned groups of 16 lanes (all lanes of a group receive the sum).
__device__ __forceinline__ float group16_sum(float v) {
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// z * sigmoid(z) with the hardware exp2 and reciprocal (about 1 ulp each).
__device__ __forceinline__ float silu(float z) {
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }


// ---- K/V tiles in LDS (attention).  Tile rows are one key's D values
// (D * 2 bytes); physical 16-byte chunk of logical chunk c in row r:
//  D = 128 (256-byte rows): c ^ g(r), g(r) = 4 (r % 4) + (r / 4) % 4.  g is a
//    bijection on 16 consecutive rows (a K fragment read: 16 rows, one chunk,
//    per 16-lane phase) and takes 4 distinct values of g / 4 on 4 aligned rows
//    (a transposing V read: 4 rows x 4 aligned chunks per 32 lanes).
//  D = 64 (128-byte rows, two per bank window): c ^ h(r / 2),
//    h(i) = 4 (i % 2) + (i / 2) % 4, distinct over the 8 rows of one parity
//    among 16, and differing in bit 2 between rows 4a and 4a + 2.
template <int D>
__device__ __forceinline__ int kv_chunk(int c, int r) {
  if constexpr (D == 128) return c ^ (((r & 3) << 2) | ((r >> 2) & 3));
  else return c ^ (((r & 2) << 1) | ((r >> 2) & 3));
}

typedef short s16x4 __attribute__((ext_vector_type(4)));

// ds_read_b64_tr_b16: within each group of 16 lanes, lane j receives element
// m = 0..3 from the 16-bit value at (address of lane 4 m + j / 4) + 2 (j % 4)
// bytes.  With the lanes of quad q pointing at 4 consecutive values of row q,
// lane j gets column j of those 4 rows: a 4 x 16 transpose.
__device__ __forceinline__ s16x4 lds_read_tr16(const bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
}


// Two fp32 -> packed bf16 pair (RNE, one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 v = {(bf16)a, (bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// Split of 8 fp32 values into bf16 hi + lo MFMA operands: hi = bf16(p)
// (RNE, packed in pairs), lo = bf16(p - hi) with the difference exact in
// fp32; hi + lo keeps ~16 significant bits of p.  Six VALU instructions per
// pair: two conversions, two unpacks (shift / mask) and two subtractions.
// (The packed pair goes through an empty asm first: otherwise the compiler
// rewrites the shift of its low half as a second conversion of p[2 i] alone
// plus the shift, one more instruction per pair.)
__device__ __forceinline__ void split_hilo8(const float (&p)[8], bf16x8& hi, bf16x8& lo) {
  u32x4 h, l;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t hv = pack_bf16x2(p[2 * i], p[2 * i + 1]);
    asm("" : "+v"(hv));
    h[i] = hv;
    l[i] = pack_bf16x2(p[2 * i] - __uint_as_float(hv << 16),
                       p[2 * i + 1] - __uint_as_float(hv & 0xffff0000u));
  }
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}

// Balanced reductions of a lane's values.  A dependent VALU result takes tens
// of cycles to come back, so a linear fold over n values is an n-deep
// latency chain; a tree is log2(n) deep.
__device__ __forceinline__ float tree_sum8(const float (&v)[8]) {
  return ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
}
// max(a, b, c) as one instruction.  (The compiler quiets each operand of an
// fmaxf first, one more instruction per operand of unknown origin; the
// operands here are matrix-instruction results, never signalling NaNs.)
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float tree_max32(const f32x16 (&s)[2]) {
  float m[11], n[4];
#pragma unroll
  for (int i = 0; i < 11; ++i) {
    const int a = 3 * i, b = 3 * i + 1, c = i < 10 ? 3 * i + 2 : 31;
    m[i] = max3f(s[a >> 4][a & 15], s[b >> 4][b & 15], s[c >> 4][c & 15]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) n[i] = max3f(m[3 * i], m[3 * i + 1], m[i < 3 ? 3 * i + 2 : 10]);
  return max3f(max3f(n[0], n[1], n[2]), n[3], n[3]);
}

// Storage of the layer's tensors (activations, cache, norms, bias): bf16
// (TRI_BF16) or fp32 (TRI_F32, the tight-parity mode).  Every load widens to
// fp32 and every store rounds from fp32 (RNE for bf16).
template <bool F32>
struct Store;
template <>
struct Store<false> {
  using T = bf16;
  __device__ __forceinline__ static float ld(const void* p, int64_t i) {
    return bf2f(((const bf16*)p)[i]);
  }
  __device__ __forceinline__ static void st(void* p, int64_t i, float v) {
    ((bf16*)p)[i] = f2bf(v);
  }
  __device__ __forceinline__ static f32x4 ld4(const void* p, int64_t i) {
    const bf16x4 v = *(const bf16x4*)((const bf16*)p + i);
    return f32x4{bf2f(v[0]), bf2f(v[1]), bf2f(v[2]), bf2f(v[3])};
  }
  __device__ __forceinline__ static void st4(void* p, int64_t i, f32x4 v) {
    bf16x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = f2bf(v[e]);
    *(bf16x4*)((bf16*)p + i) = o;
  }
};
template <>
struct Store<true> {
  using T = float;
  __device__ __forceinline__ static float ld(const void* p, int64_t i) {
    return ((const float*)p)[i];
  }
  __device__ __forceinline__ static void st(void* p, int64_t i, float v) { ((float*)p)[i] = v; }
  __device__ __forceinline__ static f32x4 ld4(const void* p, int64_t i) {
    return *(const f32x4*)((const float*)p + i);
  }
  __device__ __forceinline__ static void st4(void* p, int64_t i, f32x4 v) {
    *(f32x4*)((float*)p + i) = v;
  }
};

// Online softmax: the running max is only raised when a tile's max exceeds
// it by more than this many log2 units; weights then stay below 2^8, and
// the stale max cancels exactly in the final normalisation.
constexpr float kSoftmaxSlack = 8.0f;

}  // namespace tri
