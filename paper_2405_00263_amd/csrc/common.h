// Shared device helpers for the Clover gfx950 kernels: storage types, bf16
// conversion, matrix-core wrappers and the tiled layouts of packed weights and of
// the paged KV cache.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

typedef uint16_t bf16_t;  // bf16 bit pattern in storage

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float((uint32_t)h << 16); }
// round to nearest even (finite inputs)
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// Storage type traits.  A "lane vector" is 16 bytes: EPL elements.  A matrix-core
// fragment is 64 lanes x 16 bytes and covers 16 rows x KC columns (KC = 4 * EPL).
template <typename S> struct St;
template <> struct St<float> {
  static constexpr int EPL = 4;
  __device__ static __forceinline__ float ld(const float* p) { return *p; }
  __device__ static __forceinline__ float to_f(float v) { return v; }
  __device__ static __forceinline__ float from_f(float v) { return v; }
};
template <> struct St<bf16_t> {
  static constexpr int EPL = 8;
  __device__ static __forceinline__ float to_f(bf16_t v) { return bf2f(v); }
  __device__ static __forceinline__ bf16_t from_f(float v) { return f2bf(v); }
};

// acc[16x16] += A[16 x KC] * B[KC x 16], A/B given as one lane vector each in the
// matrix-core layout: lane l holds row (l % 16) and the EPL consecutive k values of
// lane group (l / 16).  The k order inside a fragment only has to agree between A
// and B, which the packed layouts guarantee.
__device__ __forceinline__ f32x4_t mma_frag(u32x4_t a, u32x4_t b, f32x4_t c, bf16_t) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mma_frag(u32x4_t a, u32x4_t b, f32x4_t c, float) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[0]), __uint_as_float(b[0]), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[1]), __uint_as_float(b[1]), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[2]), __uint_as_float(b[2]), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[3]), __uint_as_float(b[3]), c, 0, 0, 0);
  return c;
}

// ---- argmax keys ---------------------------------------------------------------------
// Every element maps to a 64-bit key whose order is (value ascending, index descending):
// the maximum key is the largest value with the lowest index (ties resolve to the lowest
// index), so partial maxima combine exactly and in any order.
__device__ __forceinline__ unsigned long long amax_key(float v, int i) {
  uint32_t u = __float_as_uint(v + 0.0f);  // -0 -> +0: equal values tie on the index
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((unsigned long long)u << 32) | (uint32_t)(0x7fffffff - i);
}
__device__ __forceinline__ unsigned long long umax64(unsigned long long a, unsigned long long b) {
  return a > b ? a : b;
}
// Reductions over the 16 lanes of a matrix-core row group by DPP row rotations (VALU
// only); every lane of the group ends with the result.
template <int ROR>
__device__ __forceinline__ int dpp_row_ror(int x) {
  return __builtin_amdgcn_update_dpp(0, x, 0x120 + ROR, 0xf, 0xf, false);
}
__device__ __forceinline__ float row16_max(float x) {
  x = fmaxf(x, __int_as_float(dpp_row_ror<8>(__float_as_int(x))));
  x = fmaxf(x, __int_as_float(dpp_row_ror<4>(__float_as_int(x))));
  x = fmaxf(x, __int_as_float(dpp_row_ror<2>(__float_as_int(x))));
  return fmaxf(x, __int_as_float(dpp_row_ror<1>(__float_as_int(x))));
}
__device__ __forceinline__ int row16_min(int x) {
  x = min(x, dpp_row_ror<8>(x));
  x = min(x, dpp_row_ror<4>(x));
  x = min(x, dpp_row_ror<2>(x));
  return min(x, dpp_row_ror<1>(x));
}
// argmax key of a row group's best element: v and column n of this lane (n = INT_MAX and
// v = -inf for lanes without a column); ties take the lowest column
__device__ __forceinline__ unsigned long long row16_amax_key(float v, int n) {
  const float mx = row16_max(v);
  return amax_key(mx, row16_min(v == mx ? n : 0x7fffffff));
}
__device__ __forceinline__ unsigned long long shfl_xor_u64(unsigned long long v, int o) {
  const unsigned lo = __shfl_xor((unsigned)(v & 0xffffffffu), o), hi = __shfl_xor((unsigned)(v >> 32), o);
  return ((unsigned long long)hi << 32) | lo;
}
// max over the 16 lanes of a matrix-core row group (lanes sharing l / 16)
__device__ __forceinline__ unsigned long long max16_u64(unsigned long long k) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) k = umax64(k, shfl_xor_u64(k, o));
  return k;
}

// ---- packed weight layout ----------------------------------------------------------
// W[N][K] row-major is stored as fragments (tile t = n/16, chunk c = k/KC) of 64 lanes
// x EPL elements; lane = n%16 + 16 * ((k%KC)/EPL), element = k%EPL.
__host__ __device__ __forceinline__ size_t packed_index(int n, int k, int nchunks, int EPL) {
  const int KC = 4 * EPL;
  const int t = n >> 4, c = k / KC, q = k % KC;
  const int lane = (n & 15) + 16 * (q / EPL);
  return (((size_t)t * nchunks + c) * 64 + lane) * EPL + (q % EPL);
}

// ---- paged KV cache layout --------------------------------------------------------
// Pool per layer: [n_blocks][n_kv][16 keys * hd].  Inside a block:
//  K: fragment order for the score product (keys are matrix rows): chunk c = d/KC,
//     lane = key + 16*((d%KC)/EPL), element d%EPL.
//  V: per 16-column tile nt = d/16: [g = key/4][i = d%16][e = key%4], so one lane
//     reads the 4 keys of its group for one column.
__device__ __forceinline__ int kblk_off(int key, int d, int EPL) {
  const int KC = 4 * EPL;
  const int c = d / KC, q = d % KC;
  return (c * 64 + key + 16 * (q / EPL)) * EPL + (q % EPL);
}
__device__ __forceinline__ int vblk_off(int key, int d) {
  const int nt = d >> 4, i = d & 15, g = key >> 2, e = key & 3;
  return ((nt * 4 + g) * 16 + i) * 4 + e;
}
__device__ __forceinline__ size_t kv_block_base(const int* block_table, int max_blocks, int seq,
                                                int slot, int kvh, int n_kv, int hd) {
  const int blk = block_table[(size_t)seq * max_blocks + (slot >> 4)];
  return ((size_t)blk * n_kv + kvh) * (size_t)(16 * hd);
}

// Sum over the 64 lanes of a wave in a fixed order with lane moves that stay in the VALU (no
// LDS round trip per step): DPP inside each 16-lane row (quad swaps 1 and 2, half-row and row mirrors), then the
// 16- and 32-lane swaps.  Every lane ends with the same value.
#define CLOVER_DPP_ADD(v, ctrl) \
  (v) += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), (ctrl), 0xF, 0xF, true))
__device__ __forceinline__ float wave_sum(float v) {
  CLOVER_DPP_ADD(v, 0xB1);   // quad_perm [1,0,3,2]
  CLOVER_DPP_ADD(v, 0x4E);   // quad_perm [2,3,0,1]
  CLOVER_DPP_ADD(v, 0x141);  // row_half_mirror
  CLOVER_DPP_ADD(v, 0x140);  // row_mirror
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(b[0]) + __uint_as_float(b[1]);
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}
#define CLOVER_DPP_MAX(v, ctrl) \
  (v) = fmaxf((v), __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), (ctrl), 0xF, 0xF, true)))
__device__ __forceinline__ float wave_max(float v) {
  CLOVER_DPP_MAX(v, 0xB1);
  CLOVER_DPP_MAX(v, 0x4E);
  CLOVER_DPP_MAX(v, 0x141);
  CLOVER_DPP_MAX(v, 0x140);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
}
#undef CLOVER_DPP_MAX
#undef CLOVER_DPP_ADD
__device__ __forceinline__ float silu_f(float x) { return x / (1.0f + __expf(-x)); }

// ---- counter-based random numbers and Gumbel-max sampling ----------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
// SC 2011): ten rounds of two 32x32->64 multiplies with the round keys bumped by the Weyl
// constants; returns the first output word for counter (c0, c1, c2, c3) and key (k0, k1).
__device__ __forceinline__ uint32_t philox4x32_10_w0(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                     uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t hi0 = __umulhi(0xD2511F53u, c0), lo0 = 0xD2511F53u * c0;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c2), lo1 = 0xCD9E8D57u * c2;
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c0;
}

// Standard Gumbel noise -log(-log(u)) from a 32-bit word: u = (m + 1/2) * 2^-23 with m the
// top 23 bits.  m + 1/2 fits the 24-bit float significand, so u is exact and lies in
// [2^-24, 1 - 2^-24]: both logarithms stay finite.
__device__ __forceinline__ float gumbel_from_bits(uint32_t x) {
  const float u = ((float)(x >> 9) + 0.5f) * 1.1920928955078125e-07f;  // 2^-23
  return -logf(-logf(u));
}
