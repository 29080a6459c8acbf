// Matrix-core GEMM for hundreds of rows (the verify of batches of trees), bf16 storage.
//
//   Y[M][N] = X[M][K] * W[N][K]^T: fp32 split-K partials, or, unsplit, the Q|K|V epilogue
//   (rotary, Q rows, paged KV append) or the SwiGLU epilogue (silu(gate) * up of each feature).
//
// With hundreds of rows the verify GEMMs are compute-bound (Sec. 1 of the paper: batches times
// trees move decoding from memory- to compute-bound), so the design is set by the matrix cores:
//  * v_mfma_f32_32x32x16_bf16: on gfx950 it sustains about 2 PFLOP/s where the 16x16x32 form
//    sustains about 0.85 (measured with independent accumulator chains on every CU);
//  * a workgroup is 4 waves (2 x 2) over a 128 x (64 NB) output tile, each wave MB x NB 32x32
//    blocks (2 x NB), accumulators in registers;
//  * per 32-wide k chunk an LDS stage holds one 1 KB operand per 16 rows of X (the chunk's 64
//    bytes of each row, its four 16-byte pieces swizzled by row) and, for each 16-k half, one
//    per 32-column block of W in the matrix-core lane order (lane l: column l % 32, k (l / 32)
//    * 8 .. + 8); gfx950's direct-to-LDS loads gather them straight from global memory, 16
//    bytes per lane (X as whole row segments; W from two of its packed 16 x 32 fragments: the
//    packed weight layout stays the one the other kernels use), so operands never pass
//    through registers on their way into LDS, and every LDS read of a product operand is one
//    conflict-free 16-byte load per lane;
//  * NST stages in flight, one barrier per chunk (without the workgroup fence, which would
//    wait for every load in flight: each wave waits for its own loads of the chunk by count);
//    the next chunk's operands are read into a second register set while the current chunk is
//    multiplied, and the scheduler spreads those reads and the loads among the matrix-core
//    instructions;
//  * the Q|K|V epilogue passes each 32x32 block through LDS, where 8 consecutive columns of a
//    row meet their rotary partners (the other half of the 16-column tile) and leave with
//    16-byte stores;
//  * for SwiGLU a workgroup's columns are the gate rows of BN / 2 features (waves wn = 0)
//    followed by the up rows of the same features (wn = 1); the up waves hand their
//    accumulators to the gate waves through LDS at the end.
// gemm_wide.hip instantiates the shapes whose accumulators fit the ordinary VGPRs (built with
// the VGPR form of the matrix-core instructions), gemm_wide_acc.hip the 256-row SwiGLU shape,
// whose 192 accumulators per lane live in the accumulation registers.
#pragma once
#include "common.h"
#include "gemm_epi.h"
#include "kernels.h"

#include <hip/hip_ext.h>

#include <algorithm>

namespace clover {

typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void gbl_void_t;

static constexpr int WIDE_THREADS = 256;

// s_waitcnt on the vector-memory counter only (expcnt and lgkmcnt left at their maxima)
#define WIDE_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (((n) >> 4) << 14) | (0x7 << 4) | (0xF << 8))
// workgroup barrier without a memory fence: the waits by count above order the loads
#define WIDE_BARRIER() asm volatile("s_barrier" ::: "memory")

template <int MB, int NB, int NST, int MODE>
__global__ __launch_bounds__(WIDE_THREADS) __attribute__((amdgpu_waves_per_eu(1, 1))) void wide_kernel(const GemmParams p) {
  using S = bf16_t;
  constexpr int BM = 2 * MB * 32, BN = 2 * NB * 32;
  constexpr int FA = 2 * BM / 32, FB = 2 * BN / 32, F = FA + FB;  // 1 KB operands per stage
  constexpr int LPW = F / 4;                                      // loads per wave per chunk
  static_assert(F % 4 == 0 && NST >= 3, "operands split over the four waves; at least three stages");
  static_assert(MODE != EP_SWIGLU || 2 * MB * NB * 16 * 64 * 4 <= NST * F * 1024, "SwiGLU hand-over fits the stages");
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  __shared__ int s_kvbase[BM];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave >> 1, wn = wave & 1;
  // XCD-aware order: the row tiles of one (column group, split) take consecutive ids on one
  // XCD and find each other's weight blocks in its L2
  const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3;
  const int mc = q % p.mchunks, r = (q / p.mchunks) * 8 + xcd;
  if (r >= p.ngroups * p.S) return;  // padding of the last round
  const int g = r % p.ngroups, split = r / p.ngroups;
  const int c0 = split * p.cps, nk = min(p.nchunks, c0 + p.cps) - c0;
  const int m0 = mc * BM, n0 = g * BN;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  int kvb = 0;  // KV-append target of row m0 + threadIdx.x (Q|K|V epilogue), staged in LDS at the end
  if (MODE == EP_QKV && threadIdx.x < BM) kvb = p.row_kb[min(m0 + (int)threadIdx.x, p.M - 1)];

  // Sources of this wave's LPW operands of chunk c0: a wave-uniform base (advanced per chunk)
  // plus a per-lane byte offset.  Operand f < FA: X rows 16 f .. 16 f + 15, the whole chunk;
  // else W columns of block (f - FA) / 2, k half (f - FA) % 2.  Rows past M and columns past N
  // read valid rows and tiles whose results are never stored.
  const char* ubase[LPW];
  uint32_t loff[LPW];
  int ustep[LPW];
  const int tl0 = p.seg[0].tiles, tl1 = p.seg[1].tiles;
#pragma unroll
  for (int i = 0; i < LPW; ++i) {
    const int f = wv * LPW + i;
    if (f < FA) {
      // X operand f: rows 16 f .. 16 f + 15 of the workgroup, the chunk's 64 bytes of each row
      // as four 16-byte pieces, lane 4 r + q taking piece q ^ (r / 4 % 4) of row r (whole row
      // segments per load; the swizzle keeps the matrix-core reads below conflict-free)
      const int r16 = lane >> 2, piece = (lane & 3) ^ ((r16 >> 2) & 3);
      const int row = min(m0 + 16 * f + r16, p.M - 1);
      ubase[i] = reinterpret_cast<const char*>(p.X) + (size_t)c0 * 64;
      loff[i] = (uint32_t)row * (uint32_t)p.ldx * 2u + (uint32_t)piece * 16u;
      ustep[i] = 64;
    } else {
      const int cb = (f - FA) >> 1, h = (f - FA) & 1;
      int t;
      const void* w = p.seg[0].w;
      if constexpr (MODE == EP_SWIGLU) {
        // blocks 0 .. NB-1: gate tile pairs of features g BN/2 ..; NB .. 2NB-1: the same
        // features' up tile pairs (segment 1, as long as segment 0); past the last feature
        // the last pair
        t = min(g * (BN / 32) + 2 * (cb < NB ? cb : cb - NB), tl0 - 2);
        if (cb >= NB) w = p.seg[1].w;
      } else {
        t = (n0 >> 4) + 2 * cb;                 // the block's first (even) 16-column tile
        t = min(t, p.ntiles - 2);               // blocks past N: the last two tiles
        if (p.nseg > 1 && t >= tl0) {           // segment of the tile pair (segments hold
          t -= tl0;                             // whole pairs of tiles)
          w = p.seg[1].w;
          if (p.nseg > 2 && t >= tl1) {
            t -= tl1;
            w = p.seg[2].w;
          }
        }
      }
      const int tt = t + ((lane & 31) >> 4);
      ubase[i] = reinterpret_cast<const char*>(w) + (size_t)c0 * 1024;
      loff[i] = (uint32_t)tt * (uint32_t)p.nchunks * 1024u + (uint32_t)((lane & 15) + 16 * (2 * h + (lane >> 5))) * 16u;
      ustep[i] = 1024;
    }
  }
  auto issue = [&](int c, int stg) {  // operands of chunk c (clamped to the split) into stage stg
    const int cc = min(c, nk - 1);
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      const char* u = ubase[i] + (size_t)cc * ustep[i];
      __builtin_amdgcn_global_load_lds((gbl_void_t*)(u + loff[i]),
                                       (lds_void_t*)(smem + (size_t)stg * F * 1024 + (wv * LPW + i) * 1024), 16, 0, 0);
    }
  };
  f32x16_t acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  u32x4_t a[2][2][MB], b[2][2][NB];  // [register set][k half][block]
  // X operand of product row block i, k half h for lane l: row l % 32 of the block, piece
  // 2 h + l / 32 of that row (k (l / 32) 8 .. + 8 of the half), at its swizzled slot
  uint32_t aoff[2];
#pragma unroll
  for (int h = 0; h < 2; ++h)
    aoff[h] = ((lane >> 4) & 1) * 1024 + ((lane & 15) * 4 + ((2 * h + (lane >> 5)) ^ ((lane >> 2) & 3))) * 16;
  auto read = [&](int stg, int set) {
    const char* st = smem + (size_t)stg * F * 1024;
    const char* s = st + lane * 16;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int i = 0; i < MB; ++i) a[set][h][i] = *reinterpret_cast<const u32x4_t*>(st + 2 * (wm * MB + i) * 1024 + aoff[h]);
#pragma unroll
      for (int j = 0; j < NB; ++j) b[set][h][j] = *reinterpret_cast<const u32x4_t*>(s + (FA + 2 * (wn * NB + j) + h) * 1024);
    }
  };
  auto mma = [&](int set) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a[set][h][i]),
                                                            __builtin_bit_cast(bf16x8_t, b[set][h][j]), acc[i][j], 0, 0, 0);
  };

  // Prologue: chunks 0 .. NST-2 in flight, chunk 0 in registers.
#pragma unroll
  for (int s = 0; s < NST - 1; ++s) issue(s, s);
  WIDE_WAIT_VM((NST - 2) * LPW);
  WIDE_BARRIER();
  read(0, 0);
  // Iteration c: wait for chunk c + 1 (every iteration issues one load group, past the end the
  // last chunk again into a stage nobody reads, so the count of groups after it is fixed),
  // refill the stage of chunk c - 1 (read an iteration ago) with chunk c + NST - 1, read chunk
  // c + 1 into the other register set, multiply chunk c.
  auto iter = [&](int c, int set) {
    WIDE_WAIT_VM((NST - 3) * LPW);
    WIDE_BARRIER();
    issue(c + NST - 1, (c + NST - 1) % NST);
    read((c + 1) % NST, set ^ 1);
    mma(set);
#pragma unroll
    for (int k = 0; k < LPW; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // a matrix-core instruction
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // a load into LDS
    }
#pragma unroll
    for (int k = 0; k < 2 * (MB + NB); ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // a matrix-core instruction
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // an LDS read
    }
  };
  int c = 0;
  for (; c + 1 < nk; c += 2) {
    iter(c, 0);
    iter(c + 1, 1);
  }
  if (c < nk) iter(c, 0);
  // loads past the last chunk are still landing in LDS: they finish before the workgroup does
  WIDE_WAIT_VM(0);

  // Epilogues.  Accumulator element e of block (i, j) is row m0 + (wm MB + i) 32 + 8 (e / 4) +
  // 4 (lane / 32) + e % 4, column n0 + (wn NB + j) 32 + lane % 32.
  if constexpr (MODE == EP_PARTIAL) {
    float* out = p.part + (size_t)split * p.M * p.N;
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int n = n0 + (wn * NB + j) * 32 + (lane & 31);
        if (n >= p.N) continue;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = m0 + (wm * MB + i) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          if (m < p.M) out[(size_t)m * p.N + n] = acc[i][j][e];
        }
      }
  } else if constexpr (MODE == EP_SWIGLU) {
    // the up waves (wn = 1) write their accumulators to the idle stage buffers, element (i, j,
    // e) of lane l at [(i NB + j) 16 + e][l]; the gate wave of the same rows (wn = 0, same i, j,
    // e and lane: the same row and feature) finishes silu(gate) * up
    __syncthreads();  // every wave is past its last stage read
    float* xch = reinterpret_cast<float*>(smem) + (size_t)wm * MB * NB * 16 * 64;
    if (wn == 1) {
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) xch[((i * NB + j) * 16 + e) * 64 + lane] = acc[i][j][e];
    }
    __syncthreads();
    if (wn == 0) {
      S* out = reinterpret_cast<S*>(p.out_s);
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int fe = g * (BN / 2) + j * 32 + (lane & 31);
        if (fe >= p.N) continue;
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int m = m0 + (wm * MB + i) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            const float up = xch[((i * NB + j) * 16 + e) * 64 + lane];
            if (m < p.M) out[(size_t)m * p.ldos + fe] = St<S>::from_f(silu_f(acc[i][j][e]) * up);
          }
      }
    }
  } else {
    // EP_QKV, one 32x32 block at a time through this wave's slice of the (now idle) stage
    // buffers: a lane then takes 8 consecutive columns of a row with the 8 of their rotary
    // partners (the other half of the 16-column tile) and stores 16 bytes at a time
    if (threadIdx.x < BM) s_kvbase[threadIdx.x] = kvb;
    __syncthreads();  // every wave is past its last stage read; s_kvbase complete
    constexpr int TS = 36;  // floats per LDS row (16-byte aligned rows)
    float* tile = reinterpret_cast<float*>(smem) + wave * 32 * TS;
    const int ncols = (p.n_heads + 2 * p.n_kv) * p.hd;
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) {
#pragma unroll
        for (int e = 0; e < 16; ++e) tile[(8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)) * TS + (lane & 31)] = acc[i][j][e];
        const int rb = (wm * MB + i) * 32, cb = n0 + (wn * NB + j) * 32;
#pragma unroll
        for (int it = 0; it < 2; ++it) {  // 32 rows x 4 eight-column groups = 128 items
          const int item = lane + 64 * it, rr = item >> 2, gq = item & 3;
          const int m = m0 + rb + rr, pc0 = cb + gq * 8;
          if (m >= p.M || pc0 >= ncols) continue;
          const float4* src = reinterpret_cast<const float4*>(tile + rr * TS + gq * 8);
          const float4* prt = reinterpret_cast<const float4*>(tile + rr * TS + (gq ^ 1) * 8);
          const float4 v0 = src[0], v1 = src[1], w0 = prt[0], w1 = prt[1];
          float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
          const float w[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
          const QkvCols8 cols = qkv_cols8(p, pc0);
          float4 cs4[4];
          qkv_cs8(p, m, cols, cs4);
          qkv_store8<S>(p, m, cols, v, w, cs4, s_kvbase[rb + rr]);
        }
      }
  }
}

// ---- host side ------------------------------------------------------------------------

struct WideShape {
  int mb, nb, nst;
};
constexpr int WIDE_N_CU = 256;
constexpr WideShape kWideQkv = {2, 3, 4};      // 128 x 192: the 7B Q|K|V at 512 rows is 256 workgroups
constexpr WideShape kWidePartial = {2, 4, 4};  // 128 x 256, K split until the grid covers the CUs
constexpr WideShape kWideSwiglu = {4, 3, 4};   // 256 x (96 gate + 96 up): the 7B gate|up at 512 rows is 230 workgroups

inline size_t wide_lds(const WideShape& sh) { return (size_t)sh.nst * (size_t)(2 * (2 * sh.mb + 2 * sh.nb)) * 1024; }

inline GemmPlan make_wide(const WideShape& sh, int M, int ntiles, int nchunks, int S) {
  GemmPlan pl{};
  pl.tiled = 2;
  pl.nw = 4;
  pl.mt = sh.mb;
  pl.tw = sh.nb;
  pl.ring = sh.nst;
  const int bm = 64 * sh.mb, btiles = 4 * sh.nb;  // rows and 16-column tiles per workgroup
  pl.mchunks = (M + bm - 1) / bm;
  pl.ngroups = (ntiles + btiles - 1) / btiles;
  pl.cps = (nchunks + S - 1) / S;
  pl.S = (nchunks + pl.cps - 1) / pl.cps;
  pl.lds_bytes = wide_lds(sh);
  pl.part_floats = (size_t)pl.S * M * ntiles * 16;
  return pl;
}

template <int MB, int NB, int NST, int MODE>
hipError_t launch_wide_shape(const GemmPlan& pl, GemmParams& p, hipStream_t st, const LaunchTiming* lt) {
  auto kern = wide_kernel<MB, NB, NST, MODE>;
  static bool lds_attr = false;  // dynamic LDS above 64 KB is opted into once per kernel
  if (!lds_attr) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)pl.lds_bytes);
    if (e != hipSuccess) return e;
    lds_attr = true;
  }
  dim3 grid(8 * ((pl.ngroups * pl.S + 7) / 8) * pl.mchunks), block(WIDE_THREADS);
  if (lt) hipExtLaunchKernelGGL(kern, grid, block, (uint32_t)pl.lds_bytes, st, lt->start, lt->stop, 0, p);
  else hipLaunchKernelGGL(kern, grid, block, pl.lds_bytes, st, p);
  return hipGetLastError();
}

// The 256-row SwiGLU shape (gemm_wide_acc.hip).
hipError_t launch_wide_acc(GemmParams& p, const GemmPlan& pl, hipStream_t st, const LaunchTiming* lt);

}  // namespace clover
