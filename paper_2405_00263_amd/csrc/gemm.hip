// Weight-streaming GEMM for small M on gfx950 matrix cores.
//
//   Y[M][N] = X[M][K] * W[N][K]^T, fused epilogues (rotary + KV append, SwiGLU) or
//   fp32 split-K partials.
//
// Decoding streams every weight once per forward while only M (= tree tokens) rows
// use it, so the kernel is bound by HBM bandwidth (Sec. 1 of the paper: decoding is
// memory-bound).  Design:
//  * weights are pre-tiled (packed_index) so one wave's 16-byte-per-lane load of a
//    16 x KC fragment is 1 KB of contiguous memory, streamed with non-temporal loads
//    and a register prefetch ring;
//  * a workgroup is NW waves (2..8), one 16-row weight tile each, all sharing the X
//    tile, which is staged through LDS in double-buffered stages; X is prefetched into
//    registers as many stages ahead as the weight ring, so waiting for an X load never
//    forces younger weight loads to land (loads complete in order);
//  * on gfx950 a compute unit moves roughly 40-50 GB/s of weight plus X bytes in this
//    loop, so the planner picks NW and the K split per shape to keep every CU busy with
//    one workgroup while keeping the X bytes per weight byte low (plan_gemm);
//  * Q/K weights are packed so that each 16-row tile holds 8 rows of the first rotary
//    half and their 8 partners of the second half: the rotary epilogue is tile-local and
//    any NW works;
//  * K may be split over workgroups (EP_PARTIAL): each split writes its own fp32
//    partial [split][M][N] and the consumer kernel sums them in split order, so the
//    result does not depend on scheduling and no cross-workgroup synchronisation (and
//    no device-scope fence, which on gfx950 writes back and invalidates the L2) is
//    needed inside the GEMM;
//  * fused epilogues (rotary + KV append, SwiGLU) run unsplit on an LDS tile.
#include "common.h"
#include "gemm_epi.h"
#include "kernels.h"

#include <hip/hip_ext.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

namespace clover {

static constexpr int STAGE_CHUNKS = 4;   // chunks of X per LDS stage
// Weight fragments in flight per wave (8 KB).  A sweep of 8, 16, 24 and 32 (and of 2- and
// 4-chunk stages) on MI355X put 8 first on every 64-row shape: the shallower ring leaves
// 112-130 VGPRs, so two 8-wave (or 6-wave) workgroups share a compute unit, and two
// workgroups' loads in flight beat one workgroup's deeper ring.
static constexpr int PF = 8;
static constexpr int RING = PF / STAGE_CHUNKS;  // stages covered by the prefetch ring
static_assert(RING % 2 == 0, "stages alternate between two LDS buffers inside a superstage");

template <int NW>
__device__ __forceinline__ const u32x4_t* wave_weight_ptr(const GemmParams& p, int g, int wave,
                                                          bool& active) {
  // The segment fields are read at constant indices (scalar loads of the argument block) and
  // selected per wave: indexing them by the wave's segment would make them vector loads from
  // the argument block, two dependent memory round trips before the first weight load.
  const int tl0 = p.seg[0].tiles, tl1 = p.seg[1].tiles;
  const void* w0 = p.seg[0].w;
  const void* w1 = p.seg[1].w;
  const void* w2 = p.seg[2].w;
  const void* w = w0;
  int t;
  if (p.mode == EP_SWIGLU) {  // waves [0, NW/2) gate tiles, [NW/2, NW) the matching up tiles
    constexpr int H = NW / 2;
    const bool up = wave >= H;
    t = g * H + wave - (up ? H : 0);
    active = t < (up ? tl1 : tl0);
    w = up ? w1 : w0;
  } else {  // tile t of the concatenated segments; the last segment takes the rest
    t = g * NW + wave;
    active = t < p.ntiles;
    if (p.nseg > 1 && t >= tl0) {
      t -= tl0;
      w = w1;
      if (p.nseg > 2 && t >= tl1) {
        t -= tl1;
        w = w2;
      }
    }
  }
  if (!active) return nullptr;
  return reinterpret_cast<const u32x4_t*>(w) + (size_t)t * p.nchunks * 64;
}

template <typename S, int NW>
__device__ void gemm_epilogue(const GemmParams& p, const float* tile, int g, int m0, int mrows,
                              const int* s_kvbase) {
  using T = St<S>;
  constexpr int THREADS = NW * 64, COLS = NW * 16, TSTRIDE = COLS + 4;
  const int tid = threadIdx.x;
  if (p.mode == EP_SWIGLU) {
    constexpr int HC = COLS / 2;  // SwiGLU outputs per group
    const int F = p.N;
    for (int e = tid; e < mrows * HC; e += THREADS) {
      const int r = e / HC, j = e % HC, m = m0 + r, n = g * HC + j;
      if (m >= p.M || n >= F) continue;
      const float gt = tile[r * TSTRIDE + j], up = tile[r * TSTRIDE + HC + j];
      reinterpret_cast<S*>(p.out_s)[(size_t)m * p.ldos + n] = T::from_f(silu_f(gt) * up);
    }
    return;
  }
  // EP_QKV.  Each thread owns one column of the tile (THREADS / COLS == 4 rows at a time).
  const int col = tid % COLS;
  const int pc = g * COLS + col;  // physical column over the packed [q; k; v] tiles
  if (pc >= (p.n_heads + 2 * p.n_kv) * p.hd) return;
  for (int r = tid / COLS; r < mrows; r += THREADS / COLS) {
    const int m = m0 + r;
    if (m >= p.M) break;
    qkv_store<S>(p, m, pc, tile[r * TSTRIDE + col], tile[r * TSTRIDE + (col ^ 8)], s_kvbase[r]);
  }
}

// AMAX: the EP_PARTIAL epilogue also leaves per-(group, row) argmax keys in p.amax_part
// (a separate instantiation, so the other GEMMs keep their code unchanged)
template <typename S, int MT, int NW, bool AMAX>
__global__ __launch_bounds__(NW * 64) void gemm_kernel(const GemmParams p) {
  using T = St<S>;
  constexpr int THREADS = NW * 64, COLS = NW * 16, TSTRIDE = COLS + 4;
  constexpr int EPL = T::EPL, KC = 4 * EPL, MROWS = 16 * MT;
  constexpr int XSTRIDE = STAGE_CHUNKS * KC + EPL;          // elements per LDS row
  constexpr int XBUF = MROWS * XSTRIDE;                      // elements per stage buffer
  constexpr int VEC_PER_ROW = STAGE_CHUNKS * 4;              // 16-byte vectors per row per stage
  constexpr int XVEC = (MROWS * VEC_PER_ROW + THREADS - 1) / THREADS;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  S* xs = reinterpret_cast<S*>(smem);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  // Workgroup ids are dealt to the 8 XCDs round-robin.  The row chunks of one (group, split)
  // take consecutive ids on one XCD, so they stream the same weight tiles at about the same
  // time and all but the first find them in that XCD's L2 (one chunk: the identity map).
  const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3;
  const int mc = q % p.mchunks, r = (q / p.mchunks) * 8 + xcd;
  if (r >= p.ngroups * p.S) return;  // padding of the last round
  const int g = r % p.ngroups, split = r / p.ngroups;
  const int m0 = mc * MROWS;
  const int c0 = split * p.cps;
  const int c1 = min(p.nchunks, c0 + p.cps);
  const int nk = c1 - c0;
  const int nst = (nk + STAGE_CHUNKS - 1) / STAGE_CHUNKS;

  // KV-append targets of the fused epilogue: loaded up front into a register (nothing waits
  // for it before the epilogue) and staged in LDS for the epilogue's row loop
  __shared__ int s_kvbase[MROWS];
  int kvb = 0;
  if (p.mode == EP_QKV && threadIdx.x < MROWS) kvb = p.row_kb[min(m0 + (int)threadIdx.x, p.M - 1)];

  bool active;
  const u32x4_t* wp = wave_weight_ptr<NW>(p, g, wave, active);
  // Inactive waves (past the last tile) stream a valid tile and discard the result, so no
  // load sits behind a branch.
  if (!active) wp = reinterpret_cast<const u32x4_t*>(p.seg[0].w);
  wp += (size_t)c0 * 64 + lane;

  u32x4_t wb[PF];

  // X stage loader: rows m0.., chunks [c0 + st*STAGE_CHUNKS, ...).  Addresses are clamped
  // into range so every load is unconditional (a load whose result may be discarded by a
  // select would need to complete before the select); rows past M are zeroed at store
  // time, and chunks past the split are never read.
  const S* X = reinterpret_cast<const S*>(p.X);
  auto load_x = [&](int st, u32x4_t* regs) {
#pragma unroll
    for (int i = 0; i < XVEC; ++i) {
      const int v = min((int)threadIdx.x + i * THREADS, MROWS * VEC_PER_ROW - 1);
      const int r = min(v / VEC_PER_ROW, p.M - 1 - m0), cv = v % VEC_PER_ROW;
      const int cchunk = min(st * STAGE_CHUNKS + cv / 4, nk - 1);
      regs[i] = *reinterpret_cast<const u32x4_t*>(X + (size_t)(m0 + r) * p.ldx +
                                                  (size_t)(c0 + cchunk) * KC + (cv % 4) * EPL);
    }
  };
  auto store_x = [&](int buf, const u32x4_t* regs) {
#pragma unroll
    for (int i = 0; i < XVEC; ++i) {
      const int v = threadIdx.x + i * THREADS;
      if (v < MROWS * VEC_PER_ROW) {
        const int r = v / VEC_PER_ROW, cv = v % VEC_PER_ROW;
        const u32x4_t zero = {0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4_t*>(xs + buf * XBUF + r * XSTRIDE + cv * EPL) = (m0 + r < p.M) ? regs[i] : zero;
      }
    }
  };

  // X register ring, RING stages deep: stage st lives in xr[st % RING].  Loads are issued
  // stage by stage -- X(q) then the weights of stage q -- both in the prologue and in the
  // loop, so waiting for any load only waits for loads that are needed no later.
  u32x4_t xr[RING][XVEC];
#pragma unroll
  for (int q = 0; q < RING; ++q) {
    load_x(q, xr[q]);
#pragma unroll
    for (int u = q * STAGE_CHUNKS; u < (q + 1) * STAGE_CHUNKS; ++u)
      wb[u] = __builtin_nontemporal_load(wp + (size_t)min(u, nk - 1) * 64);
  }
  store_x(0, xr[0]);
  __syncthreads();

  f32x4_t acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // One stage: issue X(st + RING) into the slot stage st vacated, consume the stage's
  // weight fragments (each slot refilled right after use, so the load lands in a dead
  // register), stage X(st + 1) into the other LDS buffer.  Stages alternate between
  // the two buffers; walking them RING at a time keeps the ring slot (chunk % PF) and
  // the buffer a compile-time index.
  auto stage = [&](int st, int par, bool guard) {
    load_x(st + RING, xr[par]);
    const S* xb = xs + (par & 1) * XBUF + (lane & 15) * XSTRIDE + (lane >> 4) * EPL;
#pragma unroll
    for (int u = 0; u < STAGE_CHUNKS; ++u) {
      const int c = st * STAGE_CHUNKS + u;
      if (!guard || c < nk) {
        const u32x4_t w = wb[par * STAGE_CHUNKS + u];
        const S* xc = xb + u * KC;
#pragma unroll
        for (int t = 0; t < MT; ++t) {
          const u32x4_t a = *reinterpret_cast<const u32x4_t*>(xc + t * 16 * XSTRIDE);
          acc[t] = mma_frag(a, w, acc[t], S{});
        }
      }
      wb[par * STAGE_CHUNKS + u] = __builtin_nontemporal_load(wp + (size_t)min(c + PF, nk - 1) * 64);
    }
    store_x((par & 1) ^ 1, xr[(par + 1) % RING]);
    __syncthreads();
  };
  // steady state: whole superstages of PF chunks, branch-free so the wait counts stay exact
  const int nsuper = nk / PF;
  for (int ss = 0; ss < nsuper; ++ss) {
#pragma unroll
    for (int par = 0; par < RING; ++par) stage(ss * RING + par, par, false);
  }
  // ragged tail: fewer than PF chunks left
#pragma unroll
  for (int par = 0; par < RING; ++par) {
    const int st = nsuper * RING + par;
    if (st < nst) stage(st, par, true);
  }

  if (p.mode == EP_PARTIAL) {
    // split `split` writes rows m0.. of its own [M][N] fp32 slice
    if (!AMAX && !active) return;
    const int n = (g * NW + wave) * 16 + (lane & 15);  // segments are contiguous in N
    // with argmax keys the logits themselves are optional (p.part null: keys only)
    if (active && (!AMAX || p.part)) {
      float* out = p.part + (size_t)split * p.M * p.N;
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = m0 + t * 16 + 4 * (lane >> 4) + r;
          if (m < p.M) out[(size_t)m * p.N + n] = acc[t][r];
        }
    }
    if constexpr (AMAX) {
      // each row's best (value, column) over this group's columns: lanes, then waves
      unsigned long long* s_key = reinterpret_cast<unsigned long long*>(smem);  // [NW][MROWS]
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = min(m0 + t * 16 + 4 * (lane >> 4) + r, p.M - 1);  // rows past M: not stored
          const unsigned long long k =
              row16_amax_key(active ? amax_value(p, acc[t][r], m, n) : -INFINITY, active ? n : 0x7fffffff);
          if ((lane & 15) == 0) s_key[wave * MROWS + t * 16 + 4 * (lane >> 4) + r] = k;
        }
      __syncthreads();
      for (int i = threadIdx.x; i < MROWS; i += THREADS) {
        if (m0 + i >= p.M) break;
        unsigned long long best = 0ull;
        for (int w = 0; w < NW; ++w) best = umax64(best, s_key[w * MROWS + i]);
        p.amax_part[(size_t)g * p.M + m0 + i] = best;
      }
    }
    return;
  }
  if (threadIdx.x < MROWS) s_kvbase[threadIdx.x] = kvb;
  const int col = wave * 16 + (lane & 15);
  float* tile = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) tile[(t * 16 + 4 * (lane >> 4) + r) * TSTRIDE + col] = acc[t][r];
  __syncthreads();
  gemm_epilogue<S, NW>(p, tile, g, m0, MROWS, s_kvbase);
}

// ---- host side ------------------------------------------------------------------------

static int es_of(int dtype) { return dtype == 1 ? 2 : 4; }

// Cost model of one launch (microseconds), from per-workgroup timings on MI355X: a CU
// streams weight + X bytes at about CU_GBS while the whole chip reads HBM at about
// HBM_GBS; fp32 partials are written once and read once by the consumer.
static constexpr double CU_GBS = 45.0, HBM_GBS = 6500.0;
static constexpr int N_CU = 256, N_XCD = 8;

static double plan_cost(const GemmPlan& pl, int es, int M, int ntiles, int nchunks) {
  const int KC = 64 / es;
  const long wgs = (long)pl.ngroups * pl.S * pl.mchunks;
  const long per_xcd = (wgs + N_XCD - 1) / N_XCD;
  const long rounds = (per_xcd + N_CU / N_XCD - 1) / (N_CU / N_XCD);
  const double wg_bytes = (double)pl.nw * pl.cps * 1024.0 + 16.0 * pl.mt * pl.cps * KC * es;
  const double t_cu = rounds * wg_bytes / (CU_GBS * 1e3);
  const double part = pl.S > 1 ? 2.0 * pl.S * M * ntiles * 16.0 * 4.0 : 0.0;
  const double t_hbm = ((double)ntiles * nchunks * 1024.0 + part) / (HBM_GBS * 1e3);
  return std::max(t_cu, t_hbm) + 0.1 * std::min(t_cu, t_hbm);
}

// Shapes of the shipped workloads whose best (waves, splits) a forced-plan sweep over every
// combination measured on MI355X; the cost model above ranks these few percent off.
struct TunedPlan {
  int mt, ntiles, nchunks;
  bool swiglu;
  int nw, S;
};
static const TunedPlan kTuned[] = {
    // 7B-shape bf16 (d 4096, 32 heads of 128, SwiGLU 11008, vocab 125696)
    {4, 768, 128, false, 6, 2},   // Q|K|V, 64 rows (split: the fix-up pass applies rotary)
    {4, 256, 128, false, 6, 4},   // O, 64 rows
    {4, 256, 344, false, 8, 8},   // down, 64 rows
    {4, 1376, 128, true, 6, 1},   // gate|up, 64 rows
    {4, 7856, 128, false, 8, 1},  // LM head, 64 rows
    {2, 7856, 128, false, 8, 1},  // LM head, 32 rows
    {1, 7856, 128, false, 2, 1},  // LM head, 1-16 rows
};

// From this many rows on, bf16 GEMMs use the register-blocked kernel (gemm_tiled.hip).
static constexpr int TILED_MIN_M = 129;

// Rows per chunk (16 * mt) of the streaming kernel.  Up to 128 rows a bf16 GEMM takes all
// its rows in one chunk: each weight fragment is loaded into a CU once and feeds mt
// matrix-core products (two 64-row chunks would load every fragment twice per CU, and a
// CU's load rate, not HBM, would bound the kernel).
static int chunk_mt(int dtype, int M) {
  if (M <= 16) return 1;
  if (M <= 32) return 2;
  return (M <= 64 || dtype != 1) ? 4 : 8;
}

GemmPlan plan_gemm(int dtype, int M, int ntiles, int nchunks, bool swiglu, int max_splits, int mode,
                   const int* seg_tiles, int nseg, bool amax) {
  GemmPlan wide;
  if (dtype == 1 && !amax && plan_wide(M, ntiles, nchunks, swiglu ? EP_SWIGLU : mode, max_splits, seg_tiles, nseg, wide))
    return wide;
  if (dtype == 1 && M >= TILED_MIN_M) return plan_tiled(M, ntiles, nchunks, swiglu, max_splits);
  const int es = es_of(dtype), EPL = 16 / es, KC = 4 * EPL;
  GemmPlan best{};
  double best_cost = 1e30;
  for (int nw : {4, 2, 3, 6, 8}) {
    if (swiglu && (nw & 1)) continue;
    GemmPlan pl{};
    pl.nw = nw;
    pl.mt = chunk_mt(dtype, M);
    if (pl.mt == 8 && nw != 8) continue;  // the 128-row X ring fits registers with 8 waves only
    const int mrows = 16 * pl.mt;
    pl.mchunks = (std::max(M, 1) + mrows - 1) / mrows;
    pl.ngroups = swiglu ? ((ntiles / 2) + nw / 2 - 1) / (nw / 2) : (ntiles + nw - 1) / nw;
    const int smax = std::max(1, std::min(max_splits, nchunks / (2 * STAGE_CHUNKS)));
    for (int S0 = 1; S0 <= smax; ++S0) {
      const int cps = (nchunks + S0 - 1) / S0;
      pl.cps = cps;
      pl.S = (nchunks + cps - 1) / cps;
      if (pl.S != S0) continue;
      const double c = plan_cost(pl, es, M, ntiles, nchunks);
      if (c < best_cost) {
        best_cost = c;
        best = pl;
      }
    }
  }
  if (dtype == 1) {
    const int mt = chunk_mt(dtype, M);
    for (const TunedPlan& t : kTuned) {
      if (t.mt != mt || t.ntiles != ntiles || t.nchunks != nchunks || t.swiglu != swiglu) continue;
      if (t.S > std::max(1, std::min(max_splits, nchunks / (2 * STAGE_CHUNKS)))) continue;
      const int cps = (nchunks + t.S - 1) / t.S;
      if ((nchunks + cps - 1) / cps != t.S) continue;
      best.nw = t.nw;
      best.mt = mt;
      best.mchunks = (std::max(M, 1) + 16 * mt - 1) / (16 * mt);
      best.ngroups = swiglu ? ((ntiles / 2) + t.nw / 2 - 1) / (t.nw / 2) : (ntiles + t.nw - 1) / t.nw;
      best.S = t.S;
      best.cps = cps;
    }
  }
  const int mrows = 16 * best.mt;
  const size_t xbytes = 2ull * mrows * (STAGE_CHUNKS * KC + EPL) * es;
  const size_t tbytes = (size_t)mrows * (best.nw * 16 + 4) * 4;
  best.lds_bytes = std::max(xbytes, tbytes);
  best.part_floats = (size_t)best.S * M * ntiles * 16;
  return best;
}

template <typename S, int MT, bool AMAX>
static void launch_nw(const GemmPlan& pl, GemmParams& p, hipStream_t st, const LaunchTiming* lt) {
  dim3 grid(8 * ((pl.ngroups * pl.S + 7) / 8) * pl.mchunks), block(pl.nw * 64);
  auto go = [&](auto kern) {
    if (lt) hipExtLaunchKernelGGL(kern, grid, block, (uint32_t)pl.lds_bytes, st, lt->start, lt->stop, 0, p);
    else hipLaunchKernelGGL(kern, grid, block, pl.lds_bytes, st, p);
  };
  switch (pl.nw) {
    case 2: go(gemm_kernel<S, MT, 2, AMAX>); break;
    case 3: go(gemm_kernel<S, MT, 3, AMAX>); break;
    case 6: go(gemm_kernel<S, MT, 6, AMAX>); break;
    case 8: go(gemm_kernel<S, MT, 8, AMAX>); break;
    default: go(gemm_kernel<S, MT, 4, AMAX>); break;
  }
}

// 128-row chunks (bf16 only) run with 8 waves
template <bool AMAX>
static hipError_t launch_mt8(const GemmPlan& pl, GemmParams& p, hipStream_t st, const LaunchTiming* lt) {
  dim3 grid(8 * ((pl.ngroups * pl.S + 7) / 8) * pl.mchunks), block(pl.nw * 64);
  auto go = [&](auto kern) {
    if (lt) hipExtLaunchKernelGGL(kern, grid, block, (uint32_t)pl.lds_bytes, st, lt->start, lt->stop, 0, p);
    else hipLaunchKernelGGL(kern, grid, block, pl.lds_bytes, st, p);
  };
  if (pl.nw != 8) return hipErrorInvalidValue;
  go(gemm_kernel<bf16_t, 8, 8, AMAX>);
  return hipSuccess;
}

template <typename S>
static hipError_t launch_gemm_t(GemmParams& p, const GemmPlan& pl, hipStream_t st, const LaunchTiming* lt) {
  if (pl.mt == 8) {
    if constexpr (std::is_same<S, bf16_t>::value) {
      const hipError_t e = p.amax_part ? launch_mt8<true>(pl, p, st, lt) : launch_mt8<false>(pl, p, st, lt);
      if (e != hipSuccess) return e;
      return hipGetLastError();
    }
    return hipErrorInvalidValue;
  }
  if (p.amax_part) {
    switch (pl.mt) {
      case 1: launch_nw<S, 1, true>(pl, p, st, lt); break;
      case 2: launch_nw<S, 2, true>(pl, p, st, lt); break;
      default: launch_nw<S, 4, true>(pl, p, st, lt); break;
    }
  } else {
    switch (pl.mt) {
      case 1: launch_nw<S, 1, false>(pl, p, st, lt); break;
      case 2: launch_nw<S, 2, false>(pl, p, st, lt); break;
      default: launch_nw<S, 4, false>(pl, p, st, lt); break;
    }
  }
  return hipGetLastError();
}

hipError_t launch_gemm(int dtype, GemmParams& p, hipStream_t st, const LaunchTiming* lt) {
  const int maxs = p.mode == EP_PARTIAL && !p.amax_part ? std::max(1, p.max_splits) : 1;
  int seg_tiles[3];
  for (int s = 0; s < p.nseg && s < 3; ++s) seg_tiles[s] = p.seg[s].tiles;
  const GemmPlan pl = plan_gemm(dtype, p.M, p.ntiles, p.nchunks, p.mode == EP_SWIGLU, maxs, p.mode, seg_tiles,
                                std::min(p.nseg, 3), p.amax_part != nullptr);
  p.ngroups = pl.ngroups;
  p.mchunks = pl.mchunks;
  p.S = pl.S;
  p.cps = pl.cps;
  if (p.M <= 0) {  // nothing to launch: an empty timed interval
    if (lt) {
      (void)hipEventRecord(lt->start, st);
      (void)hipEventRecord(lt->stop, st);
    }
    return hipSuccess;
  }
  if (pl.tiled == 2) return launch_wide(p, pl, st, lt);
  if (pl.tiled) return launch_tiled(p, pl, st, lt);
  return dtype == 1 ? launch_gemm_t<bf16_t>(p, pl, st, lt) : launch_gemm_t<float>(p, pl, st, lt);
}

// Q|K|V finished from K-split partials part[s][m][pc] (packed column order), summed in split
// order, then rotary and stores with the same arithmetic as the fused epilogue (qkv_store8).
// One thread per (row, 8-column half of a 16-column tile).  Thread 2t holds the first half of
// a tile and 2t + 1 its rotary partners, so each reads only its own 8 columns and takes the
// partner sums from the neighbouring lane (DPP quad swap).  Every load (partials, rotary
// factors, KV slot) is issued before any is used: one memory round trip.
static constexpr int FIX_QKV_MAXS = 4;
template <typename S, int NS>
__global__ __launch_bounds__(256) void qkv_fix_kernel(const GemmParams p, const float* __restrict__ part, int N) {
  const int N8 = N >> 3, id = blockIdx.x * 256 + threadIdx.x;
  // rows past M (the grid's last workgroup) read row M - 1 and store nothing, so every lane
  // takes part in the partner exchange
  const int m_raw = id / N8, m = min(m_raw, p.M - 1), pc0 = (id % N8) * 8;
  const QkvCols8 cols = qkv_cols8(p, pc0);
  float4 pa[NS][2];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const float* r = part + ((size_t)s * p.M + m) * N + pc0;
    pa[s][0] = *reinterpret_cast<const float4*>(r);
    pa[s][1] = *reinterpret_cast<const float4*>(r + 4);
  }
  float4 cs4[4];
  qkv_cs8(p, m, cols, cs4);
  const int kb = p.row_kb[m];
  float v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    v[0] += pa[s][0].x; v[1] += pa[s][0].y; v[2] += pa[s][0].z; v[3] += pa[s][0].w;
    v[4] += pa[s][1].x; v[5] += pa[s][1].y; v[6] += pa[s][1].z; v[7] += pa[s][1].w;
  }
  // partner sums: lane id ^ 1 (the same row, the other half of the tile)
  float w[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) w[e] = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v[e]), 0xB1, 0xF, 0xF, true));
  if (m_raw >= p.M) return;
  qkv_store8<S>(p, m, cols, v, w, cs4, kb);
}

template <typename S>
static void launch_qkv_fix_t(const GemmParams& p, const float* part, int S_, int N, dim3 grid, hipStream_t st) {
  switch (S_) {
    case 1: hipLaunchKernelGGL((qkv_fix_kernel<S, 1>), grid, dim3(256), 0, st, p, part, N); break;
    case 2: hipLaunchKernelGGL((qkv_fix_kernel<S, 2>), grid, dim3(256), 0, st, p, part, N); break;
    case 3: hipLaunchKernelGGL((qkv_fix_kernel<S, 3>), grid, dim3(256), 0, st, p, part, N); break;
    default: hipLaunchKernelGGL((qkv_fix_kernel<S, 4>), grid, dim3(256), 0, st, p, part, N); break;
  }
}

hipError_t launch_qkv_fix(int dtype, const GemmParams& p, const float* part, int S, hipStream_t st) {
  const int N = (p.n_heads + 2 * p.n_kv) * p.hd;
  if (p.M <= 0) return hipSuccess;
  if (N % 16 || p.hd % 16 || S < 1 || S > FIX_QKV_MAXS) return hipErrorInvalidValue;
  // a whole number of 256-thread workgroups; partner lanes (2t, 2t + 1) share a row
  dim3 grid((unsigned)(((size_t)p.M * (N / 8) + 255) / 256));
  if (dtype == 1) launch_qkv_fix_t<bf16_t>(p, part, S, N, grid, st);
  else launch_qkv_fix_t<float>(p, part, S, N, grid, st);
  return hipGetLastError();
}

// ---- packing ------------------------------------------------------------------------------

template <typename S>
__global__ void pack_kernel(const S* __restrict__ src, int rows, int cols, S* __restrict__ dst, int rope_hd) {
  constexpr int EPL = St<S>::EPL, KC = 4 * EPL;
  const int nchunks = cols / KC;
  const size_t nvec = (size_t)(rows / 16) * nchunks * 64;
  for (size_t v = blockIdx.x * (size_t)blockDim.x + threadIdx.x; v < nvec;
       v += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(v % 64);
    const size_t tc = v / 64;
    const int c = (int)(tc % nchunks);
    const int t = (int)(tc / nchunks);
    const int n = rope_hd ? rope_row(t, lane & 15, rope_hd) : t * 16 + (lane & 15);
    const int k = c * KC + (lane >> 4) * EPL;
    *reinterpret_cast<u32x4_t*>(dst + v * EPL) =
        *reinterpret_cast<const u32x4_t*>(src + (size_t)n * cols + k);
  }
}

size_t packed_matrix_bytes(int dtype, int rows, int cols) {
  return (size_t)rows * cols * es_of(dtype);
}

hipError_t launch_pack(int dtype, const void* src, int rows, int cols, void* dst, int rope_hd,
                       hipStream_t st) {
  const int rope = rope_hd;
  if (rope && (rope % 16 || rows % rope)) return hipErrorInvalidValue;
  const size_t nvec = (size_t)rows * cols * es_of(dtype) / 16;
  const int grid = (int)std::min<size_t>((nvec + 255) / 256, 65536);
  if (dtype == 1)
    hipLaunchKernelGGL(pack_kernel<bf16_t>, dim3(grid), dim3(256), 0, st,
                       (const bf16_t*)src, rows, cols, (bf16_t*)dst, rope);
  else
    hipLaunchKernelGGL(pack_kernel<float>, dim3(grid), dim3(256), 0, st, (const float*)src, rows,
                       cols, (float*)dst, rope);
  return hipGetLastError();
}

}  // namespace clover
