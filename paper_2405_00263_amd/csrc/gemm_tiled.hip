// Register-blocked matrix-core GEMM for large M (verify of big batches or big trees, prefill
// chunks), bf16 storage.
//
//   Y[M][N] = X[M][K] * W[N][K]^T with the same epilogues as the weight-streaming kernel.
//
// With hundreds of rows the tree-verify GEMMs reach the compute bound (Sec. 1 of the paper:
// large batches times large trees move decoding from memory- to compute-bound), so the
// design maximises matrix-core work per byte that reaches a compute unit:
//  * a workgroup is 4 waves over 16*MT rows and 4*TW 16-column weight tiles; each wave owns
//    TW tiles for all the rows, i.e. MT x TW accumulator fragments (8 x 4: 128 x 64 outputs
//    per wave, 128 x 256 per workgroup), so each weight fragment feeds MT products and each
//    X fragment TW;
//  * weight fragments go straight from the packed layout into registers (one 1 KB
//    fragment per load instruction, 16 bytes per lane, the exact operand layout) through a
//    RING-stage register prefetch ring; X goes through double-buffered LDS stages of two
//    32-wide k chunks, prefetched as far ahead as the weights;
//  * at the 128 x 256 tile a compute unit needs about 48 bytes per clock from L2 and 64 from
//    LDS at the matrix-core peak, within both limits; smaller tiles are not;
//  * the epilogues work on the accumulators in registers: the rotary partner (column ^ 8,
//    the same tile) is one lane exchange away, and the SwiGLU gate and up tiles of a column
//    sit in the same wave.
#include "common.h"
#include "gemm_epi.h"
#include "kernels.h"

#include <hip/hip_ext.h>

#include <algorithm>

namespace clover {

static constexpr int TWAVES = 4;  // waves per row of waves (column groups per workgroup)
static constexpr int TSC = 2;     // 32-wide k chunks per LDS stage

template <int MT, int TW, int RING, int WR, int AMAX>
__global__ __launch_bounds__(WR * TWAVES * 64) void tiled_kernel(const GemmParams p) {
  using S = bf16_t;
  using T = St<S>;
  constexpr int THREADS = WR * TWAVES * 64;
  constexpr int EPL = T::EPL, KC = 4 * EPL, WM = 16 * MT, BM = WR * WM, HT = TW / 2;
  constexpr int XSTRIDE = TSC * KC + EPL;  // elements per LDS row (16-byte pad: no bank conflicts)
  constexpr int XBUF = BM * XSTRIDE;
  constexpr int VPR = TSC * 4;             // 16-byte vectors per row per stage
  constexpr int XV = BM * VPR / THREADS;   // X vectors per thread per stage
  static_assert((BM * VPR) % THREADS == 0, "X stage must split evenly over the threads");
  static_assert(RING % 2 == 0, "stages alternate between two LDS buffers inside a superstage");
  static_assert(TW % 2 == 0, "SwiGLU pairs gate and up tiles inside a wave");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  S* xs = reinterpret_cast<S*>(smem);
  __shared__ int s_kvbase[BM];

  const int wave = (threadIdx.x >> 6) % TWAVES, wrow = (threadIdx.x >> 6) / TWAVES, lane = threadIdx.x & 63;
  // XCD-aware order as in the streaming kernel: the row chunks of one (group, split) take
  // consecutive ids on one XCD and find each other's weight tiles in its L2.
  const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3;
  const int mc = q % p.mchunks, r = (q / p.mchunks) * 8 + xcd;
  if (r >= p.ngroups * p.S) return;  // padding of the last round
  const int g = r % p.ngroups, split = r / p.ngroups;
  const int m0 = mc * BM;
  const int c0 = split * p.cps;
  const int c1 = min(p.nchunks, c0 + p.cps);
  const int nk = c1 - c0;
  const int nst = (nk + TSC - 1) / TSC;

  int kvb = 0;  // KV-append target of row threadIdx.x (fused epilogue), staged in LDS at the end
  if (p.mode == EP_QKV && threadIdx.x < BM) kvb = p.row_kb[min(m0 + (int)threadIdx.x, p.M - 1)];

  // This wave's weight tiles.  SwiGLU: tiles [0, HT) are gate tiles and [HT, TW) the up
  // tiles of the same columns.  Otherwise tile j is column tile (g*4 + wave)*TW + j over
  // the concatenated segments.  Tiles past the end stream tile 0 and store nothing.
  // (segment fields at constant indices: scalar loads of the argument block, selected per tile)
  const int tl0 = p.seg[0].tiles, tl1 = p.seg[1].tiles;
  const u32x4_t* w0 = reinterpret_cast<const u32x4_t*>(p.seg[0].w);
  const u32x4_t* w1 = reinterpret_cast<const u32x4_t*>(p.seg[1].w);
  const u32x4_t* w2 = reinterpret_cast<const u32x4_t*>(p.seg[2].w);
  const u32x4_t* wp[TW];
  int otile[TW];
  bool act[TW];
#pragma unroll
  for (int j = 0; j < TW; ++j) {
    int t;
    const u32x4_t* w = w0;
    if (p.mode == EP_SWIGLU) {
      t = (g * TWAVES + wave) * HT + (j % HT);
      act[j] = t < tl0;
      otile[j] = t;
      if (j >= HT) w = w1;
    } else {
      t = (g * TWAVES + wave) * TW + j;
      act[j] = t < p.ntiles;
      otile[j] = t;
      if (p.nseg > 1 && t >= tl0) {
        t -= tl0;
        w = w1;
        if (p.nseg > 2 && t >= tl1) {
          t -= tl1;
          w = w2;
        }
      }
    }
    const u32x4_t* base = act[j] ? w + (size_t)t * p.nchunks * 64 : w0;
    wp[j] = base + (size_t)c0 * 64 + lane;
  }

  // X stage loader: rows m0.., chunks [c0 + st*TSC, ...).  Addresses are clamped into range
  // so every load is unconditional; rows past M are zeroed at store time.
  const S* X = reinterpret_cast<const S*>(p.X);
  auto load_x = [&](int st, u32x4_t* regs) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int v = threadIdx.x + i * THREADS;
      const int rr = min(v / VPR, p.M - 1 - m0), cv = v % VPR;
      const int ch = min(st * TSC + cv / 4, nk - 1);
      regs[i] = *reinterpret_cast<const u32x4_t*>(X + (size_t)(m0 + rr) * p.ldx + (size_t)(c0 + ch) * KC +
                                                  (cv % 4) * EPL);
    }
  };
  auto store_x = [&](int buf, const u32x4_t* regs) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int v = threadIdx.x + i * THREADS;
      const int rr = v / VPR, cv = v % VPR;
      const u32x4_t zero = {0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4_t*>(xs + buf * XBUF + rr * XSTRIDE + cv * EPL) = (m0 + rr < p.M) ? regs[i] : zero;
    }
  };
  u32x4_t wb[RING][TSC][TW];
  auto load_w = [&](int st, u32x4_t (&dst)[TSC][TW]) {
#pragma unroll
    for (int u = 0; u < TSC; ++u)
#pragma unroll
      for (int j = 0; j < TW; ++j) dst[u][j] = wp[j][(size_t)min(st * TSC + u, nk - 1) * 64];
  };

  // Prologue: X then W of each of the first RING stages, in consumption order (loads
  // complete in order, so waiting for one never waits for a later-needed one).
  u32x4_t xr[RING][XV];
#pragma unroll
  for (int s = 0; s < RING; ++s) {
    load_x(s, xr[s]);
    load_w(s, wb[s]);
  }
  store_x(0, xr[0]);
  __syncthreads();

  f32x4_t acc[MT][TW];
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int j = 0; j < TW; ++j) acc[t][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // One stage: issue X(st + RING) into the slot stage st vacated, multiply the stage's
  // chunks (A fragments from LDS, weight fragments from the ring), refill each weight slot
  // right after its last use, stage X(st + 1) into the other LDS buffer.
  auto stage = [&](int st, int par, bool guard) {
    load_x(st + RING, xr[par]);
    const S* xb = xs + (par & 1) * XBUF + (wrow * WM + (lane & 15)) * XSTRIDE + (lane >> 4) * EPL;
#pragma unroll
    for (int u = 0; u < TSC; ++u) {
      const int c = st * TSC + u;
      if (!guard || c < nk) {
        u32x4_t a[MT];
#pragma unroll
        for (int t = 0; t < MT; ++t) a[t] = *reinterpret_cast<const u32x4_t*>(xb + u * KC + t * 16 * XSTRIDE);
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
          for (int j = 0; j < TW; ++j) acc[t][j] = mma_frag(a[t], wb[par][u][j], acc[t][j], S{});
      }
#pragma unroll
      for (int j = 0; j < TW; ++j) wb[par][u][j] = wp[j][(size_t)min(c + RING * TSC, nk - 1) * 64];
    }
    store_x((par & 1) ^ 1, xr[(par + 1) % RING]);
    __syncthreads();
  };
  const int nsuper = nk / (RING * TSC);  // whole superstages: branch-free
  for (int ss = 0; ss < nsuper; ++ss) {
#pragma unroll
    for (int par = 0; par < RING; ++par) stage(ss * RING + par, par, false);
  }
#pragma unroll
  for (int par = 0; par < RING; ++par) {
    const int st = nsuper * RING + par;
    if (st < nst) stage(st, par, true);
  }

  // Epilogues from the accumulators: fragment (t, j) element i is row
  // m0 + 16t + 4*(lane/16) + i, column 16*tile + lane%16.
  const int rbase = m0 + wrow * WM + 4 * (lane >> 4), ccol = lane & 15;
  if (p.mode == EP_PARTIAL) {
    // with argmax keys the logits themselves are optional (p.part null: keys only)
    float* out = p.part + (size_t)split * p.M * p.N;
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      if (!act[j] || (AMAX != 0 && !p.part)) continue;
      const int n = otile[j] * 16 + ccol;
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = rbase + t * 16 + i;
          if (m < p.M) out[(size_t)m * p.N + n] = acc[t][j][i];
        }
    }
    if constexpr (AMAX != 0) {
      // each row's best (value, column) over this group's columns: tiles, lanes, waves
      __syncthreads();  // the LDS stages are no longer read
      unsigned long long* s_key = reinterpret_cast<unsigned long long*>(smem);  // [TWAVES][BM]
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // this lane's best over its tiles (tiles ascend in column: strict > keeps the lowest)
          float v = -INFINITY;
          int n = 0x7fffffff;
          const int m = min(m0 + wrow * WM + t * 16 + 4 * (lane >> 4) + i, p.M - 1);  // rows past M: not stored
          uint32_t sslot = 0, sstep = 0;
          if constexpr (AMAX == 2) {
            sslot = (uint32_t)p.samp_slot[m];
            sstep = (uint32_t)p.samp_step[sslot];
          }
#pragma unroll
          for (int j = 0; j < TW; ++j) {
            float a = acc[t][j][i];
            if constexpr (AMAX == 2)
              a = gumbel_score_call(a, p.inv_temp, (uint32_t)(otile[j] * 16 + ccol), (uint32_t)(m % p.samp_rows),
                                    sstep, sslot, p.samp_seed, p.samp_domain);
            if (act[j] && a > v) {
              v = a;
              n = otile[j] * 16 + ccol;
            }
          }
          const unsigned long long k = row16_amax_key(v, n);
          if (ccol == 0) s_key[wave * BM + wrow * WM + t * 16 + 4 * (lane >> 4) + i] = k;
        }
      __syncthreads();
      for (int r = threadIdx.x; r < BM; r += THREADS) {
        if (m0 + r >= p.M) break;
        unsigned long long best = 0ull;
        for (int w = 0; w < TWAVES; ++w) best = umax64(best, s_key[w * BM + r]);
        p.amax_part[(size_t)g * p.M + m0 + r] = best;
      }
    }
  } else if (p.mode == EP_SWIGLU) {
    S* out = reinterpret_cast<S*>(p.out_s);
#pragma unroll
    for (int j = 0; j < HT; ++j) {
      if (!act[j]) continue;
      const int n = otile[j] * 16 + ccol;
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = rbase + t * 16 + i;
          if (m < p.M) out[(size_t)m * p.ldos + n] = T::from_f(silu_f(acc[t][j][i]) * acc[t][j + HT][i]);
        }
    }
  } else {  // EP_QKV
    // One tile at a time through this wave's slice of the (now idle) X buffers, so the
    // store loop (rotary partner = column ^ 8 of the same tile) is a short runtime loop and
    // the accumulators keep compile-time indices.
    constexpr int TS = 17;  // floats per LDS row
    static_assert(WR * TWAVES * WM * TS * 4 <= 2 * XBUF * 2, "epilogue tile fits the X buffers");
    float* tile = reinterpret_cast<float*>(smem) + (wrow * TWAVES + wave) * WM * TS;
    if (threadIdx.x < BM) s_kvbase[threadIdx.x] = kvb;
#pragma unroll
    for (int j = 0; j < TW; ++j) {
      __syncthreads();  // previous readers of this LDS space are done
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) tile[(t * 16 + 4 * (lane >> 4) + i) * TS + ccol] = acc[t][j][i];
      __syncthreads();
      if (!act[j]) continue;
      for (int e = lane; e < WM * 16; e += 64) {
        const int rr = e >> 4, c = e & 15, mr = wrow * WM + rr, m = m0 + mr;
        if (m < p.M) qkv_store<S>(p, m, otile[j] * 16 + c, tile[rr * TS + c], tile[rr * TS + (c ^ 8)], s_kvbase[mr]);
      }
    }
  }
}

// ---- host side ------------------------------------------------------------------------

namespace {
constexpr int N_CU = 256;
constexpr int MAX_SPLIT_WGS = 256;  // the rule splits K until the grid covers the CUs once

struct TiledShape {
  int mt, tw, ring, wr;
};
// Shapes the dispatcher instantiates.
constexpr TiledShape kShapes[] = {{4, 4, 2, 1}, {4, 4, 4, 1}, {4, 2, 4, 1}, {4, 4, 2, 2}, {4, 2, 4, 2}};

// Best (shape, split) of a forced-plan sweep on MI355X for the shapes of the shipped 7B
// workloads (d 4096, 32 heads of 128, SwiGLU 11008, vocab 125696) at the row counts they
// run: 512 (batch 8 x 64-token trees), 256 (prefill chunks, batch-8 draft) and 128
// (128-token trees).  At 64 rows the O and down projections alone ran 5-10% faster here
// than on the streaming kernel, but whole steps did not change, so 64 rows stay streaming.
struct TunedTiled {
  int M, ntiles, nchunks;
  bool swiglu;
  TiledShape sh;
  int S;
};
constexpr TunedTiled kTunedTiled[] = {
    {512, 768, 128, false, {4, 4, 2, 1}, 1},  {512, 1376, 128, true, {4, 4, 2, 1}, 1},
    {512, 256, 128, false, {4, 4, 2, 1}, 2},  {512, 256, 344, false, {4, 4, 2, 1}, 4},
    {512, 7856, 128, false, {4, 4, 2, 1}, 1}, {256, 768, 128, false, {4, 4, 4, 1}, 1},
    {256, 1376, 128, true, {4, 2, 4, 1}, 1},  {256, 256, 128, false, {4, 2, 4, 1}, 2},
    {256, 256, 344, false, {4, 4, 2, 1}, 4},  {128, 768, 128, false, {4, 2, 4, 1}, 1},
    {128, 1376, 128, true, {4, 2, 4, 2}, 1},  {128, 256, 128, false, {4, 2, 4, 1}, 4},
    {128, 256, 344, false, {4, 2, 4, 1}, 4},
};

GemmPlan make_plan(const TiledShape& sh, int M, int ntiles, int nchunks, bool swiglu, int S) {
  GemmPlan pl{};
  pl.tiled = 1;
  pl.nw = TWAVES * sh.wr;
  pl.mt = sh.mt;
  pl.tw = sh.tw;
  pl.ring = sh.ring;
  const int bm = 16 * sh.mt * sh.wr;
  pl.mchunks = (std::max(M, 1) + bm - 1) / bm;
  pl.ngroups = swiglu ? ((ntiles / 2) + TWAVES * (sh.tw / 2) - 1) / (TWAVES * (sh.tw / 2))
                      : (ntiles + TWAVES * sh.tw - 1) / (TWAVES * sh.tw);
  pl.cps = (nchunks + S - 1) / S;
  pl.S = (nchunks + pl.cps - 1) / pl.cps;
  pl.lds_bytes = std::max<size_t>(2ull * bm * (TSC * 32 + 8) * 2, 8ull * TWAVES * bm);  // X stages; argmax keys
  pl.part_floats = (size_t)pl.S * M * ntiles * 16;
  return pl;
}

int max_tiled_splits(const TiledShape& sh, int nchunks, int max_splits) {
  return std::max(1, std::min(max_splits, nchunks / (2 * TSC * sh.ring)));
}
}  // namespace

// A swept entry when there is one; otherwise 64 x 256 workgroup tiles (the most robust
// shape of the sweep) with K split until the grid covers the compute units once.
GemmPlan plan_tiled(int M, int ntiles, int nchunks, bool swiglu, int max_splits) {
  for (const TunedTiled& t : kTunedTiled)
    if (t.M == M && t.ntiles == ntiles && t.nchunks == nchunks && t.swiglu == swiglu &&
        t.S <= max_tiled_splits(t.sh, nchunks, max_splits))
      return make_plan(t.sh, M, ntiles, nchunks, swiglu, t.S);
  const TiledShape sh = kShapes[0];
  GemmPlan pl = make_plan(sh, M, ntiles, nchunks, swiglu, 1);
  const int smax = max_tiled_splits(sh, nchunks, max_splits);
  for (int S = 2; S <= smax && (long)pl.ngroups * pl.S * pl.mchunks < MAX_SPLIT_WGS; ++S) {
    const GemmPlan q = make_plan(sh, M, ntiles, nchunks, swiglu, S);
    if (q.S == S) pl = q;
  }
  return pl;
}

GemmPlan plan_tiled_forced(int M, int ntiles, int nchunks, bool swiglu, int mt, int tw, int ring, int nw, int S) {
  return make_plan(TiledShape{mt, tw, ring, nw / TWAVES}, M, ntiles, nchunks, swiglu, S);
}

template <int MT, int TW, int RING, int WR>
static void launch_shape(const GemmPlan& pl, GemmParams& p, hipStream_t st, const LaunchTiming* lt) {
  // argmax epilogue: greedy (1) or Gumbel-max sampling (2), separate instantiations so the
  // greedy one carries no generator code
  auto kern = !p.amax_part ? tiled_kernel<MT, TW, RING, WR, 0>
              : p.inv_temp != 0.f ? tiled_kernel<MT, TW, RING, WR, 2> : tiled_kernel<MT, TW, RING, WR, 1>;
  dim3 grid(8 * ((pl.ngroups * pl.S + 7) / 8) * pl.mchunks), block(WR * TWAVES * 64);
  if (lt) hipExtLaunchKernelGGL(kern, grid, block, (uint32_t)pl.lds_bytes, st, lt->start, lt->stop, 0, p);
  else hipLaunchKernelGGL(kern, grid, block, pl.lds_bytes, st, p);
}

hipError_t launch_tiled(GemmParams& p, const GemmPlan& pl, hipStream_t st, const LaunchTiming* lt) {
  const int wr = pl.nw / TWAVES;
  if (pl.mt == 4 && pl.tw == 4 && pl.ring == 2 && wr == 1) launch_shape<4, 4, 2, 1>(pl, p, st, lt);
  else if (pl.mt == 4 && pl.tw == 4 && pl.ring == 4 && wr == 1) launch_shape<4, 4, 4, 1>(pl, p, st, lt);
  else if (pl.mt == 4 && pl.tw == 2 && pl.ring == 4 && wr == 1) launch_shape<4, 2, 4, 1>(pl, p, st, lt);
  else if (pl.mt == 4 && pl.tw == 4 && pl.ring == 2 && wr == 2) launch_shape<4, 4, 2, 2>(pl, p, st, lt);
  else if (pl.mt == 4 && pl.tw == 2 && pl.ring == 4 && wr == 2) launch_shape<4, 2, 4, 2>(pl, p, st, lt);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace clover
