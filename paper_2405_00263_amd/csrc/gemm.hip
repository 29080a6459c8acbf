// Weight-streaming GEMM for small M on gfx950 matrix cores.
//
//   Y[M][N] = X[M][K] * W[N][K]^T, fused epilogues (residual, rotary + KV append,
//   SwiGLU, head MLP).
//
// Decoding streams every weight once per forward while only M (= tree tokens) rows
// use it, so the kernel is bound by HBM bandwidth (Sec. 1 of the paper: decoding is
// memory-bound).  Design:
//  * weights are pre-tiled (packed_index) so one wave's 16-byte-per-lane load of a
//    16 x KC fragment is 1 KB of contiguous memory, streamed with non-temporal loads
//    and a register prefetch ring;
//  * a workgroup is 4 waves, one 16-row weight tile each (64 output columns), all
//    sharing the X tile, which is staged through LDS in double-buffered stages; X is
//    prefetched into registers as many stages ahead as the weight ring, so waiting for
//    an X load never forces younger weight loads to land (loads complete in order);
//  * Q/K weights of 128-wide heads are packed with their rotary halves interleaved by
//    16-row tiles, so a 64-row group holds complete rotary pairs;
//  * K may be split over workgroups (EP_PARTIAL): each split writes its own fp32
//    partial [split][M][N] and the consumer kernel sums them in split order, so the
//    result does not depend on scheduling and no cross-workgroup synchronisation (and
//    no device-scope fence, which on gfx950 writes back and invalidates the L2) is
//    needed inside the GEMM;
//  * fused epilogues (rotary + KV append, SwiGLU) run unsplit on an LDS tile.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace clover {

static constexpr int GEMM_WAVES = 4;
static constexpr int GEMM_THREADS = GEMM_WAVES * 64;
static constexpr int STAGE_CHUNKS = 4;   // chunks of X per LDS stage
static constexpr int PF = 16;            // weight fragments in flight per wave (16 KB)
static constexpr int TILE_STRIDE = 68;   // floats per row of the 64-column epilogue tile
static constexpr int TARGET_WGS = 256;
static constexpr int RING = PF / STAGE_CHUNKS;  // stages covered by the prefetch ring

template <typename S>
__device__ __forceinline__ const u32x4_t* wave_weight_ptr(const GemmParams& p, int g, int wave,
                                                          bool& active) {
  int seg = 0, t;
  if (p.mode == EP_SWIGLU) {
    seg = wave >> 1;
    t = g * 2 + (wave & 1);
    active = t < p.seg[seg].tiles;
  } else {
    t = g * GEMM_WAVES + wave;
    active = t < p.ntiles;
    while (active && seg < p.nseg - 1 && t >= p.seg[seg].tiles) {
      t -= p.seg[seg].tiles;
      ++seg;
    }
  }
  if (!active) return nullptr;
  return reinterpret_cast<const u32x4_t*>(p.seg[seg].w) + (size_t)t * p.nchunks * 64;
}

// logical 16-row tile of physical tile p in a rotary-interleaved Q/K weight (128-wide heads)
__host__ __device__ __forceinline__ int rope_tile(int p) {
  const int q = p & 7;
  return (p & ~7) + ((q & 1) ? 4 + (q >> 1) : (q >> 1));
}

template <typename S>
__device__ void gemm_epilogue(const GemmParams& p, const float* tile, int g, int m0, int mrows,
                              const int* s_pos, const int* s_kvbase) {
  using T = St<S>;
  const int tid = threadIdx.x;
  constexpr int COLS = GEMM_WAVES * 16;
  if (p.mode == EP_SWIGLU) {
    const int F = p.N;
    for (int e = tid; e < mrows * 32; e += GEMM_THREADS) {
      const int r = e >> 5, j = e & 31, m = m0 + r, n = g * 32 + j;
      if (m >= p.M || n >= F) continue;
      const float gt = tile[r * TILE_STRIDE + j], up = tile[r * TILE_STRIDE + 32 + j];
      reinterpret_cast<S*>(p.out_s)[(size_t)m * p.ldos + n] = T::from_f(silu_f(gt) * up);
    }
    return;
  }
  // EP_QKV.  Each thread owns one column of the 64-wide tile (GEMM_THREADS % 64 == 0).
  const int col = tid & (COLS - 1), w = col >> 4, jj = col & 15;
  const int hd = p.hd, half = hd >> 1, qd = p.n_heads * hd, kvd = p.n_kv * hd;
  const int pt = g * GEMM_WAVES + w;  // physical tile over [q; k; v]
  const int qt = qd / 16, kt = kvd / 16;
  if (pt >= qt + 2 * kt) return;
  int n, pc;  // logical output column, partner column in the tile
  if (hd == 128 && pt < qt + kt) {  // interleaved rotary halves
    const int seg0 = pt < qt ? 0 : qt;
    n = seg0 * 16 + rope_tile(pt - seg0) * 16 + jj;
    pc = ((w ^ 1) << 4) + jj;
  } else {
    n = pt * 16 + jj;
    const int dd = n % hd;
    pc = dd < half ? col + half : col - half;
  }
  const int d = n % hd;
  const bool rot = n < qd + kvd;
  double inv = 0.0;
  if (rot) inv = pow((double)p.theta, -2.0 * (double)((d < half) ? d : d - half) / (double)hd);
  for (int r = tid / COLS; r < mrows; r += GEMM_THREADS / COLS) {
    const int m = m0 + r;
    if (m >= p.M) break;
    float v = tile[r * TILE_STRIDE + col];
    if (rot) {
      const float partner = tile[r * TILE_STRIDE + pc];
      double ang = (double)s_pos[r] * inv;
      ang -= 6.283185307179586 * rint(ang * 0.15915494309189535);
      float sn, cs;
      sincosf((float)ang, &sn, &cs);
      v = (d < half) ? (v * cs - partner * sn) : (v * cs + partner * sn);
    }
    if (n < qd) {
      reinterpret_cast<S*>(p.qbuf)[(size_t)m * p.ldq + n] = T::from_f(v);
    } else {
      const bool isk = n < qd + kvd;
      const int kvh = (isk ? n - qd : n - qd - kvd) / hd;
      const int kb = s_kvbase[r];  // physical block * 16 + key
      const size_t base = ((size_t)(kb >> 4) * p.n_kv + kvh) * (size_t)(16 * hd);
      const int key = kb & 15;
      if (isk)
        reinterpret_cast<S*>(p.kcache)[base + kblk_off(key, d, T::EPL)] = T::from_f(v);
      else
        reinterpret_cast<S*>(p.vcache)[base + vblk_off(key, d)] = T::from_f(v);
    }
  }
}

template <typename S, int MT>
__global__ __launch_bounds__(GEMM_THREADS) void gemm_kernel(const GemmParams p) {
  using T = St<S>;
  constexpr int EPL = T::EPL, KC = 4 * EPL, MROWS = 16 * MT;
  constexpr int XSTRIDE = STAGE_CHUNKS * KC + EPL;          // elements per LDS row
  constexpr int XBUF = MROWS * XSTRIDE;                      // elements per stage buffer
  constexpr int VEC_PER_ROW = STAGE_CHUNKS * 4;              // 16-byte vectors per row per stage
  constexpr int XVEC = (MROWS * VEC_PER_ROW + GEMM_THREADS - 1) / GEMM_THREADS;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  S* xs = reinterpret_cast<S*>(smem);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = blockIdx.x, split = blockIdx.y, mc = blockIdx.z;
  const int m0 = mc * MROWS;
  const int c0 = split * p.cps;
  const int c1 = min(p.nchunks, c0 + p.cps);
  const int nk = c1 - c0;
  const int nst = (nk + STAGE_CHUNKS - 1) / STAGE_CHUNKS;

  // row metadata of the fused rotary + KV-append epilogue, loaded once up front so the
  // epilogue's row loop has no dependent global loads
  __shared__ int s_pos[MROWS], s_kvbase[MROWS];
  if (p.mode == EP_QKV && threadIdx.x < MROWS) {
    const int m = min(m0 + (int)threadIdx.x, p.M - 1);
    const int slot = p.row_slot[m];
    s_pos[threadIdx.x] = p.row_pos[m];
    s_kvbase[threadIdx.x] = p.block_table[(size_t)p.row_seq[m] * p.max_blocks + (slot >> 4)] * 16 + (slot & 15);
  }

  bool active;
  const u32x4_t* wp = wave_weight_ptr<S>(p, g, wave, active);
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
      const int v = min(threadIdx.x + i * GEMM_THREADS, MROWS * VEC_PER_ROW - 1);
      const int r = min(v / VEC_PER_ROW, p.M - 1 - m0), cv = v % VEC_PER_ROW;
      const int cchunk = min(st * STAGE_CHUNKS + cv / 4, nk - 1);
      regs[i] = *reinterpret_cast<const u32x4_t*>(X + (size_t)(m0 + r) * p.ldx +
                                                  (size_t)(c0 + cchunk) * KC + (cv % 4) * EPL);
    }
  };
  auto store_x = [&](int buf, const u32x4_t* regs) {
#pragma unroll
    for (int i = 0; i < XVEC; ++i) {
      const int v = threadIdx.x + i * GEMM_THREADS;
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
  static_assert(PF == RING * STAGE_CHUNKS, "ring covers whole stages");
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

  const int col = wave * 16 + (lane & 15);
  if (p.mode == EP_PARTIAL) {
    // split `split` writes rows m0.. of its own [M][N] fp32 slice
    if (!active) return;
    const int n = (g * GEMM_WAVES + wave) * 16 + (lane & 15);  // segments are contiguous in N
    float* out = p.part + (size_t)split * p.M * p.N;
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + t * 16 + 4 * (lane >> 4) + r;
        if (m < p.M) out[(size_t)m * p.N + n] = acc[t][r];
      }
    return;
  }
  float* tile = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int t = 0; t < MT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) tile[(t * 16 + 4 * (lane >> 4) + r) * TILE_STRIDE + col] = acc[t][r];
  __syncthreads();
  gemm_epilogue<S>(p, tile, g, m0, MROWS, s_pos, s_kvbase);
}

// ---- host side ------------------------------------------------------------------------

static int es_of(int dtype) { return dtype == 1 ? 2 : 4; }

GemmPlan plan_gemm(int dtype, int M, int ntiles, int nchunks, bool swiglu, int max_splits) {
  GemmPlan pl{};
  pl.mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  const int mrows = 16 * pl.mt;
  pl.mchunks = (M + mrows - 1) / mrows;
  pl.ngroups = swiglu ? ((ntiles / 2) + 1) / 2 : (ntiles + GEMM_WAVES - 1) / GEMM_WAVES;
  const int base = pl.ngroups * pl.mchunks;
  int S = 1;
  if (max_splits > 1) {
    S = (TARGET_WGS + base - 1) / base;
    S = std::max(1, std::min({S, max_splits, nchunks / (2 * STAGE_CHUNKS)}));
  }
  int cps = (nchunks + S - 1) / S;
  S = (nchunks + cps - 1) / cps;
  pl.S = S;
  pl.cps = cps;
  const int es = es_of(dtype), EPL = 16 / es, KC = 4 * EPL;
  const size_t xbytes = 2ull * mrows * (STAGE_CHUNKS * KC + EPL) * es;
  const size_t tbytes = (size_t)mrows * TILE_STRIDE * 4;
  pl.lds_bytes = std::max(xbytes, tbytes);
  pl.part_floats = (size_t)S * M * ntiles * 16;
  return pl;
}

template <typename S>
static hipError_t launch_gemm_t(GemmParams& p, const GemmPlan& pl, hipStream_t st) {
  dim3 grid(pl.ngroups, pl.S, pl.mchunks), block(GEMM_THREADS);
  switch (pl.mt) {
    case 1: hipLaunchKernelGGL((gemm_kernel<S, 1>), grid, block, pl.lds_bytes, st, p); break;
    case 2: hipLaunchKernelGGL((gemm_kernel<S, 2>), grid, block, pl.lds_bytes, st, p); break;
    default: hipLaunchKernelGGL((gemm_kernel<S, 4>), grid, block, pl.lds_bytes, st, p); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(int dtype, GemmParams& p, hipStream_t st) {
  const int maxs = p.mode == EP_PARTIAL ? std::max(1, p.max_splits) : 1;
  const GemmPlan pl = plan_gemm(dtype, p.M, p.ntiles, p.nchunks, p.mode == EP_SWIGLU, maxs);
  p.ngroups = pl.ngroups;
  p.mchunks = pl.mchunks;
  p.S = pl.S;
  p.cps = pl.cps;
  if (p.M <= 0) return hipSuccess;
  return dtype == 1 ? launch_gemm_t<bf16_t>(p, pl, st) : launch_gemm_t<float>(p, pl, st);
}

// ---- packing ------------------------------------------------------------------------------

template <typename S>
__global__ void pack_kernel(const S* __restrict__ src, int rows, int cols, S* __restrict__ dst, int rope) {
  constexpr int EPL = St<S>::EPL, KC = 4 * EPL;
  const int nchunks = cols / KC;
  const size_t nvec = (size_t)(rows / 16) * nchunks * 64;
  for (size_t v = blockIdx.x * (size_t)blockDim.x + threadIdx.x; v < nvec;
       v += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(v % 64);
    const size_t tc = v / 64;
    const int c = (int)(tc % nchunks);
    const int t = (int)(tc / nchunks);
    const int n = (rope ? rope_tile(t) : t) * 16 + (lane & 15);
    const int k = c * KC + (lane >> 4) * EPL;
    *reinterpret_cast<u32x4_t*>(dst + v * EPL) =
        *reinterpret_cast<const u32x4_t*>(src + (size_t)n * cols + k);
  }
}

size_t packed_matrix_bytes(int dtype, int rows, int cols) {
  return (size_t)rows * cols * es_of(dtype);
}

hipError_t launch_pack(int dtype, const void* src, int rows, int cols, void* dst, bool rope_interleave,
                       hipStream_t st) {
  const int rope = rope_interleave ? 1 : 0;
  if (rope && rows % 128) return hipErrorInvalidValue;
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
