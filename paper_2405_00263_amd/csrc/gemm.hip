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
//  * a workgroup is 8 waves, one 16-row weight tile each (128 output columns), all
//    sharing the X tile, which is staged through LDS in double-buffered stages;
//  * K is split over workgroups to fill 256 CUs; the last workgroup of a column group
//    (per-group counter) sums the partials in split order, so results do not depend
//    on arrival order, then runs the epilogue on an LDS tile.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace clover {

static constexpr int GEMM_WAVES = 8;
static constexpr int GEMM_THREADS = GEMM_WAVES * 64;
static constexpr int STAGE_CHUNKS = 4;   // chunks of X per LDS stage
static constexpr int PF = 8;             // weight fragments in flight per wave
static constexpr int TILE_STRIDE = 132;  // floats per row of the epilogue tile
static constexpr int TARGET_WGS = 512;

template <typename S>
__device__ __forceinline__ const u32x4_t* wave_weight_ptr(const GemmParams& p, int g, int wave,
                                                          bool& active) {
  int seg = 0, t;
  if (p.mode == EP_SWIGLU) {
    seg = wave >> 2;
    t = g * 4 + (wave & 3);
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

template <typename S>
__device__ void gemm_epilogue(const GemmParams& p, const float* tile, int g, int m0, int mrows) {
  using T = St<S>;
  const int tid = threadIdx.x;
  if (p.mode == EP_SWIGLU) {
    const int F = p.N;
    for (int e = tid; e < mrows * 64; e += GEMM_THREADS) {
      const int r = e >> 6, j = e & 63, m = m0 + r, n = g * 64 + j;
      if (m >= p.M || n >= F) continue;
      const float gt = tile[r * TILE_STRIDE + j], up = tile[r * TILE_STRIDE + 64 + j];
      reinterpret_cast<S*>(p.out_s)[(size_t)m * p.ldos + n] = T::from_f(silu_f(gt) * up);
    }
    return;
  }
  // Each thread owns one column of the 128-wide tile (GEMM_THREADS is a multiple of 128).
  const int col = tid & 127, n = g * 128 + col;
  if (n >= p.N) return;
  // rotary constants of this column
  const int hd = p.hd, half = hd >> 1, qd = p.n_heads * hd, kvd = p.n_kv * hd;
  const int d = n % hd;
  const bool rot = p.mode == EP_QKV && n < qd + kvd;
  const int pc = (d < half) ? col + half : col - half;
  double inv = 0.0;
  if (rot) inv = pow((double)p.theta, -2.0 * (double)((d < half) ? d : d - half) / (double)hd);
  const float bias = (p.mode == EP_HEAD) ? T::to_f(reinterpret_cast<const S*>(p.bias)[n]) : 0.f;
  for (int r = tid >> 7; r < mrows; r += GEMM_THREADS / 128) {
    const int m = m0 + r;
    if (m >= p.M) break;
    float v = tile[r * TILE_STRIDE + col];
    switch (p.mode) {
      case EP_F32:
        p.out_f[(size_t)m * p.ldo + n] = v;
        break;
      case EP_RESID: {
        const float o = p.resid[(size_t)m * p.ldr + n] + v;
        p.out_f[(size_t)m * p.ldo + n] = o;
        if (p.out_s) reinterpret_cast<S*>(p.out_s)[(size_t)m * p.ldos + n] = T::from_f(o);
        break;
      }
      case EP_HEAD: {
        const float o = p.resid[(size_t)m * p.ldr + n] + silu_f(v + bias);
        p.out_f[(size_t)m * p.ldo + n] = o;
        if (p.out_s) reinterpret_cast<S*>(p.out_s)[(size_t)m * p.ldos + n] = T::from_f(o);
        break;
      }
      case EP_QKV: {
        if (rot) {
          const float partner = tile[r * TILE_STRIDE + pc];
          double ang = (double)p.row_pos[m] * inv;
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
          const int seq = p.row_seq[m], slot = p.row_slot[m];
          const size_t base = kv_block_base(p.block_table, p.max_blocks, seq, slot, kvh, p.n_kv, hd);
          const int key = slot & 15;
          if (isk)
            reinterpret_cast<S*>(p.kcache)[base + kblk_off(key, d, T::EPL)] = T::from_f(v);
          else
            reinterpret_cast<S*>(p.vcache)[base + vblk_off(key, d)] = T::from_f(v);
        }
        break;
      }
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

  bool active;
  const u32x4_t* wp = wave_weight_ptr<S>(p, g, wave, active);
  if (active) wp += (size_t)c0 * 64 + lane;

  // weight prefetch ring
  u32x4_t wb[PF];
#pragma unroll
  for (int u = 0; u < PF; ++u)
    if (active && u < nk) wb[u] = __builtin_nontemporal_load(wp + (size_t)u * 64);

  // X stage loader: rows m0.., chunks [c0 + st*STAGE_CHUNKS, ...)
  const S* X = reinterpret_cast<const S*>(p.X);
  auto load_x = [&](int st, u32x4_t* regs) {
#pragma unroll
    for (int i = 0; i < XVEC; ++i) {
      const int v = threadIdx.x + i * GEMM_THREADS;
      u32x4_t val = {0u, 0u, 0u, 0u};
      const int r = v / VEC_PER_ROW, cv = v % VEC_PER_ROW;
      const int cchunk = st * STAGE_CHUNKS + cv / 4;
      if (v < MROWS * VEC_PER_ROW && m0 + r < p.M && cchunk < nk)
        val = *reinterpret_cast<const u32x4_t*>(X + (size_t)(m0 + r) * p.ldx +
                                                (size_t)(c0 + cchunk) * KC + (cv % 4) * EPL);
      regs[i] = val;
    }
  };
  auto store_x = [&](int buf, const u32x4_t* regs) {
#pragma unroll
    for (int i = 0; i < XVEC; ++i) {
      const int v = threadIdx.x + i * GEMM_THREADS;
      if (v < MROWS * VEC_PER_ROW) {
        const int r = v / VEC_PER_ROW, cv = v % VEC_PER_ROW;
        *reinterpret_cast<u32x4_t*>(xs + buf * XBUF + r * XSTRIDE + cv * EPL) = regs[i];
      }
    }
  };

  u32x4_t xr[XVEC];
  load_x(0, xr);
  store_x(0, xr);
  __syncthreads();

  f32x4_t acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Stages alternate between the two LDS buffers; walking them in pairs keeps the
  // prefetch-ring slot (chunk % PF, PF = 2 stages) a compile-time index.
  static_assert(PF == 2 * STAGE_CHUNKS, "ring covers two stages");
  for (int st0 = 0; st0 < nst; st0 += 2) {
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      const int st = st0 + par;
      if (st < nst) {
        if (st + 1 < nst) load_x(st + 1, xr);
        const S* xb = xs + par * XBUF + (lane & 15) * XSTRIDE + (lane >> 4) * EPL;
        if (active) {
#pragma unroll
          for (int u = 0; u < STAGE_CHUNKS; ++u) {
            const int c = st * STAGE_CHUNKS + u;
            if (c < nk) {
              const u32x4_t w = wb[par * STAGE_CHUNKS + u];
              if (c + PF < nk) wb[par * STAGE_CHUNKS + u] = __builtin_nontemporal_load(wp + (size_t)(c + PF) * 64);
              const S* xc = xb + u * KC;
#pragma unroll
              for (int t = 0; t < MT; ++t) {
                const u32x4_t a = *reinterpret_cast<const u32x4_t*>(xc + t * 16 * XSTRIDE);
                acc[t] = mma_frag(a, w, acc[t], S{});
              }
            }
          }
        }
        if (st + 1 < nst) store_x(par ^ 1, xr);
        __syncthreads();
      }
    }
  }

  float* tile = reinterpret_cast<float*>(smem);
  const int col = wave * 16 + (lane & 15);
  if (p.S == 1) {
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) tile[(t * 16 + 4 * (lane >> 4) + r) * TILE_STRIDE + col] = acc[t][r];
    __syncthreads();
  } else {
    const size_t tile_elems = (size_t)MROWS * 128;
    float* pp = p.part + ((size_t)(mc * p.ngroups + g) * p.S + split) * tile_elems;
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) pp[(t * 16 + 4 * (lane >> 4) + r) * 128 + col] = acc[t][r];
    __threadfence();
    __syncthreads();
    __shared__ int last;
    if (threadIdx.x == 0) {
      int* sem = p.sem + mc * p.ngroups + g;
      const int old = atomicAdd(sem, 1);
      last = (old == p.S - 1);
      if (last) atomicExch(sem, 0);
    }
    __syncthreads();
    if (!last) return;
    __threadfence();
    const float* base = p.part + (size_t)(mc * p.ngroups + g) * p.S * tile_elems;
    for (int e = threadIdx.x; e < MROWS * 128; e += GEMM_THREADS) {
      float v = 0.f;
      for (int s2 = 0; s2 < p.S; ++s2) v += __builtin_nontemporal_load(base + (size_t)s2 * tile_elems + e);
      tile[(e >> 7) * TILE_STRIDE + (e & 127)] = v;
    }
    __syncthreads();
  }
  gemm_epilogue<S>(p, tile, g, m0, MROWS);
}

// ---- host side ------------------------------------------------------------------------

static int es_of(int dtype) { return dtype == 1 ? 2 : 4; }

GemmPlan plan_gemm(int dtype, int M, int ntiles, int nchunks, bool swiglu) {
  GemmPlan pl{};
  pl.mt = M <= 16 ? 1 : (M <= 32 ? 2 : 4);
  const int mrows = 16 * pl.mt;
  pl.mchunks = (M + mrows - 1) / mrows;
  pl.ngroups = swiglu ? ((ntiles / 2) + 3) / 4 : (ntiles + GEMM_WAVES - 1) / GEMM_WAVES;
  const int base = pl.ngroups * pl.mchunks;
  int S = (TARGET_WGS + base - 1) / base;
  S = std::max(1, std::min(S, nchunks / 2));
  int cps = (nchunks + S - 1) / S;
  S = (nchunks + cps - 1) / cps;
  pl.S = S;
  pl.cps = cps;
  const int es = es_of(dtype), EPL = 16 / es, KC = 4 * EPL;
  const size_t xbytes = 2ull * mrows * (STAGE_CHUNKS * KC + EPL) * es;
  const size_t tbytes = (size_t)mrows * TILE_STRIDE * 4;
  pl.lds_bytes = std::max(xbytes, tbytes);
  pl.part_floats = S > 1 ? (size_t)base * S * mrows * 128 : 0;
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
  const GemmPlan pl = plan_gemm(dtype, p.M, p.ntiles, p.nchunks, p.mode == EP_SWIGLU);
  p.ngroups = pl.ngroups;
  p.mchunks = pl.mchunks;
  p.S = pl.S;
  p.cps = pl.cps;
  if (p.M <= 0) return hipSuccess;
  return dtype == 1 ? launch_gemm_t<bf16_t>(p, pl, st) : launch_gemm_t<float>(p, pl, st);
}

// ---- packing ------------------------------------------------------------------------------

template <typename S>
__global__ void pack_kernel(const S* __restrict__ src, int rows, int cols, S* __restrict__ dst) {
  constexpr int EPL = St<S>::EPL, KC = 4 * EPL;
  const int nchunks = cols / KC;
  const size_t nvec = (size_t)(rows / 16) * nchunks * 64;
  for (size_t v = blockIdx.x * (size_t)blockDim.x + threadIdx.x; v < nvec;
       v += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(v % 64);
    const size_t tc = v / 64;
    const int c = (int)(tc % nchunks);
    const int t = (int)(tc / nchunks);
    const int n = t * 16 + (lane & 15);
    const int k = c * KC + (lane >> 4) * EPL;
    *reinterpret_cast<u32x4_t*>(dst + v * EPL) =
        *reinterpret_cast<const u32x4_t*>(src + (size_t)n * cols + k);
  }
}

size_t packed_matrix_bytes(int dtype, int rows, int cols) {
  return (size_t)rows * cols * es_of(dtype);
}

hipError_t launch_pack(int dtype, const void* src, int rows, int cols, void* dst, hipStream_t st) {
  const size_t nvec = (size_t)rows * cols * es_of(dtype) / 16;
  const int grid = (int)std::min<size_t>((nvec + 255) / 256, 65536);
  if (dtype == 1)
    hipLaunchKernelGGL(pack_kernel<bf16_t>, dim3(grid), dim3(256), 0, st,
                       (const bf16_t*)src, rows, cols, (bf16_t*)dst);
  else
    hipLaunchKernelGGL(pack_kernel<float>, dim3(grid), dim3(256), 0, st, (const float*)src, rows,
                       cols, (float*)dst);
  return hipGetLastError();
}

}  // namespace clover
