// Row-wise kernels of the Clover step: token embedding, RMSNorm, the Regressive
// Connection embedding and Attention Decoder mini-attention (Sec. 3.1, 3.2, 3.4), and
// the shared LM head's reductions (greedy argmax for verification, top-k with
// log-softmax for drafting).
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace clover {

// ---- embedding: x[m] = emb[tok[m]] --------------------------------------------------------
// 16-byte vectors of storage elements <-> floats
__device__ __forceinline__ void vec_unpack(u32x4_t v, float* out, bf16_t) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(v[i] << 16);
    out[2 * i + 1] = __uint_as_float(v[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void vec_unpack(u32x4_t v, float* out, float) {
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = __uint_as_float(v[i]);
}
__device__ __forceinline__ u32x4_t vec_pack(const float* in, bf16_t) {
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = (uint32_t)f2bf(in[2 * i]) | ((uint32_t)f2bf(in[2 * i + 1]) << 16);
  return v;
}
__device__ __forceinline__ u32x4_t vec_pack(const float* in, float) {
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(in[i]);
  return v;
}

template <typename S>
__global__ void embed_kernel(const S* __restrict__ emb, const int* __restrict__ tok, int d,
                             float* __restrict__ x) {
  // 16-byte segments of the embedding row (EPL elements each), widened to float
  constexpr int EPL = St<S>::EPL;
  const int m = blockIdx.x;
  const u32x4_t* row = reinterpret_cast<const u32x4_t*>(emb + (size_t)tok[m] * d);
  float* out = x + (size_t)m * d;
  for (int sg = threadIdx.x; sg < d / EPL; sg += blockDim.x) {
    float v[EPL];
    vec_unpack(row[sg], v, S{});
#pragma unroll
    for (int q = 0; q < EPL / 4; ++q)
      *reinterpret_cast<float4*>(out + sg * EPL + 4 * q) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  }
}

// Rotary factors of each row's position (rotate-half pairing): the angle is formed and
// reduced to [-pi, pi] in double precision, then sin/cos are taken in single precision.
__global__ void rope_table_kernel(const int* __restrict__ pos, int M, int hd, float theta,
                                  float* __restrict__ cs, const int* __restrict__ seq,
                                  const int* __restrict__ slot, const int* __restrict__ bt,
                                  int max_blocks, int* __restrict__ kb) {
  const int half = hd / 2;
  if (kb)
    for (int m = blockIdx.x * blockDim.x + threadIdx.x; m < M; m += gridDim.x * blockDim.x) {
      const int s = slot[m];
      kb[m] = bt[(size_t)seq[m] * max_blocks + (s >> 4)] * 16 + (s & 15);
    }
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < M * half; e += gridDim.x * blockDim.x) {
    const int m = e / half, i = e % half;
    const double inv = pow((double)theta, -2.0 * (double)i / (double)hd);
    double ang = (double)pos[m] * inv;
    ang -= 6.283185307179586 * rint(ang * 0.15915494309189535);
    float sn, c;
    sincosf((float)ang, &sn, &c);
    cs[2 * (size_t)e] = c;
    cs[2 * (size_t)e + 1] = sn;
  }
}

hipError_t launch_rope_table(const int* pos, int M, int hd, float theta, float* cs, hipStream_t st,
                             const int* seq, const int* slot, const int* block_table, int max_blocks, int* kb) {
  if (M <= 0) return hipSuccess;
  if (kb && (!seq || !slot || !block_table || max_blocks <= 0)) return hipErrorInvalidValue;
  const int n = M * (hd / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3((n + 255) / 256), dim3(256), 0, st, pos, M, hd, theta, cs,
                     seq, slot, block_table, max_blocks, kb);
  return hipGetLastError();
}

hipError_t launch_embed(int dtype, const void* emb, const int* tok, int M, int d, float* x,
                        hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(M), dim3(256), 0, st, (const bf16_t*)emb, tok, d, x);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(256), 0, st, (const float*)emb, tok, d, x);
  return hipGetLastError();
}

// block-wide sum over 256 threads
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// ---- argmax (lowest index on ties) ---------------------------------------------------------
// Chunks of a row reduce to one key each (amax_key) and combine with a 64-bit atomic
// max, which is exact and order-independent, so the result is deterministic.
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

static constexpr int RED_THREADS = 256;
static constexpr int AMAX_CHUNKS = 32;

__global__ __launch_bounds__(RED_THREADS) void argmax_kernel(const float* __restrict__ logits, int V,
                                                             unsigned long long* __restrict__ keys) {
  const int m = blockIdx.x, ch = blockIdx.y;
  const int per = (V + AMAX_CHUNKS - 1) / AMAX_CHUNKS;
  const int c0 = ch * per, c1 = min(V, c0 + per);
  const float* row = logits + (size_t)m * V;
  unsigned long long best = 0ull;
  constexpr int U = 8;
  for (int c = c0 + threadIdx.x; c < c1; c += RED_THREADS * U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = c + u * RED_THREADS;
      v[u] = i < c1 ? row[i] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = c + u * RED_THREADS;
      if (i < c1) best = umax64(best, amax_key(v[u], i));
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long ob = ((unsigned long long)__shfl_xor((int)(best >> 32), o) << 32) |
                                  (uint32_t)__shfl_xor((int)(best & 0xffffffffu), o);
    best = umax64(best, ob);
  }
  if ((threadIdx.x & 63) == 0) atomicMax(keys + m, best);
}

__global__ void argmax_finish_kernel(const unsigned long long* __restrict__ keys, int M, int* __restrict__ out) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m < M) out[m] = 0x7fffffff - (int)(keys[m] & 0xffffffffu);
}

// Row m's argmax from the per-(group, row) keys a GEMM's epilogue left in keys[G][M].
__global__ __launch_bounds__(RED_THREADS) void argmax_groups_kernel(const unsigned long long* __restrict__ keys, int G,
                                                                    int M, int* __restrict__ out) {
  const int m = blockIdx.x;
  unsigned long long best = 0ull;
  for (int g = threadIdx.x; g < G; g += RED_THREADS) best = umax64(best, keys[(size_t)g * M + m]);
  best = umax64(best, max16_u64(best));
  best = umax64(best, shfl_xor_u64(best, 16));
  best = umax64(best, shfl_xor_u64(best, 32));
  __shared__ unsigned long long s_best[RED_THREADS / 64];
  if ((threadIdx.x & 63) == 0) s_best[threadIdx.x >> 6] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < RED_THREADS / 64; ++w) best = umax64(best, s_best[w]);
    out[m] = 0x7fffffff - (int)(best & 0xffffffffu);
  }
}

hipError_t launch_argmax_groups(const unsigned long long* keys, int G, int M, int* out, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (G < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(argmax_groups_kernel, dim3(M), dim3(RED_THREADS), 0, st, keys, G, M, out);
  return hipGetLastError();
}

__global__ void zero_u64_kernel(unsigned long long* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0ull;
}

hipError_t launch_argmax(const float* logits, int M, int V, int* out, unsigned long long* keys,
                         bool keys_zeroed, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (!keys_zeroed) hipLaunchKernelGGL(zero_u64_kernel, dim3((M + 255) / 256), dim3(256), 0, st, keys, M);
  hipLaunchKernelGGL(argmax_kernel, dim3(M, AMAX_CHUNKS), dim3(RED_THREADS), 0, st, logits, V, keys);
  hipLaunchKernelGGL(argmax_finish_kernel, dim3((M + 255) / 256), dim3(256), 0, st, keys, M, out);
  return hipGetLastError();
}

// ---- top-k with log-softmax, two stages ---------------------------------------------------
// Stage 1: each (row, chunk) workgroup finds its chunk's k best (value desc, index asc) and
// the chunk's (max, sum exp(x - max)).  Stage 2: one workgroup per row merges the chunk
// lists the same way and combines the chunk sums in chunk order into the log-sum-exp.
// Both stages select inside each wave first (k rounds of a wave-wide argmax over register-
// resident candidates, no barrier), then one wave selects among the waves' lists, so a
// stage costs two barriers whatever k is.
static constexpr int KMAX = 16;
static constexpr int TOPK_EPT = 16;  // elements per thread in stage 1
static constexpr int TOPK_S2 = 4;    // candidates per thread in stage 2
static constexpr int TOPK_WAVES = RED_THREADS / 64;
static_assert(TOPK_WAVES * KMAX <= 64, "one candidate per lane when the waves' lists merge");

// The k best of the wave's candidates (each lane holds N, index INT_MAX = empty) into
// res_v/res_i[0..k) (written by lane 0), best first.  The candidates taken are emptied.
// The wave's best (value, index) pair under `better`, left in every lane: rotations inside
// each 16-lane row (DPP), then the row pairs 16 and 32 lanes apart swapped in (VALU lane
// swaps) -- no LDS-routed shuffles.  `better` is a total order, so the result does not
// depend on the order of the comparisons.
__device__ __forceinline__ void wave_best_step(float& bv, int& bi, float ov, int oi) {
  if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
}
__device__ __forceinline__ void wave_best(float& bv, int& bi) {
  wave_best_step(bv, bi, __int_as_float(dpp_row_ror<8>(__float_as_int(bv))), dpp_row_ror<8>(bi));
  wave_best_step(bv, bi, __int_as_float(dpp_row_ror<4>(__float_as_int(bv))), dpp_row_ror<4>(bi));
  wave_best_step(bv, bi, __int_as_float(dpp_row_ror<2>(__float_as_int(bv))), dpp_row_ror<2>(bi));
  wave_best_step(bv, bi, __int_as_float(dpp_row_ror<1>(__float_as_int(bv))), dpp_row_ror<1>(bi));
  {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(bv), __float_as_uint(bv), false, false);
    const auto b = __builtin_amdgcn_permlane16_swap((unsigned)bi, (unsigned)bi, false, false);
    float v0 = __uint_as_float(a[0]);
    int i0 = (int)b[0];
    wave_best_step(v0, i0, __uint_as_float(a[1]), (int)b[1]);
    bv = v0; bi = i0;
  }
  {
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(bv), __float_as_uint(bv), false, false);
    const auto b = __builtin_amdgcn_permlane32_swap((unsigned)bi, (unsigned)bi, false, false);
    float v0 = __uint_as_float(a[0]);
    int i0 = (int)b[0];
    wave_best_step(v0, i0, __uint_as_float(a[1]), (int)b[1]);
    bv = v0; bi = i0;
  }
}

template <int N>
__device__ __forceinline__ void wave_topk(float (&v)[N], int (&ix)[N], int k, float* res_v, int* res_i) {
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int u = 0; u < N; ++u)
      if (better(v[u], ix[u], bv, bi)) { bv = v[u]; bi = ix[u]; }
    wave_best(bv, bi);
    if ((threadIdx.x & 63) == 0) { res_v[r] = bv; res_i[r] = bi; }
#pragma unroll
    for (int u = 0; u < N; ++u)
      if (ix[u] == bi && bi != 0x7fffffff) { v[u] = -INFINITY; ix[u] = 0x7fffffff; }
  }
}

// Lists of the workgroup's waves (s_v/s_i [TOPK_WAVES][KMAX]) merged by wave 0 into
// res_v/res_i[0..k).
__device__ __forceinline__ void merge_wave_lists(int k, const float* s_v, const int* s_i, float* res_v,
                                                 int* res_i) {
  if (threadIdx.x >= 64) return;
  const int lane = threadIdx.x, w = lane / KMAX, r = lane % KMAX;
  float v[1] = {(w < TOPK_WAVES && r < k) ? s_v[w * KMAX + r] : -INFINITY};
  int ix[1] = {(w < TOPK_WAVES && r < k) ? s_i[w * KMAX + r] : 0x7fffffff};
  wave_topk<1>(v, ix, k, res_v, res_i);
}

__global__ __launch_bounds__(RED_THREADS) void topk_stage1_kernel(const float* __restrict__ logits, int V, int k,
                                                                   int nch, float* __restrict__ pv,
                                                                   int* __restrict__ pi, float* __restrict__ pms) {
  __shared__ float sred[RED_THREADS / 64];
  __shared__ float s_v[TOPK_WAVES * KMAX];
  __shared__ int s_i[TOPK_WAVES * KMAX];
  const int m = blockIdx.x, ch = blockIdx.y;
  const int per = (V + nch - 1) / nch;
  const int c0 = ch * per, c1 = min(V, c0 + per);
  const float* row = logits + (size_t)m * V;
  float v[TOPK_EPT];
  int ix[TOPK_EPT];
  float mx = -INFINITY;
#pragma unroll
  for (int u = 0; u < TOPK_EPT; ++u) {
    const int i = c0 + threadIdx.x + u * RED_THREADS;
    v[u] = i < c1 ? row[i] : -INFINITY;
    ix[u] = i < c1 ? i : 0x7fffffff;
    mx = fmaxf(mx, v[u]);
  }
  // chunk max and sum of exponentials
  float bm = wave_max(mx);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sred[w] = bm;
  __syncthreads();
  float cmax = sred[0];
  for (int q = 1; q < RED_THREADS / 64; ++q) cmax = fmaxf(cmax, sred[q]);
  float se = 0.f;
#pragma unroll
  for (int u = 0; u < TOPK_EPT; ++u) se += (v[u] == -INFINITY) ? 0.f : expf(v[u] - cmax);
  se = wave_sum(se);
  // the wave's k best, then the chunk's from the waves' lists
  wave_topk<TOPK_EPT>(v, ix, k, s_v + w * KMAX, s_i + w * KMAX);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sred[w] = se;
  __syncthreads();
  if (threadIdx.x == 0) {
    float tot = 0.f;
    for (int q = 0; q < RED_THREADS / 64; ++q) tot += sred[q];
    pms[((size_t)m * nch + ch) * 2] = cmax;
    pms[((size_t)m * nch + ch) * 2 + 1] = tot;
  }
  merge_wave_lists(k, s_v, s_i, pv + ((size_t)m * nch + ch) * k, pi + ((size_t)m * nch + ch) * k);
}

__global__ __launch_bounds__(RED_THREADS) void topk_stage2_kernel(const TopkParams p, int nch,
                                                                   const float* __restrict__ pv,
                                                                   const int* __restrict__ pi,
                                                                   const float* __restrict__ pms) {
  __shared__ float s_v[TOPK_WAVES * KMAX];
  __shared__ int s_i[TOPK_WAVES * KMAX];
  __shared__ float res_v[KMAX];
  __shared__ int res_i[KMAX];
  __shared__ float s_lse;
  const int m = blockIdx.x, k = p.k;
  const int ncand = nch * k;  // <= TOPK_S2 * RED_THREADS
  float cv[TOPK_S2];
  int ci[TOPK_S2];
#pragma unroll
  for (int u = 0; u < TOPK_S2; ++u) {
    const int c = threadIdx.x + u * RED_THREADS;
    cv[u] = c < ncand ? pv[(size_t)m * ncand + c] : -INFINITY;
    ci[u] = c < ncand ? pi[(size_t)m * ncand + c] : 0x7fffffff;
  }
  if (threadIdx.x == 0) {
    float M = -INFINITY;
    for (int c = 0; c < nch; ++c) M = fmaxf(M, pms[((size_t)m * nch + c) * 2]);
    float S = 0.f;
    for (int c = 0; c < nch; ++c) {
      const float cm = pms[((size_t)m * nch + c) * 2];
      if (cm != -INFINITY) S += pms[((size_t)m * nch + c) * 2 + 1] * expf(cm - M);
    }
    s_lse = M + logf(S);
  }
  const int w = threadIdx.x >> 6;
  wave_topk<TOPK_S2>(cv, ci, k, s_v + w * KMAX, s_i + w * KMAX);
  __syncthreads();
  merge_wave_lists(k, s_v, s_i, res_v, res_i);
  __syncthreads();
  if (threadIdx.x < k) {
    const int r = threadIdx.x;
    const float logp = res_v[r] - s_lse;
    if (p.tok) {
      p.tok[(size_t)m * k + r] = res_i[r];
      p.logp[(size_t)m * k + r] = logp;
    }
    if (p.cand_token) {
      const int b = m / p.F, fl = m % p.F;
      const int slot = p.seq_ids[b];
      const size_t cb = (size_t)slot * p.cand_stride;
      const int parent = p.base_parent + fl;
      const int child = p.base_child + fl * k + r;
      p.cand_token[cb + child] = res_i[r];
      p.cand_parent[cb + child] = parent;
      p.cand_depth[cb + child] = p.depth;
      p.cand_lp[cb + child] = p.cand_lp[cb + parent] + logp;
    }
  }
}

// chunks per row: enough that one chunk fits the stage-1 registers, at most what the
// stage-2 merge holds
static int topk_chunks(int V, int k) {
  const int need = (V + TOPK_EPT * RED_THREADS - 1) / (TOPK_EPT * RED_THREADS);
  return std::max(need, std::min(32, TOPK_S2 * RED_THREADS / k));
}

size_t topk_scratch_floats(int M, int V, int k) { return (size_t)M * topk_chunks(V, k) * (2 * k + 2); }

hipError_t launch_topk(TopkParams& p, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  if (p.k < 1 || p.k > KMAX) return hipErrorInvalidValue;
  const int nch = topk_chunks(p.V, p.k);
  if (nch * p.k > TOPK_S2 * RED_THREADS) return hipErrorInvalidValue;
  float* pv = p.scratch;
  int* pi = reinterpret_cast<int*>(p.scratch + (size_t)p.M * nch * p.k);
  float* pms = p.scratch + (size_t)p.M * nch * 2 * p.k;
  hipLaunchKernelGGL(topk_stage1_kernel, dim3(p.M, nch), dim3(RED_THREADS), 0, st, p.logits, p.V, p.k, nch,
                     pv, pi, pms);
  hipLaunchKernelGGL(topk_stage2_kernel, dim3(p.M), dim3(RED_THREADS), 0, st, p, nch, pv, pi, pms);
  return hipGetLastError();
}

// ---- reduce split-K partials, residual, activation, RMSNorm ---------------------------------
// One workgroup per row.  result = resid + y with y = sum_s part[s] (act 0) or
// silu(sum_s part[s] + bias) (act 1), summed in split order; then optional copies and
// out_norm = RMSNorm(result) * gain in the storage type.
static constexpr int FIX_THREADS = 1024;
static constexpr int FIX_MAXS = 8;
static constexpr int FIX_VEC = 2;  // float4 per thread: d <= 8192

// four consecutive storage elements in one store
__device__ __forceinline__ void store4(bf16_t* p, float a, float b, float c, float d) {
  *reinterpret_cast<u32x2_t*>(p) = u32x2_t{(uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16),
                                           (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16)};
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}

// four consecutive storage elements as one packed load, unpacked to floats later
template <typename S> struct Raw4;
template <> struct Raw4<bf16_t> { typedef u32x2_t type; };
template <> struct Raw4<float> { typedef float4 type; };
__device__ __forceinline__ float4 raw4_to_f(u32x2_t r) {
  return make_float4(__uint_as_float(r[0] << 16), __uint_as_float(r[0] & 0xffff0000u), __uint_as_float(r[1] << 16),
                     __uint_as_float(r[1] & 0xffff0000u));
}
__device__ __forceinline__ float4 raw4_to_f(float4 r) { return r; }

// VEC float4 per thread (d <= VEC * 4096), NS split partials.  Every load is unconditional, at
// a clamped column (lanes past d re-read the row's last 4 elements and store nothing), and the
// gain and bias come from a valid row when unused, so all loads are in flight before the first
// use: one memory round trip.  The gain and bias stay packed storage words until then.
template <typename S, int VEC, int NS>
__global__ __launch_bounds__(FIX_THREADS) void rowfix_kernel(const RowFixParams p) {
  using T = St<S>;
  using R4 = typename Raw4<S>::type;
  __shared__ float red[FIX_THREADS / 64];
  const int m = blockIdx.x, d = p.d;
  if (p.zero_keys && m == 0)
    for (int i = threadIdx.x; i < p.zero_n; i += FIX_THREADS) p.zero_keys[i] = 0ull;
  const S* gp = reinterpret_cast<const S*>(p.out_norm ? p.gain : static_cast<const void*>(p.resid));
  const S* bp = reinterpret_cast<const S*>(p.act == 1 ? p.bias : static_cast<const void*>(p.resid));
  float4 acc[VEC];
  float4 part[NS > 0 ? NS : 1][VEC];
  float4 res[VEC];
  R4 graw[VEC], braw[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    const int e = min((int)threadIdx.x * 4 + i * FIX_THREADS * 4, d - 4);
    graw[i] = *reinterpret_cast<const R4*>(gp + e);
    braw[i] = *reinterpret_cast<const R4*>(bp + e);
    res[i] = *reinterpret_cast<const float4*>(p.resid + (size_t)m * p.ldr + e);
#pragma unroll
    for (int s = 0; s < NS; ++s) part[s][i] = *reinterpret_cast<const float4*>(p.part + ((size_t)s * p.M + m) * p.ldp + e);
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    const int e = threadIdx.x * 4 + i * FIX_THREADS * 4;
    float4 y = NS > 0 ? part[0][i] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int s = 1; s < NS; ++s) { y.x += part[s][i].x; y.y += part[s][i].y; y.z += part[s][i].z; y.w += part[s][i].w; }
    // the activation as a select, so the bias load is not moved behind a branch on act
    const float4 b = raw4_to_f(braw[i]);
    const bool act = p.act == 1;
    y.x = act ? silu_f(y.x + b.x) : y.x; y.y = act ? silu_f(y.y + b.y) : y.y;
    y.z = act ? silu_f(y.z + b.z) : y.z; y.w = act ? silu_f(y.w + b.w) : y.w;
    if (p.no_resid) res[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    float4 o = make_float4(res[i].x + y.x, res[i].y + y.y, res[i].z + y.z, res[i].w + y.w);
    acc[i] = o;
    if (e < d) {
      if (p.out_f) *reinterpret_cast<float4*>(p.out_f + (size_t)m * p.ldo + e) = o;
      if (p.out_copy_f) *reinterpret_cast<float4*>(p.out_copy_f + (size_t)m * d + e) = o;
      if (p.out_copy_s) store4(reinterpret_cast<S*>(p.out_copy_s) + (size_t)m * d + e, o.x, o.y, o.z, o.w);
      ss += o.x * o.x + o.y * o.y + o.z * o.z + o.w * o.w;
    }
  }
  if (!p.out_norm) return;
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int q = 0; q < FIX_THREADS / 64; ++q) tot += red[q];
  const float rinv = 1.0f / sqrtf(tot / (float)d + p.eps);
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    const int e = threadIdx.x * 4 + i * FIX_THREADS * 4;
    if (e >= d) continue;
    S* on = reinterpret_cast<S*>(p.out_norm) + (size_t)m * p.ldn + e;
    const float4 gn = raw4_to_f(graw[i]);
    store4(on, acc[i].x * rinv * gn.x, acc[i].y * rinv * gn.y, acc[i].z * rinv * gn.z, acc[i].w * rinv * gn.w);
  }
}

template <typename S, int VEC>
static void launch_rowfix_v(RowFixParams& p, hipStream_t st) {
  const dim3 g(p.M), b(FIX_THREADS);
  switch (p.S) {
    case 0: hipLaunchKernelGGL((rowfix_kernel<S, VEC, 0>), g, b, 0, st, p); break;
    case 1: hipLaunchKernelGGL((rowfix_kernel<S, VEC, 1>), g, b, 0, st, p); break;
    case 2: hipLaunchKernelGGL((rowfix_kernel<S, VEC, 2>), g, b, 0, st, p); break;
    case 3: hipLaunchKernelGGL((rowfix_kernel<S, VEC, 3>), g, b, 0, st, p); break;
    case 4: hipLaunchKernelGGL((rowfix_kernel<S, VEC, 4>), g, b, 0, st, p); break;
    case 5: hipLaunchKernelGGL((rowfix_kernel<S, VEC, 5>), g, b, 0, st, p); break;
    case 6: hipLaunchKernelGGL((rowfix_kernel<S, VEC, 6>), g, b, 0, st, p); break;
    case 7: hipLaunchKernelGGL((rowfix_kernel<S, VEC, 7>), g, b, 0, st, p); break;
    default: hipLaunchKernelGGL((rowfix_kernel<S, VEC, 8>), g, b, 0, st, p); break;
  }
}

template <typename S>
static void launch_rowfix_t(RowFixParams& p, hipStream_t st) {
  if (p.d <= FIX_THREADS * 4) launch_rowfix_v<S, 1>(p, st);
  else launch_rowfix_v<S, 2>(p, st);
}

hipError_t launch_rowfix(int dtype, RowFixParams& p, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  if (p.S < 0 || p.S > FIX_MAXS || p.d < 4 || p.d > FIX_VEC * FIX_THREADS * 4 || p.d % 4) return hipErrorInvalidValue;
  if ((p.S > 0 && !p.part) || (p.out_norm && !p.gain) || (p.act == 1 && !p.bias)) return hipErrorInvalidValue;
  // the residual is read unconditionally: without one the kernel reads the first partial's
  // rows in its place and zeroes them
  p.no_resid = 0;
  if (!p.resid) {
    if (p.S < 1) return hipErrorInvalidValue;
    p.resid = p.part;
    p.ldr = p.ldp;
    p.no_resid = 1;
  }
  if (dtype == 1) launch_rowfix_t<bf16_t>(p, st);
  else launch_rowfix_t<float>(p, st);
  return hipGetLastError();
}

// ---- Attention Decoder input preparation (Sec. 3.2 Eq. 1, Sec. 3.4) -------------------------
// For frontier row f: h = parent state, a = RMSNorm_ad(h), e = W_lm[token] / ||W_lm[token]||.
// Attention Decoder inputs of one frontier row (Sec. 3.2, 3.4): a = RMSNorm(h) * g (storage),
// e = W_lm[tok] / max(||W_lm[tok]||_2, 1e-12) (storage) and a float copy of h.  Each
// thread owns whole 16-byte segments s (elements [s*EPL, s*EPL + EPL)): of h, of the gain,
// and of the token's LM-head row, which the packed layout keeps as one vector per segment
// (fragment s/4, lane group s%4).  Everything is loaded once, up front; one combined
// reduction gives both norms.
static constexpr int AD_MAXV = 8;  // segments per thread: d <= 256 * 8 * EPL
template <typename S>
__global__ __launch_bounds__(256) void ad_prep_kernel(const AdPrepParams p) {
  using T = St<S>;
  constexpr int EPL = T::EPL;
  __shared__ float red[2][4];
  const int f = blockIdx.x, b = f / p.F, fl = f % p.F;
  const int slot = p.seq_ids[b];
  const int d = p.d, nseg = d / EPL;
  const float* h = p.use_slot_state ? p.prev + (size_t)slot * d
                                    : p.prev + (size_t)(b * p.Fprev + fl / p.kprev) * d;
  float hv[AD_MAXV][EPL];
#pragma unroll
  for (int i = 0; i < AD_MAXV; ++i) {
    const int sg = threadIdx.x + i * 256;
    if (sg < nseg) {
#pragma unroll
      for (int q = 0; q < EPL / 4; ++q) {
        const float4 v = *reinterpret_cast<const float4*>(h + (size_t)sg * EPL + 4 * q);
        hv[i][4 * q] = v.x; hv[i][4 * q + 1] = v.y; hv[i][4 * q + 2] = v.z; hv[i][4 * q + 3] = v.w;
      }
    }
  }
  const int tok = p.cand_token[(size_t)slot * p.cand_stride + p.base_node + fl];
  const u32x4_t* lm = reinterpret_cast<const u32x4_t*>(p.lm_packed) + (size_t)(tok >> 4) * p.lm_nchunks * 64 + (tok & 15);
  const u32x4_t* gain = reinterpret_cast<const u32x4_t*>(p.ad_norm);
  u32x4_t lv[AD_MAXV], gv[AD_MAXV];
#pragma unroll
  for (int i = 0; i < AD_MAXV; ++i) {
    const int sg = threadIdx.x + i * 256;
    if (sg < nseg) {
      lv[i] = lm[(size_t)(sg >> 2) * 64 + 16 * (sg & 3)];
      gv[i] = gain[sg];
    }
  }
  float ss = 0.f, se = 0.f;
  float ev[AD_MAXV][EPL];
#pragma unroll
  for (int i = 0; i < AD_MAXV; ++i) {
    const int sg = threadIdx.x + i * 256;
    if (sg < nseg) {
      vec_unpack(lv[i], ev[i], S{});
#pragma unroll
      for (int q = 0; q < EPL; ++q) {
        ss += hv[i][q] * hv[i][q];
        se += ev[i][q] * ev[i][q];
      }
    }
  }
  ss = wave_sum(ss);
  se = wave_sum(se);
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = ss;
    red[1][threadIdx.x >> 6] = se;
  }
  __syncthreads();
  ss = red[0][0] + red[0][1] + red[0][2] + red[0][3];
  se = red[1][0] + red[1][1] + red[1][2] + red[1][3];
  const float rinv = 1.0f / sqrtf(ss / (float)d + p.eps);
  const float einv = 1.0f / fmaxf(sqrtf(se), 1e-12f);
  const size_t ld = p.ld_out ? (size_t)p.ld_out : (size_t)d;
  u32x4_t* a = reinterpret_cast<u32x4_t*>(reinterpret_cast<S*>(p.a_out) + (size_t)f * ld);
  u32x4_t* e = reinterpret_cast<u32x4_t*>(reinterpret_cast<S*>(p.e_out) + (size_t)f * ld);
  float* hin = p.hin + (size_t)f * d;
#pragma unroll
  for (int i = 0; i < AD_MAXV; ++i) {
    const int sg = threadIdx.x + i * 256;
    if (sg < nseg) {
      float g[EPL], av[EPL], eo[EPL];
      vec_unpack(gv[i], g, S{});
#pragma unroll
      for (int q = 0; q < EPL; ++q) {
        av[q] = hv[i][q] * rinv * g[q];
        eo[q] = ev[i][q] * einv;
      }
      a[sg] = vec_pack(av, S{});
      e[sg] = vec_pack(eo, S{});
#pragma unroll
      for (int q = 0; q < EPL / 4; ++q)
        *reinterpret_cast<float4*>(hin + (size_t)sg * EPL + 4 * q) =
            make_float4(hv[i][4 * q], hv[i][4 * q + 1], hv[i][4 * q + 2], hv[i][4 * q + 3]);
    }
  }
}

hipError_t launch_ad_prep(int dtype, AdPrepParams& p, hipStream_t st) {
  const int M = p.nbatch * p.F;
  if (M <= 0) return hipSuccess;
  const int epl = dtype == 1 ? 8 : 4;
  if (p.d % epl || p.d > 256 * AD_MAXV * epl) return hipErrorInvalidValue;
  if (dtype == 1)
    hipLaunchKernelGGL(ad_prep_kernel<bf16_t>, dim3(M), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(ad_prep_kernel<float>, dim3(M), dim3(256), 0, st, p);
  return hipGetLastError();
}

// ---- Attention Decoder attention (Eq. 1-2) ----------------------------------------------
// One workgroup (one wave) per (frontier row, head).  The query and every key/value are the
// split-K sums of their GEMM partials; the softmax runs over the row's key set (see
// AdAttnParams) in fp32: scores q.k / sqrt(hd), max-subtracted exponentials, normalised
// weighted sum of the values.  With a single key the weight is exactly 1.
static constexpr int AD_MAX_KEYS = 9;   // path keys: one per depth 0..H-1, plus headroom
static constexpr int AD_DPL = 2;        // dims per lane: hd <= 128
template <typename S>
__global__ __launch_bounds__(64) void ad_attn_kernel(const AdAttnParams p) {
  const int f = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int qd = p.n_heads * p.hd, M = p.M, hd = p.hd;
  if (p.values_only) {  // one key: the output is its value (weight exactly 1)
#pragma unroll
    for (int u = 0; u < AD_DPL; ++u) {
      const int i = lane + 64 * u;
      if (i >= hd) continue;
      float v = 0.f;
      for (int s = 0; s < p.Skv; ++s) v += p.kv[((size_t)s * M + f) * qd + h * hd + i];
      reinterpret_cast<S*>(p.out)[(size_t)f * qd + h * hd + i] = St<S>::from_f(v);
    }
    return;
  }
  const int kvrows = p.keys == AD_KEYS_TWO ? 2 * M : M;
  // split-K sum of one key/value row of the K|V GEMM for this lane's dims
  auto sum_kv = [&](int row, float* k, float* v) {
#pragma unroll
    for (int u = 0; u < AD_DPL; ++u) {
      const int i = lane + 64 * u;
      k[u] = v[u] = 0.f;
      if (i < hd)
        for (int s = 0; s < p.Skv; ++s) {
          const float* r = p.kv + ((size_t)s * kvrows + row) * 2 * qd + h * hd + i;
          k[u] += r[0];
          v[u] += r[qd];
        }
    }
  };
  // key slots (static indices): path keys take slots 0..depth-1 for the ancestors and
  // `depth` for the row's own token; two keys take slot 0 for the state, 1 for the token
  const int own = p.keys == AD_KEYS_PATH ? p.depth : (p.keys == AD_KEYS_TWO ? 1 : 0);
  const int nk = own + 1;
  float ko[AD_DPL], vo[AD_DPL], ks[AD_DPL], vs[AD_DPL];
  sum_kv(p.keys == AD_KEYS_TWO ? M + f : f, ko, vo);
  if (p.keys == AD_KEYS_TWO) sum_kv(f, ks, vs);
  float kk[AD_MAX_KEYS][AD_DPL], vv[AD_MAX_KEYS][AD_DPL];
  const int b = f / p.F, fl = f % p.F;
#pragma unroll
  for (int t = 0; t < AD_MAX_KEYS; ++t) {
#pragma unroll
    for (int u = 0; u < AD_DPL; ++u) {
      const int i = lane + 64 * u;
      float k = ko[u], v = vo[u];
      if (t < own) {
        if (p.keys == AD_KEYS_TWO) {
          k = ks[u];
          v = vs[u];
        } else {  // path: the ancestor at depth t
          const size_t row = p.kv_path_off[t] + (size_t)b * p.path_nodes[t] + fl / p.anc_div[t];
          k = i < hd ? p.kv_path[row * 2 * qd + h * hd + i] : 0.f;
          v = i < hd ? p.kv_path[row * 2 * qd + qd + h * hd + i] : 0.f;
        }
      }
      kk[t][u] = k;
      vv[t][u] = v;
    }
  }
  if (p.keys == AD_KEYS_PATH) {  // this depth's rows for the deeper depths' path keys
    const size_t row = p.kv_path_off[p.depth] + f;
#pragma unroll
    for (int u = 0; u < AD_DPL; ++u) {
      const int i = lane + 64 * u;
      if (i < hd) {
        p.kv_path[row * 2 * qd + h * hd + i] = ko[u];
        p.kv_path[row * 2 * qd + qd + h * hd + i] = vo[u];
      }
    }
  }
  float q[AD_DPL];
#pragma unroll
  for (int u = 0; u < AD_DPL; ++u) {
    const int i = lane + 64 * u;
    float x = 0.f;
    if (i < hd)
      for (int s = 0; s < p.Sq; ++s) x += p.q[((size_t)s * M + f) * qd + h * hd + i];
    q[u] = x;
  }
  const float scale = rsqrtf((float)hd);
  float sc[AD_MAX_KEYS], mx = -INFINITY;
#pragma unroll
  for (int t = 0; t < AD_MAX_KEYS; ++t) {
    float dot = 0.f;
#pragma unroll
    for (int u = 0; u < AD_DPL; ++u) dot += q[u] * kk[t][u];
    sc[t] = wave_sum(dot) * scale;
    if (t < nk) mx = fmaxf(mx, sc[t]);
  }
  float l = 0.f;
#pragma unroll
  for (int t = 0; t < AD_MAX_KEYS; ++t) {
    sc[t] = t < nk ? expf(sc[t] - mx) : 0.f;  // a single key: exp(0) = 1
    l += sc[t];
  }
#pragma unroll
  for (int u = 0; u < AD_DPL; ++u) {
    const int i = lane + 64 * u;
    float o = 0.f;
#pragma unroll
    for (int t = 0; t < AD_MAX_KEYS; ++t) o += sc[t] * vv[t][u];
    if (i < hd) reinterpret_cast<S*>(p.out)[(size_t)f * qd + h * hd + i] = St<S>::from_f(o / l);
  }
}

hipError_t launch_ad_attn(int dtype, const AdAttnParams& p, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  if (p.hd > 64 * AD_DPL || p.keys < 0 || p.keys > AD_KEYS_PATH) return hipErrorInvalidValue;
  if (p.keys == AD_KEYS_PATH && (p.depth < 0 || p.depth >= AD_MAX_KEYS - 1 || p.depth >= 8 || !p.kv_path))
    return hipErrorInvalidValue;
  if (p.values_only && p.keys != AD_KEYS_SINGLE) return hipErrorInvalidValue;
  dim3 grid(p.M, p.n_heads);
  if (dtype == 1)
    hipLaunchKernelGGL(ad_attn_kernel<bf16_t>, grid, dim3(64), 0, st, p);
  else
    hipLaunchKernelGGL(ad_attn_kernel<float>, grid, dim3(64), 0, st, p);
  return hipGetLastError();
}

// Medusa heads read the target's hidden state of the last committed token (per slot):
// gathered into batch rows, as fp32 (the residual of the head block) and in the storage
// type (the head GEMM's input).
template <typename S>
__global__ __launch_bounds__(256) void gather_state_kernel(const int* __restrict__ seq_ids,
                                                           const float* __restrict__ h0, int d,
                                                           float* __restrict__ out_f, S* __restrict__ out_s) {
  const int b = blockIdx.x;
  const float* src = h0 + (size_t)seq_ids[b] * d;
  for (int k = threadIdx.x; k < d; k += 256) {
    const float v = src[k];
    out_f[(size_t)b * d + k] = v;
    out_s[(size_t)b * d + k] = St<S>::from_f(v);
  }
}

hipError_t launch_gather_state(int dtype, const int* seq_ids, int nbatch, const float* h0, int d,
                               float* out_f, void* out_s, hipStream_t st) {
  if (nbatch <= 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(gather_state_kernel<bf16_t>, dim3(nbatch), dim3(256), 0, st, seq_ids, h0, d, out_f,
                       (bf16_t*)out_s);
  else
    hipLaunchKernelGGL(gather_state_kernel<float>, dim3(nbatch), dim3(256), 0, st, seq_ids, h0, d, out_f,
                       (float*)out_s);
  return hipGetLastError();
}

__global__ void fill_i32_kernel(int* p, int v, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}
hipError_t launch_fill_i32(int* p, int v, size_t n, hipStream_t st) {
  if (!n) return hipSuccess;
  const int grid = (int)std::min<size_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(grid), dim3(256), 0, st, p, v, n);
  return hipGetLastError();
}

}  // namespace clover
