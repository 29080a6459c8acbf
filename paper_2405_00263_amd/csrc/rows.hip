// Row-wise kernels of the Clover step: token embedding, RMSNorm, the Regressive
// Connection embedding and Attention Decoder mini-attention (Sec. 3.1, 3.2, 3.4), and
// the shared LM head's reductions (greedy argmax for verification, top-k with
// log-softmax for drafting).
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace clover {

// ---- embedding: x[m] = emb[tok[m]] --------------------------------------------------------
template <typename S>
__global__ void embed_kernel(const S* __restrict__ emb, const int* __restrict__ tok, int d,
                             float* __restrict__ x) {
  const int m = blockIdx.x;
  const S* row = emb + (size_t)tok[m] * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) x[(size_t)m * d + k] = St<S>::to_f(row[k]);
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
  v = warp_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// ---- RMSNorm: out[m] = x[m] / sqrt(mean(x^2) + eps) * g, stored in the storage type ---------
template <typename S>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ x, int ldx, int d,
                                                      const S* __restrict__ gain, float eps,
                                                      S* __restrict__ out, int ldo,
                                                      float* __restrict__ copy) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  const float* xr = x + (size_t)m * ldx;
  float ss = 0.f;
  for (int k = threadIdx.x; k < d; k += 256) ss += xr[k] * xr[k];
  ss = block_sum256(ss, red);
  const float rinv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int k = threadIdx.x; k < d; k += 256) {
    const float v = xr[k];
    out[(size_t)m * ldo + k] = St<S>::from_f(v * rinv * St<S>::to_f(gain[k]));
    if (copy) copy[(size_t)m * d + k] = v;
  }
}

hipError_t launch_rmsnorm(int dtype, const float* x, int ldx, int M, int d, const void* g,
                          float eps, void* out, int ldo, float* copy, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(M), dim3(256), 0, st, x, ldx, d,
                       (const bf16_t*)g, eps, (bf16_t*)out, ldo, copy);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(M), dim3(256), 0, st, x, ldx, d,
                       (const float*)g, eps, (float*)out, ldo, copy);
  return hipGetLastError();
}

// ---- argmax (lowest index on ties) ---------------------------------------------------------
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

static constexpr int RED_THREADS = 512;

__global__ __launch_bounds__(RED_THREADS) void argmax_kernel(const float* __restrict__ logits, int V,
                                                             int* __restrict__ out) {
  __shared__ float sv[RED_THREADS / 64];
  __shared__ int si[RED_THREADS / 64];
  const int m = blockIdx.x;
  const float* row = logits + (size_t)m * V;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int k = threadIdx.x; k < V; k += RED_THREADS) {
    const float v = row[k];
    if (better(v, k, bv, bi)) { bv = v; bi = k; }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o);
    const int oi = __shfl_xor(bi, o);
    if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { sv[w] = bv; si[w] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < RED_THREADS / 64; ++i)
      if (better(sv[i], si[i], bv, bi)) { bv = sv[i]; bi = si[i]; }
    out[m] = bi;
  }
}

hipError_t launch_argmax(const float* logits, int M, int V, int* out, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  hipLaunchKernelGGL(argmax_kernel, dim3(M), dim3(RED_THREADS), 0, st, logits, V, out);
  return hipGetLastError();
}

// ---- top-k with log-softmax ----------------------------------------------------------------
static constexpr int KMAX = 16;

__global__ __launch_bounds__(RED_THREADS) void topk_kernel(const TopkParams p) {
  __shared__ float sv[RED_THREADS / 64];
  __shared__ int si[RED_THREADS / 64];
  __shared__ float sm[RED_THREADS / 64], ss[RED_THREADS / 64];
  __shared__ float res_v[KMAX];
  __shared__ int res_i[KMAX];
  const int m = blockIdx.x;
  const float* row = p.logits + (size_t)m * p.V;
  const int k = p.k;  // 1..KMAX; each thread keeps its KMAX best, a superset of its k best
  float lv[KMAX];
  int li[KMAX];
#pragma unroll
  for (int i = 0; i < KMAX; ++i) { lv[i] = -INFINITY; li[i] = 0x7fffffff; }
  float mx = -INFINITY, se = 0.f;
  for (int c = threadIdx.x; c < p.V; c += RED_THREADS) {
    float v = row[c];
    // running log-sum-exp
    if (v > mx) { se = se * expf(mx - v) + 1.f; mx = v; }
    else se += expf(v - mx);
    // sorted insertion into the thread's list (static indices only)
    if (better(v, c, lv[KMAX - 1], li[KMAX - 1])) {
      int ci = c;
#pragma unroll
      for (int i = 0; i < KMAX; ++i) {
        if (better(v, ci, lv[i], li[i])) {
          const float tv = lv[i]; const int ti = li[i];
          lv[i] = v; li[i] = ci; v = tv; ci = ti;
        }
      }
    }
  }
  // block log-sum-exp
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(mx, o), os = __shfl_xor(se, o);
    const float nm = fmaxf(mx, om);
    se = (mx == -INFINITY ? 0.f : se * expf(mx - nm)) + (om == -INFINITY ? 0.f : os * expf(om - nm));
    mx = nm;
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { sm[w] = mx; ss[w] = se; }
  __syncthreads();
  float M = sm[0];
  for (int i = 1; i < RED_THREADS / 64; ++i) M = fmaxf(M, sm[i]);
  float S = 0.f;
  for (int i = 0; i < RED_THREADS / 64; ++i) S += ss[i] * expf(sm[i] - M);
  const float lse = M + logf(S);
  // merge: k rounds of block-wide best over list heads
  for (int r = 0; r < k; ++r) {
    float bv = lv[0];
    int bi = li[0];
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o);
      const int oi = __shfl_xor(bi, o);
      if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    __syncthreads();
    if ((threadIdx.x & 63) == 0) { sv[w] = bv; si[w] = bi; }
    __syncthreads();
    bv = sv[0]; bi = si[0];
    for (int i = 1; i < RED_THREADS / 64; ++i)
      if (better(sv[i], si[i], bv, bi)) { bv = sv[i]; bi = si[i]; }
    if (threadIdx.x == 0) { res_v[r] = bv; res_i[r] = bi; }
    if (li[0] == bi) {  // the owner pops its head
#pragma unroll
      for (int i = 0; i < KMAX - 1; ++i) { lv[i] = lv[i + 1]; li[i] = li[i + 1]; }
      lv[KMAX - 1] = -INFINITY; li[KMAX - 1] = 0x7fffffff;
    }
  }
  __syncthreads();
  if (threadIdx.x < k) {
    const int r = threadIdx.x;
    const float logp = res_v[r] - lse;
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

hipError_t launch_topk(TopkParams& p, hipStream_t st) {
  if (p.M <= 0) return hipSuccess;
  if (p.k < 1 || p.k > KMAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(topk_kernel, dim3(p.M), dim3(RED_THREADS), 0, st, p);
  return hipGetLastError();
}

// ---- Attention Decoder input preparation (Sec. 3.2 Eq. 1, Sec. 3.4) -------------------------
// For frontier row f: h = parent state, a = RMSNorm_ad(h), e = W_lm[token] / ||W_lm[token]||.
template <typename S>
__global__ __launch_bounds__(256) void ad_prep_kernel(const AdPrepParams p) {
  using T = St<S>;
  __shared__ float red[4];
  const int f = blockIdx.x, b = f / p.F, fl = f % p.F;
  const int slot = p.seq_ids[b];
  const int d = p.d;
  const float* h = p.use_slot_state ? p.prev + (size_t)slot * d
                                    : p.prev + (size_t)(b * p.Fprev + fl / p.kprev) * d;
  const int tok = p.cand_token[(size_t)slot * p.cand_stride + p.base_node + fl];
  const S* lm = reinterpret_cast<const S*>(p.lm_packed);
  float ss = 0.f, se = 0.f;
  for (int k = threadIdx.x; k < d; k += 256) {
    const float v = h[k];
    ss += v * v;
    const float w = T::to_f(lm[packed_index(tok, k, p.lm_nchunks, T::EPL)]);
    se += w * w;
  }
  ss = block_sum256(ss, red);
  se = block_sum256(se, red);
  const float rinv = 1.0f / sqrtf(ss / (float)d + p.eps);
  const float einv = 1.0f / fmaxf(sqrtf(se), 1e-12f);
  const S* gain = reinterpret_cast<const S*>(p.ad_norm);
  S* a = reinterpret_cast<S*>(p.a_out) + (size_t)f * d;
  S* e = reinterpret_cast<S*>(p.e_out) + (size_t)f * d;
  for (int k = threadIdx.x; k < d; k += 256) {
    const float v = h[k];
    p.hin[(size_t)f * d + k] = v;
    a[k] = T::from_f(v * rinv * T::to_f(gain[k]));
    e[k] = T::from_f(T::to_f(lm[packed_index(tok, k, p.lm_nchunks, T::EPL)]) * einv);
  }
}

hipError_t launch_ad_prep(int dtype, AdPrepParams& p, hipStream_t st) {
  const int M = p.nbatch * p.F;
  if (M <= 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(ad_prep_kernel<bf16_t>, dim3(M), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(ad_prep_kernel<float>, dim3(M), dim3(256), 0, st, p);
  return hipGetLastError();
}

// ---- Attention Decoder attention (Eq. 1-2): one key per frontier row ----------------------
// q: [M][H*hd] f32, kv: [M][2*H*hd] f32 (keys then values).  The softmax is taken over
// the key set of the row, which holds the single embedding e_{i-1}.
template <typename S>
__global__ __launch_bounds__(64) void ad_attn_kernel(const float* __restrict__ q,
                                                     const float* __restrict__ kv, int H, int hd,
                                                     S* __restrict__ out) {
  const int f = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int qd = H * hd;
  const float* qr = q + (size_t)f * qd + h * hd;
  const float* kr = kv + (size_t)f * 2 * qd + h * hd;
  const float* vr = kv + (size_t)f * 2 * qd + qd + h * hd;
  float dot = 0.f;
  for (int i = lane; i < hd; i += 64) dot += qr[i] * kr[i];
  dot = warp_sum(dot);
  const float s = dot * rsqrtf((float)hd);
  const float mx = s;                 // max over the single key
  const float pw = expf(s - mx);      // = 1
  const float l = pw;
  for (int i = lane; i < hd; i += 64)
    out[(size_t)f * qd + h * hd + i] = St<S>::from_f(pw * vr[i] / l);
}

hipError_t launch_ad_attn(int dtype, const float* q, const float* kv, int M, int n_heads, int hd,
                          void* out, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  dim3 grid(M, n_heads);
  if (dtype == 1)
    hipLaunchKernelGGL(ad_attn_kernel<bf16_t>, grid, dim3(64), 0, st, q, kv, n_heads, hd, (bf16_t*)out);
  else
    hipLaunchKernelGGL(ad_attn_kernel<float>, grid, dim3(64), 0, st, q, kv, n_heads, hd, (float*)out);
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
