// Tree-masked attention over the paged KV cache (tree attention, Sec. 2.2 of the
// paper: the causal mask of the verify forward is the token tree's ancestor matrix).
//
// Each query row attends to every committed key (slots 0..P-1) and to the tail keys
// P..P+n_tail-1 its mask row admits: the tree's ancestor-or-self bits during verify,
// or the causal rule during chunked prefill.  The score product is computed
// transposed (S^T = K Q^T) so the matrix-core accumulator already holds, per lane,
// four consecutive keys of one query row: exactly the operand layout the P*V product
// needs, with no shuffles.  Softmax is online in the log2 domain.  Keys are split over
// the waves of a workgroup, whose states merge in LDS in wave order.
#include "common.h"
#include "kernels.h"

#include <hip/hip_ext.h>

#include <algorithm>

namespace clover {

static constexpr int ATT_WAVES = 8;              // key splits inside a workgroup
static constexpr int ATT_THREADS = ATT_WAVES * 64;
static constexpr int ATT_MAX_BLOCKS = 4096;    // 65536 keys

__device__ __forceinline__ f32x4_t mma_pv(u32x2_t v, const float p[4], f32x4_t c, bf16_t) {
  u32x2_t pb;
  pb[0] = (uint32_t)f2bf(p[0]) | ((uint32_t)f2bf(p[1]) << 16);
  pb[1] = (uint32_t)f2bf(p[2]) | ((uint32_t)f2bf(p[3]) << 16);
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, v),
                                                   __builtin_bit_cast(s16x4_t, pb), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mma_pv(u32x4_t v, const float p[4], f32x4_t c, float) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v[0]), p[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v[1]), p[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v[2]), p[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v[3]), p[3], c, 0, 0, 0);
  return c;
}

template <typename S> struct VFrag;
template <> struct VFrag<bf16_t> { typedef u32x2_t type; };
template <> struct VFrag<float> { typedef u32x4_t type; };

template <typename S, int HD>
struct KVBlock {
  static constexpr int EPL = St<S>::EPL, NQC = HD / (4 * EPL), NT = HD / 16;
  u32x4_t k[NQC];
  typename VFrag<S>::type v[NT];
  __device__ __forceinline__ void load(const S* kc, const S* vc, size_t base, int lane) {
#pragma unroll
    for (int c = 0; c < NQC; ++c)
      k[c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(kc + base + (size_t)(c * 64 + lane) * EPL));
#pragma unroll
    for (int t = 0; t < NT; ++t)
      v[t] = __builtin_nontemporal_load(
          reinterpret_cast<const typename VFrag<S>::type*>(vc + base + (size_t)(t * 64 + lane) * 4));
  }
};

// One workgroup = one 16-row query tile of one (sequence, head); its 8 waves take
// interleaved 16-key blocks and merge their online-softmax states through LDS.
// Workgroup ids are laid out so all query tiles of one (sequence, head) land on the
// same XCD (ids are dealt to the 8 XCDs round-robin) and share its L2 copy of K/V.
template <typename S, int HD>
__global__ __launch_bounds__(ATT_THREADS) void attn_kernel(const AttnParams p) {
  using T = St<S>;
  constexpr int EPL = T::EPL, KC = 4 * EPL, NQC = HD / KC, NT = HD / 16;
  constexpr int ATT_RING = sizeof(S) == 2 ? 3 : 2;  // 16-key blocks in flight per wave
  __shared__ float s_m[ATT_WAVES][16], s_l[ATT_WAVES][16];
  __shared__ float s_o[ATT_WAVES][16][HD + 4];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, j = lane & 15;
  const int id = blockIdx.x, xcd = id & 7, slotx = id >> 3;
  const int item = (slotx / p.qtiles) * 8 + xcd, qt = slotx % p.qtiles;
  if (item >= p.nbatch * p.n_heads) return;
  const int b = item / p.n_heads, h = item % p.n_heads;
  const int slot = p.seq_ids[b];
  const int P = p.prefix_dev ? p.prefix_dev[slot] : p.prefix_host;
  const int tail = p.causal ? min(p.n_tail, qt * 16 + 16) : p.n_tail;
  const int nkeys = P + tail;
  const int kvh = h / (p.n_heads / p.n_kv);
  const int row = qt * 16 + j;
  const bool valid = row < p.nq;
  const S* Q = reinterpret_cast<const S*>(p.Q);

  u32x4_t qf[NQC];
#pragma unroll
  for (int c = 0; c < NQC; ++c) {
    qf[c] = u32x4_t{0u, 0u, 0u, 0u};
    if (valid)
      qf[c] = *reinterpret_cast<const u32x4_t*>(
          Q + (size_t)(b * p.rows_per_seq + row) * p.ldq + h * HD + c * KC + g * EPL);
  }
  uint64_t mw0 = 0, mw1 = 0;
  if (!p.causal && valid) {
    const uint64_t* mr = p.mask + (size_t)slot * p.mask_seq_stride + (size_t)row * p.mask_words;
    mw0 = mr[0];
    if (p.mask_words > 1) mw1 = mr[1];
  }

  const int nblocks = (nkeys + 15) >> 4;
  const float scale2 = rsqrtf((float)HD) * 1.4426950408889634f;
  float m_i = -INFINITY, l_i = 0.f;
  f32x4_t o[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const S* kc = reinterpret_cast<const S*>(p.kcache);
  const S* vc = reinterpret_cast<const S*>(p.vcache);
  // the sequence's block-table row, staged in LDS so no K/V load waits on a table load
  __shared__ int s_bt[ATT_MAX_BLOCKS];
  const int* bt = p.block_table + (size_t)slot * p.max_blocks;
  for (int i = threadIdx.x; i < nblocks; i += ATT_THREADS) s_bt[i] = bt[i];
  __syncthreads();
  auto base_of = [&](int kb) { return ((size_t)s_bt[kb] * p.n_kv + kvh) * (size_t)(16 * HD); };

  // this wave's blocks: kb = wave + ATT_WAVES * i, i < nmine; a ring of RB blocks in
  // flight, each slot reloaded (clamped, unconditionally) right after it is consumed
  const int nmine = wave < nblocks ? (nblocks - wave + ATT_WAVES - 1) / ATT_WAVES : 0;
  auto blk = [&](int i) { return wave + ATT_WAVES * min(i, nmine - 1); };
  auto consume = [&](const KVBlock<S, HD>& cur, int kb) {
    f32x4_t s = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NQC; ++c) s = mma_frag(cur.k[c], qf[c], s, S{});
    // s[r] = score of key kb*16 + 4g + r for query row j
    float s2[4];
    float mloc = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int key = kb * 16 + 4 * g + r;
      bool vis = valid && key < nkeys;
      if (vis && key >= P) {
        const int tk = key - P;
        if (p.causal)
          vis = tk <= row;
        else
          vis = ((tk < 64 ? mw0 >> tk : mw1 >> (tk - 64)) & 1ull) != 0;
      }
      s2[r] = vis ? s[r] * scale2 : -INFINITY;
      mloc = fmaxf(mloc, s2[r]);
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_i, mloc);
    const float alpha = (m_new == -INFINITY) ? 1.f : exp2f(m_i - m_new);
    float pr[4], lsum = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      pr[r] = (s2[r] == -INFINITY) ? 0.f : exp2f(s2[r] - m_new);
      lsum += pr[r];
    }
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    l_i = l_i * alpha + lsum;
    m_i = m_new;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      o[t] *= alpha;
      o[t] = mma_pv(cur.v[t], pr, o[t], S{});
    }
  };
  if (nmine > 0) {
    KVBlock<S, HD> ring[ATT_RING];
#pragma unroll
    for (int r = 0; r < ATT_RING; ++r) ring[r].load(kc, vc, base_of(blk(r)), lane);
    const int nfull = nmine / ATT_RING;
    for (int i0 = 0; i0 < nfull * ATT_RING; i0 += ATT_RING) {  // branch-free steady state
#pragma unroll
      for (int r = 0; r < ATT_RING; ++r) {
        consume(ring[r], wave + ATT_WAVES * (i0 + r));
        ring[r].load(kc, vc, base_of(blk(i0 + r + ATT_RING)), lane);
      }
    }
#pragma unroll
    for (int r = 0; r < ATT_RING; ++r)  // tail
      if (nfull * ATT_RING + r < nmine) consume(ring[r], wave + ATT_WAVES * (nfull * ATT_RING + r));
  }
  // merge the waves' states
  if (g == 0) {
    s_m[wave][j] = m_i;
    s_l[wave][j] = l_i;
  }
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) s_o[wave][j][t * 16 + 4 * g + r] = o[t][r];
  __syncthreads();
  S* O = reinterpret_cast<S*>(p.O);
  for (int e = threadIdx.x; e < 16 * HD; e += ATT_THREADS) {
    const int r2 = e / HD, dim = e % HD;
    const int row2 = qt * 16 + r2;
    if (row2 >= p.nq) continue;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < ATT_WAVES; ++w) M = fmaxf(M, s_m[w][r2]);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < ATT_WAVES; ++w) {
      const float ms = s_m[w][r2];
      const float wt = (ms == -INFINITY) ? 0.f : exp2f(ms - M);
      num += wt * s_o[w][r2][dim];
      den += wt * s_l[w][r2];
    }
    O[(size_t)(b * p.rows_per_seq + row2) * p.ldo + h * HD + dim] = T::from_f(den > 0.f ? num / den : 0.f);
  }
}

void plan_attention(AttnParams& p, int max_keys) {
  (void)max_keys;
  p.qtiles = (p.nq + 15) / 16;
  p.splits = 1;
  p.blocks_per_split = 0;
}

size_t attention_part_floats(int, int, int, int, int) { return 0; }

template <typename S>
static hipError_t launch_attn_t(AttnParams& p, hipStream_t st, const LaunchTiming* lt) {
  const int items = p.nbatch * p.n_heads;
  dim3 grid(8 * ((items + 7) / 8) * p.qtiles), block(ATT_THREADS);
  auto go = [&](auto kern) {
    if (lt) hipExtLaunchKernelGGL(kern, grid, block, 0, st, lt->start, lt->stop, 0, p);
    else hipLaunchKernelGGL(kern, grid, block, 0, st, p);
  };
  switch (p.hd) {
    case 32: go(attn_kernel<S, 32>); break;
    case 64: go(attn_kernel<S, 64>); break;
    case 128: go(attn_kernel<S, 128>); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, AttnParams& p, int max_keys, hipStream_t st, const LaunchTiming* lt) {
  plan_attention(p, max_keys);
  if (p.nq <= 0 || p.nbatch <= 0) {  // nothing to launch: an empty timed interval
    if (lt) {
      (void)hipEventRecord(lt->start, st);
      (void)hipEventRecord(lt->stop, st);
    }
    return hipSuccess;
  }
  return dtype == 1 ? launch_attn_t<bf16_t>(p, st, lt) : launch_attn_t<float>(p, st, lt);
}

}  // namespace clover

namespace clover {

template <typename S>
__global__ void kv_write_kernel(const S* __restrict__ K, const S* __restrict__ V, int n, int slot0,
                                int seq, S* __restrict__ kc, S* __restrict__ vc,
                                const int* __restrict__ bt, int max_blocks, int n_kv, int hd) {
  const int r = blockIdx.x;
  const int slot = slot0 + r;
  for (int e = threadIdx.x; e < n_kv * hd; e += blockDim.x) {
    const int kvh = e / hd, d = e % hd;
    const size_t base = kv_block_base(bt, max_blocks, seq, slot, kvh, n_kv, hd);
    kc[base + kblk_off(slot & 15, d, St<S>::EPL)] = K[(size_t)r * n_kv * hd + e];
    vc[base + vblk_off(slot & 15, d)] = V[(size_t)r * n_kv * hd + e];
  }
}

hipError_t launch_kv_write(int dtype, const void* K, const void* V, int n, int slot0, int seq,
                           void* kcache, void* vcache, const int* block_table, int max_blocks,
                           int n_kv, int hd, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(kv_write_kernel<bf16_t>, dim3(n), dim3(256), 0, st, (const bf16_t*)K,
                       (const bf16_t*)V, n, slot0, seq, (bf16_t*)kcache, (bf16_t*)vcache,
                       block_table, max_blocks, n_kv, hd);
  else
    hipLaunchKernelGGL(kv_write_kernel<float>, dim3(n), dim3(256), 0, st, (const float*)K,
                       (const float*)V, n, slot0, seq, (float*)kcache, (float*)vcache, block_table,
                       max_blocks, n_kv, hd);
  return hipGetLastError();
}

}  // namespace clover
