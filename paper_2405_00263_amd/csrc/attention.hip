// Tree-masked attention over the paged KV cache (tree attention, Sec. 2.2 of the
// paper: the causal mask of the verify forward is the token tree's ancestor matrix).
//
// Each query row attends to every committed key (slots 0..P-1) and to the tail keys
// P..P+n_tail-1 its mask row admits: the tree's ancestor-or-self bits during verify,
// or the causal rule during chunked prefill.
//
// Work split.  One workgroup takes one (sequence, KV head), up to four 16-row query
// tiles of the query heads sharing that KV head, and one contiguous range of the keys.
// Its K/V blocks are staged once through LDS and shared by the tiles, so each CU reads
// every key it needs exactly once; the key range is split over enough workgroups
// (attention "splits") to give every CU of the chip one workgroup.  Splits of one
// (sequence, KV head) run on the same XCD and leave fp32 partial states (unnormalised
// output, running max, running sum) that a small merge kernel combines in split order;
// with one split the output is written directly.
//
// Inside a workgroup of four query tiles, waves w and w + 4 take one query tile and the
// even / odd key blocks of each chunk, merging their states through LDS at the end.  When an
// item has eight or more query tiles (trees above 64 tokens, grouped KV heads, prefill
// chunks) a workgroup takes eight tiles, one per wave over every key block, so each K/V
// chunk staged in LDS feeds twice as many queries and the item's keys are read by half as
// many workgroups.  The score
// product is computed transposed (S^T = K Q^T) so the matrix-core accumulator already
// holds, per lane, four consecutive keys of one query row: exactly the operand layout
// the P*V product needs.  Softmax is online in the log2 domain.  The next chunk's K/V
// loads are in flight while the current chunk is computed from LDS.
#include "common.h"
#include "kernels.h"

#include <hip/hip_ext.h>

#include <algorithm>

namespace clover {

static constexpr int AT_WAVES = 8;               // 4 query tiles x 2 key halves, or 8 x 1
static constexpr int AT_THREADS = AT_WAVES * 64;
static constexpr int AT_MAX_BLOCKS = 4096;       // 65536 keys
static constexpr int AT_MAX_SPLITS = 16;
static constexpr int AT_TARGET_WGS = 256;        // one workgroup per CU
static constexpr int AT_CHUNK_BYTES = 128 * 1024;  // K + V bytes of one LDS chunk

// probabilities of one lane's 4 keys as the bf16 B operand of the P*V product
__device__ __forceinline__ u32x2_t pack_p(const float p[4], bf16_t) {
  typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
  const bf16x4_t v = {(__bf16)p[0], (__bf16)p[1], (__bf16)p[2], (__bf16)p[3]};
  return __builtin_bit_cast(u32x2_t, v);
}
__device__ __forceinline__ u32x2_t pack_p(const float*, float) { return u32x2_t{0u, 0u}; }

__device__ __forceinline__ f32x4_t mma_pv(u32x2_t v, u32x2_t pb, const float*, f32x4_t c, bf16_t) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, v),
                                                   __builtin_bit_cast(s16x4_t, pb), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mma_pv(u32x4_t v, u32x2_t, const float p[4], f32x4_t c, float) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v[0]), p[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v[1]), p[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v[2]), p[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(v[3]), p[3], c, 0, 0, 0);
  return c;
}

// P*V over two key blocks in one 16x16x32 product (bf16): the sum over keys may take them in
// any order, so the k index of lane group g pairs its 4 keys of the first block (elements 0..3)
// with its 4 keys of the second (4..7) in both operands; each lane already holds exactly those
// probabilities and value columns.  Same output layout as the single-block product.
__device__ __forceinline__ f32x4_t mma_pv2(u32x2_t v0, u32x2_t v1, u32x2_t p0, u32x2_t p1, const float*, const float*,
                                           f32x4_t c, bf16_t) {
  const u32x4_t a = {v0[0], v0[1], v1[0], v1[1]}, b = {p0[0], p0[1], p1[0], p1[1]};
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mma_pv2(u32x4_t v0, u32x4_t v1, u32x2_t p0, u32x2_t p1, const float* q0, const float* q1,
                                           f32x4_t c, float) {
  return mma_pv(v1, p1, q1, mma_pv(v0, p0, q0, c, float{}), float{});
}

// Reductions over the four lanes that hold one query row's keys (lanes j, j+16, j+32,
// j+48): VALU lane swaps (upper/lower 32 lanes, then odd/even 16-lane rows) instead of
// LDS-routed shuffles.  Every lane of the row ends with the same value, summed in the
// same order.
__device__ __forceinline__ float row4_max(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float row4_sum(float x) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

template <typename S> struct VFrag;
template <> struct VFrag<bf16_t> { typedef u32x2_t type; };
template <> struct VFrag<float> { typedef u32x4_t type; };

template <typename S, int HD>
struct AttnShape {
  static constexpr int BLK_BYTES = 16 * HD * (int)sizeof(S);                // K (or V) of a block
  static constexpr int CB = std::min(16, AT_CHUNK_BYTES / (2 * BLK_BYTES));  // blocks per chunk
  static constexpr int CH_VEC = 2 * CB * BLK_BYTES / 16;                    // 16-byte vectors
  static constexpr int LVEC = CH_VEC / AT_THREADS;                          // per thread
  static_assert(CH_VEC % AT_THREADS == 0, "chunk splits evenly over the threads");
  static constexpr size_t LDS = (size_t)CH_VEC * 16;
};

// record of one (item, split, query tile, row): o[HD] then m, l
__device__ __forceinline__ size_t part_rec(const AttnParams& p, int item, int split, int qi, int j, int hd) {
  return ((((size_t)item * p.splits + split) * p.qt_item + qi) * 16 + j) * (size_t)(hd + 2);
}

// QT: query tiles per workgroup (4: two waves per tile over the even / odd key blocks; 8:
// one wave per tile over all of them)
template <typename S, int HD, int QT>
__global__ __launch_bounds__(AT_THREADS) void attn_kernel(const AttnParams p) {
  constexpr int HALVES = AT_WAVES / QT;  // waves per query tile, each over every HALVES-th block
  using T = St<S>;
  using SH = AttnShape<S, HD>;
  constexpr int EPL = T::EPL, KC = 4 * EPL, NQC = HD / KC, NT = HD / 16;
  constexpr int CB = SH::CB, LVEC = SH::LVEC, BVEC = SH::BLK_BYTES / 16;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  u32x4_t* lds = reinterpret_cast<u32x4_t*>(smem);  // [K blocks 0..CB-1][V blocks 0..CB-1]
  __shared__ int s_bt[AT_MAX_BLOCKS];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, j = lane & 15;
  const int half = wave / QT;  // key-block parity this wave takes (HALVES = 2)
  // workgroup -> (item, query group, split); all splits and query groups of an item on
  // one XCD (workgroup ids are dealt to the 8 XCDs round-robin)
  const int per_item = p.qgroups * p.splits;
  const int id = blockIdx.x, xcd = id & 7, slotx = id >> 3;
  const int item = (slotx / per_item) * 8 + xcd, rem = slotx % per_item;
  const int qg = rem / p.splits, split = rem % p.splits;
  if (item >= p.nbatch * p.n_kv) return;
  const int b = item / p.n_kv, kvh = item % p.n_kv;
  const int G = p.n_heads / p.n_kv;
  const int slot = p.seq_ids[b];
  const int P = p.prefix_dev ? p.prefix_dev[slot] : p.prefix_host;

  // this wave's query tile
  const int qi = qg * QT + (wave % QT);
  const bool has_q = qi < p.qt_item;
  const int h = kvh * G + (has_q ? qi / p.qph : 0), qt = has_q ? qi % p.qph : 0;
  const int row = qt * 16 + j;
  const bool valid = has_q && row < p.nq;
  // keys the workgroup needs: the causal tail stops at its last query tile's rows
  int tail = p.n_tail;
  if (p.causal) {
    int qmax = 0;
    for (int w = 0; w < QT; ++w) {
      const int q2 = qg * QT + w;
      if (q2 < p.qt_item) qmax = max(qmax, q2 % p.qph);
    }
    tail = min(p.n_tail, qmax * 16 + 16);
  }
  const int nkeys = P + tail;
  const int nblocks = (nkeys + 15) >> 4;
  const int bps = (nblocks + p.splits - 1) / p.splits;
  const int kb0 = min(nblocks, split * bps), nb = min(nblocks, kb0 + bps) - kb0;

  // Q and the mask rows are loaded before the block table, so the three loads share one
  // memory round trip (the table's store to LDS waits for its load)
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
  const int* bt = p.block_table + (size_t)slot * p.max_blocks;
  for (int i = threadIdx.x; i < nb; i += AT_THREADS) s_bt[i] = bt[kb0 + i];
  __syncthreads();  // s_bt

  const S* kc = reinterpret_cast<const S*>(p.kcache);
  const S* vc = reinterpret_cast<const S*>(p.vcache);
  const int nch = (nb + CB - 1) / CB;
  // chunk loader: vector v of the chunk is K (v < CB*BVEC) or V of block v / BVEC; blocks
  // past the range are clamped to its last block (unconditional loads, never consumed)
  u32x4_t stg[LVEC];
  auto load_chunk = [&](int ch) {
#pragma unroll
    for (int i = 0; i < LVEC; ++i) {
      const int v = threadIdx.x + i * AT_THREADS;
      const int isv = v >= CB * BVEC;
      const int vv = v - isv * CB * BVEC;
      const int kbl = min(ch * CB + vv / BVEC, nb - 1);
      const size_t base = ((size_t)s_bt[kbl] * p.n_kv + kvh) * (size_t)(16 * HD);
      const S* src = (isv ? vc : kc) + base + (size_t)(vv % BVEC) * (16 / sizeof(S));
      stg[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(src));
    }
  };
  auto store_chunk = [&]() {
#pragma unroll
    for (int i = 0; i < LVEC; ++i) lds[threadIdx.x + i * AT_THREADS] = stg[i];
  };

  const float scale2 = rsqrtf((float)HD) * 1.4426950408889634f;
  float m_i = -INFINITY, l_i = 0.f;
  f32x4_t o[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // One online-softmax update over up to NG of this wave's blocks of the chunk (LDS
  // blocks cb0, cb0 + HALVES, ...; key blocks kb0g, kb0g + HALVES, ...): the cross-lane max and
  // sum reductions and the rescale of the output are paid once per NG blocks.  The
  // running max m_i is kept in raw score units; the scale folds into one multiply-add
  // per exponent.  Groups wholly inside the committed prefix skip the mask logic.
  constexpr int NG = 4;
  static_assert(CB - 1 + HALVES * (NG - 1) < 2 * CB, "score reads of a group stay inside the chunk buffer");
  using VT = typename VFrag<S>::type;
  // tail rule as data, so the score loop has no branch on the mode: causal rows see tail
  // keys up to their own index, tree rows the keys whose mask bit is set
  const bool causal_mode = p.causal != 0;
  const int tail_lim = causal_mode ? row : 0x7fffffff;
  auto consume = [&](int cb0, int kb0g, int nblk) {
    // All NG score products are computed (four independent matrix-core chains, no branch
    // between them); blocks past nblk read LDS inside the chunk buffer and are masked below.
    f32x4_t s[NG];
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const u32x4_t* kblk = lds + (cb0 + HALVES * i) * BVEC;
      f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NQC; ++c) acc = mma_frag(kblk[c * 64 + lane], qf[c], acc, S{});
      s[i] = acc;
    }
    // s[i][r] = score of key (kb0g + HALVES*i)*16 + 4g + r for query row j
    const bool plain = nblk == NG && (kb0g + HALVES * (NG - 1)) * 16 + 15 < P;  // all keys committed
    if (!plain) {
#pragma unroll
      for (int i = 0; i < NG; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = (kb0g + HALVES * i) * 16 + 4 * g + r;
          const int tk = key - P;
          const uint64_t word = tk < 64 ? mw0 : mw1;
          const bool tree_ok = causal_mode | (((word >> (tk & 63)) & 1ull) != 0);
          const bool vis = valid & (i < nblk) & (key < nkeys) & ((tk < 0) | (tree_ok & (tk <= tail_lim)));
          s[i][r] = vis ? s[i][r] : -INFINITY;
        }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int i = 0; i < NG; ++i) mloc = fmaxf(mloc, fmaxf(fmaxf(s[i][0], s[i][1]), fmaxf(s[i][2], s[i][3])));
    mloc = row4_max(mloc);
    const float m_new = fmaxf(m_i, mloc);
    // every exponent below is <= 0; exp2(-inf) = 0 removes masked keys
    const float nm = (m_new == -INFINITY) ? 0.f : -m_new * scale2;
    const float alpha = __builtin_amdgcn_exp2f(fmaf(m_i, scale2, nm));
    float lsum = 0.f;
    u32x2_t pb[NG];
    float pr[NG][4];
#pragma unroll
    for (int i = 0; i < NG; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pr[i][r] = __builtin_amdgcn_exp2f(fmaf(s[i][r], scale2, nm));
        lsum += pr[i][r];
      }
      pb[i] = pack_p(pr[i], S{});
    }
    lsum = row4_sum(lsum);
    l_i = l_i * alpha + lsum;
    m_i = m_new;
    if (!__all(alpha == 1.f)) {
#pragma unroll
      for (int t = 0; t < NT; ++t) o[t] *= alpha;
    }
#pragma unroll
    for (int i = 0; i < NG; i += 2) {
      const VT* v0 = reinterpret_cast<const VT*>(lds + (CB + cb0 + HALVES * i) * BVEC);
      if (i + 1 < nblk) {  // two blocks per product
        const VT* v1 = reinterpret_cast<const VT*>(lds + (CB + cb0 + HALVES * (i + 1)) * BVEC);
#pragma unroll
        for (int t = 0; t < NT; ++t) o[t] = mma_pv2(v0[t * 64 + lane], v1[t * 64 + lane], pb[i], pb[i + 1], pr[i], pr[i + 1], o[t], S{});
      } else if (i < nblk) {
#pragma unroll
        for (int t = 0; t < NT; ++t) o[t] = mma_pv(v0[t * 64 + lane], pb[i], pr[i], o[t], S{});
      }
    }
  };

  if (nch > 0) {
    load_chunk(0);
    store_chunk();
    __syncthreads();
    for (int ch = 0; ch < nch; ++ch) {
      const bool more = ch + 1 < nch;
      if (more) load_chunk(ch + 1);  // in flight while this chunk is computed
      if (has_q) {
        const int nbc = min(CB, nb - ch * CB);
        for (int cb0 = half; cb0 < nbc; cb0 += HALVES * NG)
          consume(cb0, kb0 + ch * CB + cb0, min(NG, (nbc - cb0 + HALVES - 1) / HALVES));
      }
      __syncthreads();
      if (more) {
        store_chunk();
        __syncthreads();
      }
    }
  }

  // from here on the running max is in log2-scaled units, as the merges expect
  m_i = (m_i == -INFINITY) ? -INFINITY : m_i * scale2;
  // merge the two key halves of each query tile through LDS (the chunk buffer is free)
  float* mo = reinterpret_cast<float*>(smem);  // [QT][16][HD + 2]
  float* rec = mo + (size_t)((wave % QT) * 16 + j) * (HD + 2);
  if (HALVES == 2 && half == 1) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) rec[t * 16 + 4 * g + r] = o[t][r];
    if (g == 0) {
      rec[HD] = m_i;
      rec[HD + 1] = l_i;
    }
  }
  if (HALVES == 2) __syncthreads();
  if (half == 1 || !has_q) return;
  if (HALVES == 2) {
    const float m1 = rec[HD], l1 = rec[HD + 1];
    const float M = fmaxf(m_i, m1);
    const float a0 = (m_i == -INFINITY) ? 0.f : exp2f(m_i - M);
    const float a1 = (m1 == -INFINITY) ? 0.f : exp2f(m1 - M);
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) o[t][r] = a0 * o[t][r] + a1 * rec[t * 16 + 4 * g + r];
    l_i = a0 * l_i + a1 * l1;
    m_i = M;
  }
  if (p.splits == 1) {
    if (!valid) return;
    const float inv = l_i > 0.f ? 1.f / l_i : 0.f;
    S* O = reinterpret_cast<S*>(p.O) + (size_t)(b * p.rows_per_seq + row) * p.ldo + h * HD;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) O[t * 16 + 4 * g + r] = T::from_f(o[t][r] * inv);
    return;
  }
  float* pr = p.part + part_rec(p, item, split, qi, j, HD);
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) pr[t * 16 + 4 * g + r] = o[t][r];
  if (g == 0) {
    pr[HD] = m_i;
    pr[HD + 1] = l_i;
  }
}

// Combine the splits of one (item, query tile) in split order; same XCD as its splits.
// One single-wave workgroup per 4 rows of a query tile: the records are spread over many
// compute units (a compute unit moves only tens of GB/s, so bytes per unit set the time).
// The live splits' records are loaded up front (one memory latency, not one per split).
static constexpr int MERGE_ROWS = 4;
template <typename S, int HD>
__global__ __launch_bounds__(64) void attn_merge_kernel(const AttnParams p) {
  using T = St<S>;
  constexpr int DPT = HD / 16;  // dims per thread
  constexpr int RG = 16 / MERGE_ROWS;  // row groups per query tile
  const int id = blockIdx.x, xcd = id & 7, slotx = id >> 3;
  const int item = (slotx / (p.qt_item * RG)) * 8 + xcd, rem = slotx % (p.qt_item * RG);
  const int qi = rem / RG, rg = rem % RG;
  if (item >= p.nbatch * p.n_kv) return;
  const int b = item / p.n_kv, kvh = item % p.n_kv, G = p.n_heads / p.n_kv;
  const int h = kvh * G + qi / p.qph, qt = qi % p.qph;
  const int j = rg * MERGE_ROWS + (threadIdx.x >> 4), d0 = (threadIdx.x & 15) * DPT;
  const int row = qt * 16 + j;
  if (row >= p.nq) return;
  float ms[AT_MAX_SPLITS], ls[AT_MAX_SPLITS], ov[AT_MAX_SPLITS][DPT];
#pragma unroll
  for (int s = 0; s < AT_MAX_SPLITS; ++s) {
    ms[s] = -INFINITY;
    ls[s] = 0.f;
#pragma unroll
    for (int e = 0; e < DPT; ++e) ov[s][e] = 0.f;
    if (s < p.splits) {
      const float* r = p.part + part_rec(p, item, s, qi, j, HD);
      ms[s] = r[HD];
      ls[s] = r[HD + 1];
#pragma unroll
      for (int e = 0; e < DPT; ++e) ov[s][e] = r[d0 + e];
    }
  }
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < AT_MAX_SPLITS; ++s)
    if (s < p.splits) M = fmaxf(M, ms[s]);
  float acc[DPT], den = 0.f;
#pragma unroll
  for (int e = 0; e < DPT; ++e) acc[e] = 0.f;
#pragma unroll
  for (int s = 0; s < AT_MAX_SPLITS; ++s) {
    const float wt = (s >= p.splits || ms[s] == -INFINITY) ? 0.f : exp2f(ms[s] - M);
    den += wt * ls[s];
#pragma unroll
    for (int e = 0; e < DPT; ++e) acc[e] += wt * ov[s][e];
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
  S* O = reinterpret_cast<S*>(p.O) + (size_t)(b * p.rows_per_seq + row) * p.ldo + h * HD + d0;
#pragma unroll
  for (int e = 0; e < DPT; ++e) O[e] = T::from_f(acc[e] * inv);
}

void plan_attention(AttnParams& p) {
  const int G = std::max(1, p.n_heads / std::max(1, p.n_kv));
  p.qph = (p.nq + 15) / 16;
  p.qt_item = G * p.qph;
  p.qtile = p.qt_item >= 8 ? 8 : 4;  // eight tiles a workgroup whenever an item has that many
  p.qgroups = (p.qt_item + p.qtile - 1) / p.qtile;
  const int base = std::max(1, p.nbatch * p.n_kv * p.qgroups);
  p.splits = std::max(1, std::min(AT_MAX_SPLITS, AT_TARGET_WGS / base));
}

size_t attention_part_floats(const AttnParams& p0) {
  AttnParams p = p0;
  plan_attention(p);
  if (p.splits == 1) return 0;
  return (size_t)p.nbatch * p.n_kv * p.splits * p.qt_item * 16 * (size_t)(p.hd + 2);
}

template <typename S, int HD>
static hipError_t launch_attn_hd(AttnParams& p, hipStream_t st, const LaunchTiming* lt) {
  const int items = p.nbatch * p.n_kv;
  const int per_xcd = (items + 7) / 8;
  dim3 grid(8 * per_xcd * p.qgroups * p.splits), block(AT_THREADS);
  const size_t lds = AttnShape<S, HD>::LDS;
  static bool lds_attr = false;  // dynamic LDS above 64 KB is opted into once per kernel
  if (!lds_attr) {
    for (const void* k : {reinterpret_cast<const void*>(&attn_kernel<S, HD, 4>),
                          reinterpret_cast<const void*>(&attn_kernel<S, HD, 8>)}) {
      const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    lds_attr = true;
  }
  static_assert((size_t)4 * 16 * (HD + 2) * 4 <= AttnShape<S, HD>::LDS, "merge records fit the chunk buffer");
  // the merge kernel, if any, closes the timed interval
  const bool merge = p.splits > 1;
  auto go = [&](auto kern) {
    if (lt) hipExtLaunchKernelGGL(kern, grid, block, (uint32_t)lds, st, lt->start, merge ? nullptr : lt->stop, 0, p);
    else hipLaunchKernelGGL(kern, grid, block, lds, st, p);
  };
  if (p.qtile == 8) go(attn_kernel<S, HD, 8>);
  else go(attn_kernel<S, HD, 4>);
  if (merge) {
    dim3 mgrid(8 * per_xcd * p.qt_item * (16 / MERGE_ROWS));
    if (lt) hipExtLaunchKernelGGL((attn_merge_kernel<S, HD>), mgrid, dim3(64), 0, st, nullptr, lt->stop, 0, p);
    else hipLaunchKernelGGL((attn_merge_kernel<S, HD>), mgrid, dim3(64), 0, st, p);
  }
  return hipGetLastError();
}

template <typename S>
static hipError_t launch_attn_t(AttnParams& p, hipStream_t st, const LaunchTiming* lt) {
  switch (p.hd) {
    case 32: return launch_attn_hd<S, 32>(p, st, lt);
    case 64: return launch_attn_hd<S, 64>(p, st, lt);
    case 128: return launch_attn_hd<S, 128>(p, st, lt);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attention(int dtype, AttnParams& p, int max_keys, hipStream_t st, const LaunchTiming* lt) {
  plan_attention(p);
  if (p.nq <= 0 || p.nbatch <= 0) {  // nothing to launch: an empty timed interval
    if (lt) {
      (void)hipEventRecord(lt->start, st);
      (void)hipEventRecord(lt->stop, st);
    }
    return hipSuccess;
  }
  if (max_keys > AT_MAX_BLOCKS * 16 || p.n_kv <= 0 || p.n_heads % p.n_kv) return hipErrorInvalidValue;
  if (p.splits > 1 && (!p.part || p.part_cap < attention_part_floats(p))) return hipErrorInvalidValue;
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
