// Device helpers shared by the GEMM kernels: the tile-local rotary packing of Q/K weights
// and the Q|K|V output stores (rotary, paged KV append).
#pragma once
#include "common.h"
#include "kernels.h"

namespace clover {

// source row of row r of physical tile t in a Q/K weight packed with tile-local rotary
// pairs: rows 0..7 are dims q*8.. of the first half of a head, rows 8..15 their partners
__host__ __device__ __forceinline__ int rope_row(int t, int r, int hd) {
  const int tph = hd / 16, h = t / tph, q = t % tph;
  return h * hd + (r < 8 ? q * 8 + r : hd / 2 + q * 8 + (r - 8));
}

// Rotary of one value v (first half of its pair when first) with its partner, at (cos, sin)
__device__ __forceinline__ float rope_apply(float v, float partner, float2 cs, bool first) {
  return first ? (v * cs.x - partner * cs.y) : (v * cs.x + partner * cs.y);
}

// Finishes one value of the packed Q|K|V output: physical column pc (tile-local rotary
// order), row m.  v and its rotary partner (physical column pc ^ 8) are the complete sums;
// kb = physical KV block * 16 + key slot of row m.  Q/K get the rotary factors of row m's
// position (rope_cs), Q goes to qbuf, K/V to the paged cache.
template <typename S>
__device__ __forceinline__ void qkv_store(const GemmParams& p, int m, int pc, float v, float partner, int kb) {
  using T = St<S>;
  const int hd = p.hd, half = hd >> 1, qd = p.n_heads * hd, kvd = p.n_kv * hd;
  const int pt = pc >> 4, jj = pc & 15;
  const int qt = qd / 16, kt = kvd / 16;
  const bool rot = pt < qt + kt;
  int n;  // logical output column
  if (rot) {
    const int seg0 = pt < qt ? 0 : qt;
    n = seg0 * 16 + rope_row(pt - seg0, jj, hd);
  } else {
    n = pc;
  }
  const int d = n % hd;
  if (rot) {
    const int dlo = (d < half) ? d : d - half;  // rotary frequency index
    const float2 cs = reinterpret_cast<const float2*>(p.rope_cs)[(size_t)m * half + dlo];
    v = rope_apply(v, partner, cs, jj < 8);
  }
  if (n < qd) {
    reinterpret_cast<S*>(p.qbuf)[(size_t)m * p.ldq + n] = T::from_f(v);
  } else {
    const bool isk = n < qd + kvd;
    const int kvh = (isk ? n - qd : n - qd - kvd) / hd;
    const size_t base = ((size_t)(kb >> 4) * p.n_kv + kvh) * (size_t)(16 * hd);
    const int key = kb & 15;
    if (isk)
      reinterpret_cast<S*>(p.kcache)[base + kblk_off(key, d, T::EPL)] = T::from_f(v);
    else
      reinterpret_cast<S*>(p.vcache)[base + vblk_off(key, d)] = T::from_f(v);
  }
}

// eight consecutive storage elements from float values
__device__ __forceinline__ void store8(bf16_t* dst, const float (&x)[8]) {
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = (uint32_t)f2bf(x[2 * i]) | ((uint32_t)f2bf(x[2 * i + 1]) << 16);
  *reinterpret_cast<u32x4_t*>(dst) = v;
}
__device__ __forceinline__ void store8(float* dst, const float (&x)[8]) {
  *reinterpret_cast<float4*>(dst) = make_float4(x[0], x[1], x[2], x[3]);
  *reinterpret_cast<float4*>(dst + 4) = make_float4(x[4], x[5], x[6], x[7]);
}

// Eight consecutive physical columns pc0 .. pc0 + 7 of the packed Q|K|V output (pc0 % 8 == 0:
// one half of a 16-column tile) are 8 consecutive dims d0 .. d0 + 7 of one head: the logical
// column of the first, and the rotary frequency index of the first (Q/K columns).
struct QkvCols8 {
  int n0, d0, dlo0;
  bool rot, first;  // rotary section; first half of its rotary pairs
};
__device__ __forceinline__ QkvCols8 qkv_cols8(const GemmParams& p, int pc0) {
  const int hd = p.hd, half = hd >> 1, qd = p.n_heads * hd, kvd = p.n_kv * hd;
  const int pt = pc0 >> 4, jj0 = pc0 & 15, qt = qd / 16, kt = kvd / 16;
  QkvCols8 c;
  c.rot = pt < qt + kt;
  c.first = jj0 < 8;
  if (c.rot) {
    const int seg0 = pt < qt ? 0 : qt;
    c.n0 = seg0 * 16 + rope_row(pt - seg0, jj0, hd);
  } else {
    c.n0 = pc0;
  }
  c.d0 = c.n0 % hd;
  c.dlo0 = c.d0 < half ? c.d0 : c.d0 - half;
  return c;
}
// the 8 (cos, sin) pairs of row m for those columns (V columns read a valid row they do not use)
__device__ __forceinline__ void qkv_cs8(const GemmParams& p, int m, const QkvCols8& c, float4 (&cs4)[4]) {
  const float4* cs = reinterpret_cast<const float4*>(reinterpret_cast<const float2*>(p.rope_cs) +
                                                     (size_t)m * (p.hd >> 1) + c.dlo0);
#pragma unroll
  for (int k = 0; k < 4; ++k) cs4[k] = cs[k];
}
// Finishes the 8 values v of row m (w: the partner half's values), with the arithmetic of
// qkv_store: rotary for Q/K, then Q to qbuf and K to the cache as one 16-byte store each (8
// consecutive dims; the cache's K fragment order keeps 8 dims of a key together), V as 8
// stores (the cache's key-minor layout).  kb = physical KV block * 16 + key slot of row m.
template <typename S>
__device__ __forceinline__ void qkv_store8(const GemmParams& p, int m, const QkvCols8& c, float (&v)[8],
                                           const float (&w)[8], const float4 (&cs4)[4], int kb) {
  using T = St<S>;
  const int hd = p.hd, qd = p.n_heads * hd, kvd = p.n_kv * hd;
  if (c.rot) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float cx = (e & 1) ? cs4[e >> 1].z : cs4[e >> 1].x, sy = (e & 1) ? cs4[e >> 1].w : cs4[e >> 1].y;
      v[e] = rope_apply(v[e], w[e], make_float2(cx, sy), c.first);
    }
  }
  if (c.n0 < qd) {
    store8(reinterpret_cast<S*>(p.qbuf) + (size_t)m * p.ldq + c.n0, v);
    return;
  }
  const int key = kb & 15;
  const bool isk = c.n0 < qd + kvd;
  const int kvh = (isk ? c.n0 - qd : c.n0 - qd - kvd) / hd;
  const size_t base = ((size_t)(kb >> 4) * p.n_kv + kvh) * (size_t)(16 * hd);
  if (isk) {
    S* kc = reinterpret_cast<S*>(p.kcache) + base;
    if constexpr (T::EPL == 8) {
      store8(kc + kblk_off(key, c.d0, 8), v);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) kc[kblk_off(key, c.d0 + e, T::EPL)] = T::from_f(v[e]);
    }
  } else {
    S* vc = reinterpret_cast<S*>(p.vcache) + base;
#pragma unroll
    for (int e = 0; e < 8; ++e) vc[vblk_off(key, c.d0 + e)] = T::from_f(v[e]);
  }
}

// Gumbel-max score of one logit: the logit times the float32 reciprocal of the temperature,
// plus standard Gumbel noise from the counter (column n, row, step, slot) under the key
// (seed, domain).  The product and the sum round separately (no fused multiply-add), as
// float32 arithmetic written out does.
__device__ __forceinline__ float gumbel_score(float v, float inv_temp, uint32_t n, uint32_t row, uint32_t step,
                                              uint32_t slot, uint32_t seed, uint32_t domain) {
#pragma clang fp contract(off)
  const uint32_t x = philox4x32_10_w0(n, row, step, slot, seed, domain);
  const float scaled = v * inv_temp;
  return scaled + gumbel_from_bits(x);
}

// The same score behind a call, for epilogues with many outputs per lane: inlining the
// generator at every output makes the epilogue too long to unroll, and the accumulators
// would then be indexed at run time (private memory).
__device__ __noinline__ float gumbel_score_call(float v, float inv_temp, uint32_t n, uint32_t row, uint32_t step,
                                                uint32_t slot, uint32_t seed, uint32_t domain) {
  return gumbel_score(v, inv_temp, n, row, step, slot, seed, domain);
}

// The value the LM-head argmax keys rank for output (row m, column n): the logit itself, or
// with sampling on the logit over the temperature plus the row's Gumbel noise for n.
__device__ __forceinline__ float amax_value(const GemmParams& p, float v, int m, int n) {
  if (p.inv_temp == 0.f) return v;
  const int slot = p.samp_slot[m];
  return gumbel_score(v, p.inv_temp, (uint32_t)n, (uint32_t)(m % p.samp_rows), (uint32_t)p.samp_step[slot],
                      (uint32_t)slot, p.samp_seed, p.samp_domain);
}

}  // namespace clover
