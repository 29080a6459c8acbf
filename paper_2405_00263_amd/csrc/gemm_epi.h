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
    v = (jj < 8) ? (v * cs.x - partner * cs.y) : (v * cs.x + partner * cs.y);
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
