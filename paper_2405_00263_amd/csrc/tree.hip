// Token tree construction, greedy acceptance and KV compaction (device side).
//
// Tree: the drafted candidates (creation order, root first) are truncated to T verify
// tokens by cumulative log-probability, ties broken by depth then creation index; the
// kept nodes keep creation (breadth-first) order and the mask row of a node is its
// parent's row plus itself, i.e. the ancestor-or-self matrix of tree attention
// (Sec. 2.2).  Acceptance (Sec. 2.1) walks from the root to the child whose token
// equals the target's greedy token at the parent; the accepted path's KV entries are
// then moved from their tree slots to consecutive committed positions.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace clover {

static constexpr int TREE_THREADS = 256;
static constexpr int MAX_CAND = 1024;
static constexpr int MAX_TREE = 128;

__device__ __forceinline__ bool cand_before(float la, int da, int ia, float lb, int db, int ib) {
  return la > lb || (la == lb && (da < db || (da == db && ia < ib)));
}

__global__ __launch_bounds__(TREE_THREADS) void tree_build_kernel(const TreeParams p) {
  __shared__ float slp[MAX_CAND];
  __shared__ int sdep[MAX_CAND];
  __shared__ int sremap[MAX_CAND];
  __shared__ unsigned char skeep[MAX_CAND];
  const int b = blockIdx.x, slot = p.seq_ids ? p.seq_ids[b] : b;
  const int n = p.n_cand, T = p.T, W = p.mask_words;
  const size_t cb = (size_t)slot * p.cand_stride;
  const int L = p.seq_len ? p.seq_len[slot] : p.seq_len_host;
  for (int i = threadIdx.x; i < n; i += TREE_THREADS) {
    slp[i] = p.cand_lp[cb + i];
    sdep[i] = p.cand_depth[cb + i];
  }
  __syncthreads();
  // rank of every non-root candidate under (lp desc, depth asc, index asc)
  for (int i = 1 + threadIdx.x; i < n; i += TREE_THREADS) {
    int rank = 0;
    const float li = slp[i];
    const int di = sdep[i];
    for (int j = 1; j < n; ++j) rank += cand_before(slp[j], sdep[j], j, li, di, i) ? 1 : 0;
    skeep[i] = rank < T - 1;
  }
  if (threadIdx.x == 0) skeep[0] = 1;
  __syncthreads();
  // new index = number of kept candidates before i (root included)
  for (int i = threadIdx.x; i < n; i += TREE_THREADS) {
    int idx = -1;
    if (skeep[i]) {
      idx = 0;
      for (int j = 0; j < i; ++j) idx += skeep[j];
    }
    sremap[i] = idx;
  }
  __syncthreads();
  __shared__ int tpar[MAX_TREE], tdep[MAX_TREE];
  __shared__ uint64_t tmask[MAX_TREE * 2];
  const size_t tb = (size_t)slot * T;
  for (int i = threadIdx.x; i < n; i += TREE_THREADS) {
    const int t = sremap[i];
    if (t < 0) continue;
    const int par = (i == 0) ? -1 : sremap[p.cand_parent[cb + i]];
    const int tok = p.cand_token[cb + i];
    const int dep = sdep[i];
    tpar[t] = par;
    tdep[t] = dep;
    p.tree_token[tb + t] = tok;
    p.tree_parent[tb + t] = par;
    p.tree_depth[tb + t] = dep;
    p.tree_pos[tb + t] = L + dep;
    if (p.row_tok) {
      const int m = b * T + t;
      p.row_tok[m] = tok;
      p.row_pos[m] = L + dep;
      p.row_slot[m] = L + t;
      p.row_seq[m] = slot;
    }
  }
  __syncthreads();
  // ancestor masks, one depth level at a time (parents precede children)
  int maxd = 0;
  for (int t = 0; t < T; ++t) maxd = max(maxd, tdep[t]);
  for (int lev = 0; lev <= maxd; ++lev) {
    for (int t = threadIdx.x; t < T; t += TREE_THREADS) {
      if (tdep[t] != lev) continue;
      const int par = tpar[t];
      for (int w = 0; w < W; ++w) {
        uint64_t v = par >= 0 ? tmask[par * W + w] : 0ull;
        if ((t >> 6) == w) v |= 1ull << (t & 63);
        tmask[t * W + w] = v;
      }
    }
    __syncthreads();
  }
  uint64_t* mask = p.tree_mask + (size_t)slot * T * W;
  for (int i = threadIdx.x; i < T * W; i += TREE_THREADS) mask[i] = tmask[i];
}

hipError_t launch_tree_build(TreeParams& p, hipStream_t st) {
  if (p.nbatch <= 0) return hipSuccess;
  if (p.n_cand > MAX_CAND || p.n_cand < p.T || p.T > MAX_TREE || p.mask_words > 2)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(tree_build_kernel, dim3(p.nbatch), dim3(TREE_THREADS), 0, st, p);
  return hipGetLastError();
}

// ---- acceptance ---------------------------------------------------------------------------
__global__ __launch_bounds__(TREE_THREADS) void accept_kernel(const AcceptParams p) {
  __shared__ int s_found;
  __shared__ int s_acc[16];
  __shared__ int s_len;
  const int b = blockIdx.x, slot = p.seq_ids ? p.seq_ids[b] : b, T = p.T;
  const int* tok = p.tree_token + (size_t)slot * T;
  const int* par = p.tree_parent + (size_t)slot * T;
  const int* tgt = p.target + (size_t)b * T;
  if (threadIdx.x == 0) { s_acc[0] = 0; s_len = 1; }
  __syncthreads();
  int cur = 0;
  for (int depth = 1; depth <= p.H; ++depth) {
    if (threadIdx.x == 0) s_found = 0x7fffffff;
    __syncthreads();
    const int want = tgt[cur];
    for (int c = threadIdx.x; c < T; c += TREE_THREADS)
      if (par[c] == cur && tok[c] == want) atomicMin(&s_found, c);
    __syncthreads();
    const int f = s_found;
    if (f == 0x7fffffff) break;
    if (threadIdx.x == 0) { s_acc[s_len] = f; s_len = s_len + 1; }
    cur = f;
    __syncthreads();
  }
  __syncthreads();
  const int A = s_len;
  const int bonus = tgt[cur];
  if (threadIdx.x <= p.H) {
    const int i = threadIdx.x;
    p.acc[(size_t)slot * (p.H + 1) + i] = i < A ? s_acc[i] : -1;
    int out = -1;
    if (i < A - 1) out = tok[s_acc[i + 1]];
    else if (i == A - 1) out = bonus;
    if (p.out_tokens) p.out_tokens[(size_t)b * (p.H + 1) + i] = out;
  }
  if (threadIdx.x == 0) {
    p.acc_len[slot] = A;
    if (p.t0) p.t0[slot] = bonus;
    if (p.step_ctr) p.step_ctr[slot] += 1;  // the sampled targets' draws move on
  }
  if (!p.h0) return;
  const float* src = p.ab_out + (size_t)(b * T + cur) * p.d;
  for (int k = threadIdx.x; k < p.d; k += TREE_THREADS) p.h0[(size_t)slot * p.d + k] = src[k];
}

hipError_t launch_accept(AcceptParams& p, hipStream_t st) {
  if (p.nbatch <= 0) return hipSuccess;
  if (p.H + 1 > 16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(accept_kernel, dim3(p.nbatch), dim3(TREE_THREADS), 0, st, p);
  return hipGetLastError();
}

// ---- KV compaction: slot L + acc[j] -> slot L + j for every layer ----------------------------
// Each thread owns fixed (head, dim) elements and loads all sources before storing, so a
// destination that is also a later source (acc[j''] == j) is read before it is written.
template <typename S>
__global__ __launch_bounds__(256) void compact_kernel(const CompactParams p) {
  constexpr int MAXA = 9;
  const int b = blockIdx.x, layer = blockIdx.y, slot = p.seq_ids ? p.seq_ids[b] : 0;
  const int A = p.acc_len ? p.acc_len[slot] : p.A_host, L = p.seq_len ? p.seq_len[slot] : p.L_host;
  const int* acc = p.acc + (size_t)slot * (p.H + 1);
  S* kp = p.kpools ? reinterpret_cast<S*>(p.kpools[layer])
                   : reinterpret_cast<S*>(p.kbase) + (size_t)layer * p.layer_elems;
  S* vp = p.vpools ? reinterpret_cast<S*>(p.vpools[layer])
                   : reinterpret_cast<S*>(p.vbase) + (size_t)layer * p.layer_elems;
  const int hd = p.hd, per = p.n_kv * hd;
  for (int e = threadIdx.x; e < per; e += 256) {
    const int kvh = e / hd, d = e % hd;
    S kv[MAXA], vv[MAXA];
#pragma unroll
    for (int j = 0; j < MAXA; ++j) {
      if (j < A && acc[j] != j) {
        const int s = L + acc[j];
        const size_t base = kv_block_base(p.block_table, p.max_blocks, slot, s, kvh, p.n_kv, hd);
        kv[j] = kp[base + kblk_off(s & 15, d, St<S>::EPL)];
        vv[j] = vp[base + vblk_off(s & 15, d)];
      }
    }
#pragma unroll
    for (int j = 0; j < MAXA; ++j) {
      if (j < A && acc[j] != j) {
        const int s = L + j;
        const size_t base = kv_block_base(p.block_table, p.max_blocks, slot, s, kvh, p.n_kv, hd);
        kp[base + kblk_off(s & 15, d, St<S>::EPL)] = kv[j];
        vp[base + vblk_off(s & 15, d)] = vv[j];
      }
    }
  }
}

hipError_t launch_compact(int dtype, CompactParams& p, hipStream_t st) {
  if (p.nbatch <= 0) return hipSuccess;
  if (p.H + 1 > 9) return hipErrorInvalidValue;
  dim3 grid(p.nbatch, p.nlayers);
  if (dtype == 1)
    hipLaunchKernelGGL(compact_kernel<bf16_t>, grid, dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(compact_kernel<float>, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace clover

namespace clover {

__global__ void set_root_kernel(const int* seq_ids, const int* t0, int* ct, int* cp, int* cd,
                                float* cl, int stride) {
  const int slot = seq_ids[blockIdx.x];
  const size_t cb = (size_t)slot * stride;
  ct[cb] = t0[slot];
  cp[cb] = -1;
  cd[cb] = 0;
  cl[cb] = 0.f;
}

hipError_t launch_set_root(const int* seq_ids, int nbatch, const int* t0, int* cand_token,
                           int* cand_parent, int* cand_depth, float* cand_lp, int cand_stride,
                           hipStream_t st) {
  if (nbatch <= 0) return hipSuccess;
  hipLaunchKernelGGL(set_root_kernel, dim3(nbatch), dim3(1), 0, st, seq_ids, t0, cand_token,
                     cand_parent, cand_depth, cand_lp, cand_stride);
  return hipGetLastError();
}

// Medusa candidates (Cartesian product, Sec. 2.3): the children of every depth-(j-1) node
// are head j's top-k_j tokens, in rank order, with lp(child) = lp(parent) + logp_j(token)
// in fp32.  Creation order matches the Clover draft's: depth by depth, parents in creation
// order, children in rank order.  One workgroup per sequence; the cumulative log-probs of
// a depth are written before the next depth reads them.
__global__ __launch_bounds__(TREE_THREADS) void medusa_expand_kernel(const MedusaExpandParams p) {
  const int b = blockIdx.x, slot = p.seq_ids[b];
  const size_t cb = (size_t)slot * p.cand_stride;
  int base_prev = 0, base = 1, fprev = 1;
  for (int j = 1; j <= p.H; ++j) {
    const int k = p.topk[j - 1];
    const size_t row = ((size_t)(j - 1) * p.nbatch + b) * p.kmax;  // head j, sequence b
    for (int e = threadIdx.x; e < fprev * k; e += TREE_THREADS) {
      const int n = e / k, r = e % k, parent = base_prev + n, child = base + e;
      p.cand_token[cb + child] = p.tok[row + r];
      p.cand_parent[cb + child] = parent;
      p.cand_depth[cb + child] = j;
      p.cand_lp[cb + child] = p.cand_lp[cb + parent] + p.logp[row + r];
    }
    __syncthreads();
    base_prev = base;
    base += fprev * k;
    fprev *= k;
  }
}

hipError_t launch_medusa_expand(const MedusaExpandParams& p, hipStream_t st) {
  if (p.nbatch <= 0) return hipSuccess;
  if (p.H < 1 || p.H > 8 || p.kmax < 1 || p.kmax > 16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(medusa_expand_kernel, dim3(p.nbatch), dim3(TREE_THREADS), 0, st, p);
  return hipGetLastError();
}

// ---- Augmenting Block at commit (Sec. 3.3: the block runs over the newly committed rows) --------
// Rows b*(H+1) + j, j = 0..H, of sequence b: the residual x_N of accepted node acc[j] (the
// last accepted node repeated past A), at position and KV slot L + j.  Rows past A stand in
// for a fixed launch size; their keys land in slots past the committed length, which the
// next tree overwrites.
__global__ void ab_commit_rows_kernel(const int* seq_ids, int T, int H, const int* acc, const int* acc_len,
                                      const int* seq_len, const float* x_tree, int d, float* x_rows,
                                      int* row_pos, int* row_slot, int* row_seq) {
  const int b = blockIdx.x, j = blockIdx.y, slot = seq_ids[b];
  const int A = acc_len[slot], L = seq_len[slot];
  const int src = acc[(size_t)slot * (H + 1) + min(j, A - 1)];
  const int row = b * (H + 1) + j;
  const float4* s = reinterpret_cast<const float4*>(x_tree + (size_t)(b * T + src) * d);
  float4* o = reinterpret_cast<float4*>(x_rows + (size_t)row * d);
  for (int k = threadIdx.x; k < d / 4; k += blockDim.x) o[k] = s[k];
  if (threadIdx.x == 0) {
    row_pos[row] = L + j;
    row_slot[row] = L + j;
    row_seq[row] = slot;
  }
}

hipError_t launch_ab_commit_rows(const int* seq_ids, int nbatch, int T, int H, const int* acc, const int* acc_len,
                                 const int* seq_len, const float* x_tree, int d, float* x_rows, int* row_pos,
                                 int* row_slot, int* row_seq, hipStream_t st) {
  if (nbatch <= 0) return hipSuccess;
  if (d % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ab_commit_rows_kernel, dim3(nbatch, H + 1), dim3(256), 0, st, seq_ids, T, H, acc, acc_len,
                     seq_len, x_tree, d, x_rows, row_pos, row_slot, row_seq);
  return hipGetLastError();
}

// h_0 of each listed sequence: the block's output at its last accepted row b*(H+1) + A - 1
__global__ void ab_commit_h0_kernel(const int* seq_ids, int H, const int* acc_len, const float* ab_rows, int d,
                                    float* h0) {
  const int b = blockIdx.x, slot = seq_ids[b];
  const float* s = ab_rows + (size_t)(b * (H + 1) + acc_len[slot] - 1) * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) h0[(size_t)slot * d + k] = s[k];
}

hipError_t launch_ab_commit_h0(const int* seq_ids, int nbatch, int H, const int* acc_len, const float* ab_rows,
                               int d, float* h0, hipStream_t st) {
  if (nbatch <= 0) return hipSuccess;
  hipLaunchKernelGGL(ab_commit_h0_kernel, dim3(nbatch), dim3(256), 0, st, seq_ids, H, acc_len, ab_rows, d, h0);
  return hipGetLastError();
}

__global__ void finish_prefill_kernel(int slot, const int* amax, const float* ab_row, int d, int* t0,
                                      float* h0) {
  if (threadIdx.x == 0) t0[slot] = amax[0];
  for (int k = threadIdx.x; k < d; k += blockDim.x) h0[(size_t)slot * d + k] = ab_row[k];
}

hipError_t launch_finish_prefill(int slot, const int* amax, const float* ab_row, int d, int* t0,
                                 float* h0, hipStream_t st) {
  hipLaunchKernelGGL(finish_prefill_kernel, dim3(1), dim3(256), 0, st, slot, amax, ab_row, d, t0, h0);
  return hipGetLastError();
}

}  // namespace clover
