// Host-side launch interfaces of the Clover gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace clover {

// Message returned by clover_last_error(NULL) after a failed context-free call.
void set_last_error(const char* msg);

}  // namespace clover

namespace clover {

// Optional events filled with a kernel's own start and end times (hipExtLaunchKernel), so
// that per-launch timing excludes the dispatch gaps that marker events would include.
struct LaunchTiming {
  hipEvent_t start, stop;
};

// ---- weight-streaming GEMM ------------------------------------------------------------
enum GemmEpilogue : int {
  EP_PARTIAL = 0,  // part[split][m][n] = partial y (fp32); S = 1 gives y itself
  EP_QKV = 2,      // rotary on q/k, q -> qbuf, k/v -> paged KV cache (unsplit)
  EP_SWIGLU = 3,   // out_s[m][j] = silu(gate) * up, gate/up tiles paired per group (unsplit)
};

struct GemmSeg {
  const void* w;  // packed weight
  int tiles;      // 16-row tiles in this segment
};

struct GemmParams {
  const void* X;  // [M][ldx] storage type
  int ldx, M, K, nchunks;
  GemmSeg seg[3];
  int nseg, ntiles, N;
  int ngroups, mchunks, S, cps;
  int max_splits;  // EP_PARTIAL: upper bound on K splits (1 = unsplit)
  float* part;     // EP_PARTIAL output [S][M][N]; with amax_part it may be null (keys only)
  // EP_PARTIAL with one split: optional per-(column group, row) argmax keys [ngroups][M]
  // of the output (amax_key order), reduced by launch_argmax_groups; null: off
  unsigned long long* amax_part;
  // Sampling with the argmax keys (amax_part): they rank logit * inv_temp + Gumbel noise,
  // so each row's argmax is a sample of softmax(logit / temperature) (Gumbel-max); inv_temp
  // 0 keeps the plain argmax.  The noise of row m, column v is the Philox word for counter
  // (v, m % samp_rows, samp_step[slot], slot), slot = samp_slot[m], key (samp_seed,
  // samp_domain).  The partial/logit outputs stay the plain logits.
  float inv_temp;
  uint32_t samp_seed, samp_domain;
  const int* samp_slot;
  const int* samp_step;
  int samp_rows;
  int mode;
  void* out_s; int ldos;
  // EP_QKV
  void* qbuf; int ldq;
  void* kcache; void* vcache;
  const int* row_kb;  // [M] physical KV slot of each row: cache block * 16 + slot % 16 (launch_rope_table)
  int n_heads, n_kv, hd;
  const float* rope_cs;  // [M][hd/2] (cos, sin) pairs of each row's position (launch_rope_table)
};

struct GemmPlan {
  int tiled;     // 0: weight-streaming kernel; 1: register-blocked kernel (bf16, large M);
                 // 2: 32x32 matrix-core kernel (gemm_wide.hip; mt, tw, ring = its MB, NB, stages)
  int nw;        // waves per workgroup (streaming: one 16-row weight tile each, 2..8; tiled: 4 or 8)
  int mt;        // m-tiles of 16 rows per chunk (streaming 1, 2 or 4) or per wave (tiled, 4)
  int tw;        // tiled: 16-row weight tiles per wave
  int ring;      // tiled: register prefetch depth in LDS stages
  int mchunks, ngroups, S, cps;
  size_t lds_bytes;
  size_t part_floats;
};

// mode: the epilogue (EP_PARTIAL, EP_QKV, EP_SWIGLU); seg_tiles/nseg: the weight segments'
// 16-row tile counts; amax: EP_PARTIAL with argmax keys.  Plans depend on all of them.
GemmPlan plan_gemm(int dtype, int M, int ntiles, int nchunks, bool swiglu, int max_splits, int mode = EP_PARTIAL,
                   const int* seg_tiles = nullptr, int nseg = 0, bool amax = false);
// From this many rows on, bf16 Q|K|V and split-K projections may use the 32x32 kernel.
constexpr int WIDE_MIN_M = 512;
bool plan_wide(int M, int ntiles, int nchunks, int mode, int max_splits, const int* seg_tiles, int nseg,
               GemmPlan& out);
hipError_t launch_wide(GemmParams& p, const GemmPlan& pl, hipStream_t st, const LaunchTiming* lt);
// Plan and launch of the register-blocked kernel (plan_gemm picks it for bf16 and large M).
GemmPlan plan_tiled(int M, int ntiles, int nchunks, bool swiglu, int max_splits);
// a plan of one instantiated shape (mt, tw, ring, nw waves) and split, for sweeps
GemmPlan plan_tiled_forced(int M, int ntiles, int nchunks, bool swiglu, int mt, int tw, int ring, int nw, int S);
hipError_t launch_tiled(GemmParams& p, const GemmPlan& pl, hipStream_t st, const LaunchTiming* lt);
// Fills plan fields of p and launches; returns hipSuccess or an error.
hipError_t launch_gemm(int dtype, GemmParams& p, hipStream_t st, const LaunchTiming* lt = nullptr);
// Q|K|V from K-split partials part[S][M][N] (a GEMM in EP_PARTIAL mode over the packed Q|K|V
// weights): sums in split order, rotary, Q to qbuf and K/V to the paged cache, exactly as the
// EP_QKV epilogue.  p carries the EP_QKV fields.
hipError_t launch_qkv_fix(int dtype, const GemmParams& p, const float* part, int S, hipStream_t st);
// rope_hd > 0: a Q/K weight of heads rope_hd wide, packed so that each 16-row tile holds
// 8 dims of a head's first rotary half and their 8 partners (tile-local rotary epilogue)
hipError_t launch_pack(int dtype, const void* src, int rows, int cols, void* dst, int rope_hd,
                       hipStream_t st);
size_t packed_matrix_bytes(int dtype, int rows, int cols);

// ---- attention -------------------------------------------------------------------------
struct AttnParams {
  const void* Q; int ldq;          // rows [M][n_heads*hd] storage
  void* O; int ldo;                // output rows, storage
  const void* kcache; const void* vcache;
  const int* block_table; int max_blocks;
  const int* seq_ids;              // batch index -> sequence slot
  const int* prefix_dev;           // per slot committed length (or null)
  int prefix_host;                 // used when prefix_dev is null
  int rows_per_seq;                // query rows of one sequence in Q (T or chunk)
  int nq;                          // valid query rows per sequence
  int n_tail;                      // tail keys (slots prefix .. prefix+n_tail-1)
  int causal;                      // tail mask: causal (1) or tree bitmask (0)
  const uint64_t* mask; int mask_words; int mask_seq_stride;  // per slot [T][words]
  int n_heads, n_kv, hd;
  int nbatch;
  float* part; size_t part_cap;    // fp32 split partials (attention_part_floats), or null
  // filled by plan_attention: query tiles per head, per (sequence, KV head), per
  // workgroup (4 or 8), workgroups per (sequence, KV head) in the query direction, key splits
  int qph, qt_item, qtile, qgroups, splits;
};
// Plans the launch (fields above) and runs it: the attention kernel and, with more than
// one key split, the merge kernel.  max_keys bounds prefix + tail over the batch.
hipError_t launch_attention(int dtype, AttnParams& p, int max_keys, hipStream_t st,
                            const LaunchTiming* lt = nullptr);
// write rows [n][n_kv*hd] (storage) of K and V into the paged cache at slots slot0.. of seq
hipError_t launch_kv_write(int dtype, const void* K, const void* V, int n, int slot0, int seq,
                           void* kcache, void* vcache, const int* block_table, int max_blocks,
                           int n_kv, int hd, hipStream_t st);
// fp32 partial floats a launch with these shape fields needs (0 with one split)
size_t attention_part_floats(const AttnParams& p);
void plan_attention(AttnParams& p);

// ---- row kernels -------------------------------------------------------------------------
hipError_t launch_embed(int dtype, const void* emb, const int* tok, int M, int d, float* x,
                        hipStream_t st);
// cs[m][i] = (cos, sin)(pos[m] * theta^(-2i/hd)), i < hd/2: the rotary factors of each row
// Per-row tables of a forward over M rows, written once before its layers: the rotary
// factors cs [M][hd/2] of each row's position and, when kb is given, each row's physical KV
// slot kb[m] = block_table[seq[m]][slot[m] / 16] * 16 + slot[m] % 16 (the Q|K|V epilogues'
// append target), so the per-layer kernels do not repeat the two dependent table loads.
hipError_t launch_rope_table(const int* pos, int M, int hd, float theta, float* cs, hipStream_t st,
                             const int* seq = nullptr, const int* slot = nullptr,
                             const int* block_table = nullptr, int max_blocks = 0, int* kb = nullptr);
// out[m] = argmax of row m from the keys[G][M] a GEMM left in GemmParams::amax_part (G =
// its plan's ngroups)
hipError_t launch_argmax_groups(const unsigned long long* keys, int G, int M, int* out, hipStream_t st);
// keys: M u64 scratch; keys_zeroed: a previous kernel already cleared them
hipError_t launch_argmax(const float* logits, int M, int V, int* out, unsigned long long* keys,
                         bool keys_zeroed, hipStream_t st);
// top-k of rows with log-softmax; writes either plain (tok/logp [M][k]) or candidate
// records (children of frontier rows).
struct TopkParams {
  const float* logits; int M, V, k;
  int* tok; float* logp;                          // plain output (may be null)
  // candidate output: frontier row f = b*F + fl, children at cand index base_child + fl*k + r
  const int* seq_ids; int F;
  int* cand_token; int* cand_parent; int* cand_depth; float* cand_lp; int cand_stride;
  int base_parent, base_child, depth;
  float* scratch;  // topk_scratch_floats(M, k)
};
size_t topk_scratch_floats(int M, int V, int k);
hipError_t launch_topk(TopkParams& p, hipStream_t st);

struct RowFixParams {
  int M, d;
  const float* part; int S; int ldp;   // split-K partials [S][M][ldp] (S = 0: none)
  const float* resid; int ldr;         // residual input (null: 0)
  int act;                             // 0: y = sum; 1: y = silu(sum + bias)
  const void* bias;                    // storage [d]
  float* out_f; int ldo;               // resid + y (may alias resid)
  float* out_copy_f;                   // optional fp32 copy [M][d]
  void* out_copy_s;                    // optional storage copy [M][d]
  const void* gain; float eps;         // RMSNorm gain (storage)
  void* out_norm; int ldn;             // optional RMSNorm(result) * gain, storage
  unsigned long long* zero_keys; int zero_n;  // optional: clear argmax keys
  int no_resid;                        // set by launch_rowfix: resid was null (read, then zeroed)
};
hipError_t launch_rowfix(int dtype, RowFixParams& p, hipStream_t st);

struct AdPrepParams {
  // frontier row f = b*F + fl of depth j; parent state row = prev[b*Fprev + fl/kprev]
  const float* prev; int Fprev, kprev;   // prev = per-slot h0 when j == 1 (indexed by slot)
  int use_slot_state;                    // 1: prev indexed by seq slot (h0), 0: by batch row
  const int* seq_ids; int nbatch, F;
  const int* cand_token; int cand_stride, base_node;
  const void* lm_packed; int lm_nchunks;
  const void* ad_norm; float eps; int d;
  float* hin; void* a_out; void* e_out;
  int ld_out;                            // row stride of a_out / e_out in elements (0: d)
};
hipError_t launch_ad_prep(int dtype, AdPrepParams& p, hipStream_t st);
// Attention Decoder attention (Eq. 1-2) of the M frontier rows of one depth.  Queries from
// the Q GEMM's split-K partials q[Sq][M][H*hd]; keys/values from the K|V GEMM's partials
// kv[Skv][rows][2*H*hd] (keys then values), where the key set of row f is
//   AD_KEYS_SINGLE: { e(token) }                      (kv row f)
//   AD_KEYS_TWO:    { RMSNorm_ad(h), e(token) }       (kv rows f and M + f)
//   AD_KEYS_PATH:   { e(t) : t on the row's root path } (earlier depths from kv_path, own: kv row f)
// With AD_KEYS_PATH the row's own key/value is also stored in kv_path at depth `depth`
// (rows [B * nodes(d)] per depth d from kv_path_off[d]); an ancestor at depth d < depth of
// frontier row f = b * F + fl is row b * nodes(d) + fl / anc_div[d] there.
enum AdKeys : int { AD_KEYS_SINGLE = 0, AD_KEYS_TWO = 1, AD_KEYS_PATH = 2 };
struct AdAttnParams {
  const float* q; int Sq;
  const float* kv; int Skv;
  // AD_KEYS_SINGLE only: kv holds values alone, [Skv][M][H*hd], and q is unused.  With one
  // key the softmax weight is exactly 1 and the output is the value, so the query and key
  // projections are not computed.
  int values_only;
  int M, F, n_heads, hd, keys, depth;
  float* kv_path;                 // AD_KEYS_PATH: [sum_d B*nodes(d)][2*H*hd] fp32
  int kv_path_off[8], path_nodes[8], anc_div[8];
  void* out;                      // [M][H*hd] storage
};
hipError_t launch_ad_attn(int dtype, const AdAttnParams& p, hipStream_t st);

// ---- tree, acceptance, compaction -----------------------------------------------------------
struct TreeParams {
  const int* seq_ids; int nbatch;
  const int* cand_token; const int* cand_parent; const int* cand_depth; const float* cand_lp;
  int cand_stride, n_cand;  // n_cand includes the root
  int T, mask_words;
  const int* seq_len;       // per slot (or null: seq_len_host)
  int seq_len_host;
  int* tree_token; int* tree_parent; int* tree_depth; int* tree_pos; uint64_t* tree_mask;
  int* row_tok; int* row_pos; int* row_slot; int* row_seq;   // verify rows [nbatch*T] (optional)
};
hipError_t launch_tree_build(TreeParams& p, hipStream_t st);

struct AcceptParams {
  const int* seq_ids; int nbatch, T, H;
  const int* tree_token; const int* tree_parent; const int* target;  // target rows [nbatch*T]
  int* acc; int* acc_len; int* out_tokens; int* t0;
  const float* ab_out; int d; float* h0;      // AB output rows [nbatch*T][d]
  const float* x_last; float* x_keep;          // optional
  int* step_ctr;                               // optional per-slot step counter, +1 per step
};
hipError_t launch_accept(AcceptParams& p, hipStream_t st);

struct CompactParams {
  const int* seq_ids; int nbatch, H;     // seq_ids null: one sequence, slot 0
  const int* acc; const int* acc_len; const int* seq_len;  // acc_len / seq_len null: A_host / L_host
  int A_host, L_host;
  void* const* kpools; void* const* vpools; int nlayers;   // device arrays of pool pointers, or
  void* kbase; void* vbase; size_t layer_elems;             // (kpools null) pools at base + layer * layer_elems
  const int* block_table; int max_blocks;
  int n_kv, hd;
};
hipError_t launch_compact(int dtype, CompactParams& p, hipStream_t st);

// Medusa draft: candidate tree of every listed sequence from the heads' top-k lists
// tok/logp [H][nbatch][kmax] (Cartesian product; the root, candidate 0, is already set)
struct MedusaExpandParams {
  const int* seq_ids; int nbatch, H, kmax;
  int topk[8];
  const int* tok; const float* logp;
  int* cand_token; int* cand_parent; int* cand_depth; float* cand_lp; int cand_stride;
};
hipError_t launch_medusa_expand(const MedusaExpandParams& p, hipStream_t st);
// Medusa draft input: row b = h0[seq_ids[b]] as fp32 (out_f) and in the storage type (out_s)
hipError_t launch_gather_state(int dtype, const int* seq_ids, int nbatch, const float* h0, int d,
                               float* out_f, void* out_s, hipStream_t st);

hipError_t launch_fill_i32(int* p, int v, size_t n, hipStream_t st);
// draft root (candidate 0 of each listed slot) from the pending token t0[slot]
hipError_t launch_set_root(const int* seq_ids, int nbatch, const int* t0, int* cand_token,
                           int* cand_parent, int* cand_depth, float* cand_lp, int cand_stride,
                           hipStream_t st);
// Augmenting Block at commit: gather each listed sequence's accepted rows of x_N (tree rows
// [nbatch*T][d]) into x_rows [nbatch*(H+1)][d] with their positions / KV slots L + j, and
// afterwards take h_0 from the block's output at the last accepted row.
hipError_t launch_ab_commit_rows(const int* seq_ids, int nbatch, int T, int H, const int* acc, const int* acc_len,
                                 const int* seq_len, const float* x_tree, int d, float* x_rows, int* row_pos,
                                 int* row_slot, int* row_seq, hipStream_t st);
hipError_t launch_ab_commit_h0(const int* seq_ids, int nbatch, int H, const int* acc_len, const float* ab_rows,
                               int d, float* h0, hipStream_t st);
// end of prefill: t0[slot] = argmax result, h0[slot] = AB output row
hipError_t launch_finish_prefill(int slot, const int* amax, const float* ab_row, int d, int* t0,
                                 float* h0, hipStream_t st);

}  // namespace clover
