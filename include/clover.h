/*
 * clover.h — C ABI of the MI355X (gfx950) Clover speculate-and-verify library.
 *
 * The library implements one decoding step of Clover speculative decoding
 * (Xiao et al., "Clover: Regressive Lightweight Speculative Decoding with
 * Sequential Knowledge", arXiv 2405.00263): a prefill phase that processes a
 * prompt and yields the first token (Sec. 1), then speculate-and-verify steps
 * in which the Clover heads draft a token tree (Sec. 3: Augmenting Block,
 * Regressive Connection, Attention Decoder, shared LM head) and the target
 * model verifies the whole tree in one tree-masked forward (Sec. 2.1, 2.2),
 * keeping the longest path that agrees with its own greedy choice.
 *
 * Conventions
 *  - All pointers documented as "device" are HIP device pointers on the current
 *    device; "host" pointers are ordinary host memory.  The library never
 *    allocates device memory: the caller provides weights and one workspace.
 *  - Every call validates its arguments on the host before enqueuing work; a
 *    status other than CLOVER_OK means nothing was enqueued and the context
 *    state is unchanged, except CLOVER_ERR_DEVICE, which is sticky.
 *  - A context is bound to one HIP stream and is not thread-safe.
 *  - Matrices are row-major [out_features, in_features] in the caller's layout;
 *    clover_pack_weight converts each into the library's tiled layout.
 */
#ifndef CLOVER_H
#define CLOVER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CLOVER_OK = 0,
  CLOVER_ERR_INVALID_ARG = 1, /* malformed config or argument */
  CLOVER_ERR_CAPACITY = 2,    /* context length, batch or workspace exceeded */
  CLOVER_ERR_STATE = 3,       /* sequence not in the state the call needs */
  CLOVER_ERR_BAD_TREE = 4,    /* planted tree malformed (parent >= index, token range) */
  CLOVER_ERR_DEVICE = 5       /* a HIP call failed; the context is unusable */
} clover_status;

typedef enum { CLOVER_F32 = 0, CLOVER_BF16 = 1 } clover_dtype;

/* Speculator of the step.
 *  CLOVER_DRAFT_CLOVER: the Clover heads (Sec. 3): Augmenting Block state, per depth the
 *    Regressive Connection and Attention Decoder on every frontier node, the head's MLP
 *    and the shared LM head; the tree grows one regressive depth per head.
 *  CLOVER_DRAFT_MEDUSA: the Medusa baseline the paper compares against (Sec. 1, 2.3;
 *    Sec. 4.3: Clover without Attention Decoder, Regressive Connection and Augmenting
 *    Block): every head reads the target's last hidden state of the last committed
 *    token, head j's top-k tokens become the depth-j children of every depth-(j-1) node
 *    (Cartesian product), and all heads share one LM-head pass.  There is no Augmenting
 *    Block and no Attention Decoder, so their weights are absent from the weight list. */
typedef enum { CLOVER_DRAFT_CLOVER = 0, CLOVER_DRAFT_MEDUSA = 1 } clover_draft_mode;

/* Augmenting Block variants explored in Sec. 4.3: a whole pre-norm transformer layer
 * (attention and MLP halves), the attention half only, the MLP half only, or none (the
 * heads then read x_N, the residual after the target's last layer).  Its output at the
 * last committed token is the drafting state h_0.  CLOVER_AB_DEFAULT is CLOVER_AB_FULL
 * for the Clover draft and CLOVER_AB_NONE for the Medusa draft; a Medusa draft with an
 * Augmenting Block is Clover without Attention Decoder and Regressive Connection. */
typedef enum {
  CLOVER_AB_DEFAULT = 0,
  CLOVER_AB_FULL = 1,
  CLOVER_AB_ATTN = 2,
  CLOVER_AB_MLP = 3,
  CLOVER_AB_NONE = 4
} clover_ab_mode;

/* Key set of the Attention Decoder (Eq. 1-2).  Read literally, Eq. 1 gives one key, the
 * embedding e_{i-1} of the previous token, so the softmax weight is exactly 1 and h_i =
 * h_{i-1} + W_O W_V e_{i-1} (W_Q and W_K do not change the result).  Sec. 3.2's remark that
 * the decoder takes only two vectors per request or beam reads as the key set
 * {RMSNorm_ad(h_{i-1}), e_{i-1}}; the third reading attends over the embeddings of every
 * token on the node's root path. */
typedef enum {
  CLOVER_AD_KEYS_SINGLE = 0, /* { e_{i-1} } (default) */
  CLOVER_AD_KEYS_TWO = 1,    /* { RMSNorm_ad(h_{i-1}), e_{i-1} } */
  CLOVER_AD_KEYS_PATH = 2    /* { e_0, ..., e_{i-1} } along the root path */
} clover_ad_keys;

/* Regressive block of the Clover draft.  The Attention Decoder (Sec. 3.2, Eq. 1-2) is the
 * paper's choice; its ablation (Sec. 3.2 last paragraph, Sec. 4.3 "Ablations on
 * Components") replaces it by an MLP over the two input vectors concatenated:
 *   h_i = h_{i-1} + SiLU(W_r [RMSNorm_r(h_{i-1}); e_{i-1}] + b_r),
 * W_r of shape [d_model, 2 d_model] (weights rb.norm, rb.w, rb.b), shared by the heads. */
typedef enum {
  CLOVER_REGRESSIVE_ATTENTION = 0, /* Attention Decoder (default) */
  CLOVER_REGRESSIVE_MLP = 1        /* MLP over [RMSNorm_r(h); e] */
} clover_regressive;

#define CLOVER_MAX_HEADS 8

/* Model and decoding configuration.  The target model is a pre-norm decoder
 * (RMSNorm, rotary embedding with rotate-half pairing, SwiGLU MLP, grouped KV
 * heads).  The speculator has n_spec_heads = number of topk entries heads. */
typedef struct {
  int32_t n_layers;     /* decoder layers of the target model */
  int32_t d_model;      /* hidden size, multiple of 32 */
  int32_t n_heads;      /* query heads */
  int32_t n_kv_heads;   /* key/value heads, divides n_heads */
  int32_t head_dim;     /* 32, 64 or 128 */
  int32_t ffn_dim;      /* SwiGLU inner size, multiple of 16 (32 for bf16) */
  int32_t vocab;        /* vocabulary size, multiple of 16 */
  float rms_eps;        /* RMSNorm epsilon */
  float rope_theta;     /* rotary base */
  int32_t dtype;        /* clover_dtype: storage type of weights, activations fed to GEMMs, KV */
  int32_t n_spec_heads; /* Clover heads H (1..CLOVER_MAX_HEADS) */
  int32_t topk[CLOVER_MAX_HEADS]; /* per-depth branching of the candidate tree */
  int32_t tree_tokens;  /* verify tokens per sequence T, root included, 1..128 */
  int32_t max_batch;    /* sequences that may be active at once */
  int32_t max_context;  /* committed tokens + T per sequence */
  int32_t kv_block;     /* KV page size in tokens; must be 16 */
  int32_t prefill_chunk;/* prompt rows per prefill chunk (multiple of 64); 0 = 256 */
  int32_t flags;        /* CLOVER_FLAG_* */
  int32_t draft_mode;   /* clover_draft_mode */
  int32_t ab_mode;      /* clover_ab_mode */
  int32_t ad_keys;      /* clover_ad_keys (Clover draft) */
  int32_t ad_per_head;  /* 0: one Attention Decoder shared by all heads (Eq. 1 has no head
                           index); 1: one per head (weights ad{j}.* for depth j + 1) */
  float temperature;    /* 0: greedy decoding (the target's argmax, Sec. 2.1).  > 0: the target
                           samples its next token from softmax(logits / temperature) at the
                           prompt's end and at every tree node (Gumbel-max over Philox4x32-10
                           draws, counter (token id, tree node, step of the sequence, slot), key
                           (sample_seed, 0 for tree nodes / 1 for the prompt's end)); acceptance
                           follows the child carrying the node's sample, so every emitted token
                           is a sample of the target given the tokens before it */
  uint32_t sample_seed;
  int32_t regressive;   /* clover_regressive (Clover draft); with CLOVER_REGRESSIVE_MLP, ad_keys
                           must be single and ad_per_head 0 */
  int32_t medusa_lm_heads; /* Medusa draft only.  0: the heads share the target's LM head (one
                           LM-head pass over every head's rows); 1: each head carries its own
                           LM head, as in the original Medusa (Sec. 3.4): weights head{j}.lm
                           [vocab, d_model], one LM-head pass per head */
} clover_config;

#define CLOVER_FLAG_KEEP_LOGITS 1 /* the verify and prefill LM heads also store their fp32 logits,
                                     readable as "verify_logits" until the next step or prefill;
                                     without it they store only the per-row argmax keys the
                                     target's choices need, and "verify_logits" keeps whatever
                                     an earlier flagged call left (the draft logits are always
                                     stored: top-k reads them) */
#define CLOVER_FLAG_PROFILE 2     /* time every kernel launch with HIP events (clover_kernel_stats);
                                     implies CLOVER_FLAG_EAGER */
#define CLOVER_FLAG_EAGER 4       /* launch the step's kernels one by one instead of replaying the
                                     HIP graphs captured per batch size on first use */
#define CLOVER_FLAG_AB_COMMIT 8   /* run the Augmenting Block at commit, over each sequence's
                                     accepted rows, for every batch size.  Without it the block
                                     runs there only when the verify has 129 or more rows
                                     (batch x tree_tokens), and otherwise over the whole tree as
                                     one more layer of the verify forward, its KV compacted with
                                     the target's: both give the same h_0 and cache */

typedef struct clover_ctx clover_ctx;

/* ---- configuration queries (pure host functions) ---------------------------------- */

/* Validate a configuration; CLOVER_OK or CLOVER_ERR_INVALID_ARG (message via
 * clover_last_error(NULL)). */
clover_status clover_check_config(const clover_config* cfg);

/* Canonical weight order: emb, layer{l}.{attn_norm,wq,wk,wv,wo,mlp_norm,w_gate,w_up,w_down},
 * final_norm, lm_head, ab.{same nine}, ad.{norm,wq,wk,wv,wo}, head{j}.{w1,b1}.
 * The ab.* tensors are the Augmenting Block (Sec. 3.3), ad.* the Attention Decoder
 * (Sec. 3.2, Eq. 1-2), head{j}.* the per-head MLP layers; lm_head is shared by all
 * heads and supplies the Regressive Connection embeddings (Sec. 3.4).  With
 * CLOVER_DRAFT_MEDUSA the ad.* entries are left out; with ad_per_head they are
 * ad{j}.{norm,wq,wk,wv,wo} for each head j instead of one ad.* set; with CLOVER_REGRESSIVE_MLP
 * they are rb.{norm [d], w [d, 2d], b [d]} instead of ad.*; with medusa_lm_heads each head's
 * entries are head{j}.{w1,b1,lm}; the ab.* entries are those of the
 * Augmenting Block's halves that clover_ab_mode keeps (attn_norm, wq, wk, wv, wo for the
 * attention half, mlp_norm, w_gate, w_up, w_down for the MLP half). */
size_t clover_weight_count(const clover_config* cfg);
/* Writes the NUL-terminated name of weight i into buf; returns its length or -1. */
int clover_weight_name(const clover_config* cfg, size_t i, char* buf, size_t buflen);
/* Writes the shape of weight i into out (row-major [rows, cols] or [n]); returns ndim or -1. */
int clover_weight_shape(const clover_config* cfg, size_t i, int64_t out[2]);
/* Bytes of weight i in the library's layout (what clover_pack_weight writes). */
size_t clover_packed_bytes(const clover_config* cfg, size_t i);
/* Bytes of the workspace clover_init needs. */
size_t clover_workspace_bytes(const clover_config* cfg);

/* Convert weight i from the caller's row-major layout (device src, storage dtype)
 * into the library's layout (device dst of clover_packed_bytes bytes).  Vectors are
 * copied unchanged; matrices are tiled for the matrix cores.  Enqueued on stream. */
clover_status clover_pack_weight(const clover_config* cfg, size_t i, const void* src, void* dst,
                                 void* hip_stream);

/* ---- context ---------------------------------------------------------------------- */

/* weights: clover_weight_count device pointers in canonical order, each in the layout
 * clover_pack_weight produced; they must outlive the context.  workspace: device
 * memory of at least clover_workspace_bytes(cfg) bytes, owned by the caller. */
clover_status clover_init(const clover_config* cfg, void* const* weights, void* workspace,
                          size_t ws_bytes, void* hip_stream, clover_ctx** out);
void clover_destroy(clover_ctx* ctx);

/* Message of the last failure on ctx (or of the last context-free call when ctx is NULL). */
const char* clover_last_error(const clover_ctx* ctx);

/* Prefill (Sec. 1): process the n prompt tokens (host array) of sequence slot seq
 * and return the first generated token (greedy) in *first_token (host).  The
 * Augmenting Block runs over the prompt so the first draft can start.  Errors:
 * INVALID_ARG (seq out of range, n < 1, token outside [0, vocab)), STATE (seq
 * active), CAPACITY (n + tree_tokens > max_context).  Blocks until done. */
clover_status clover_prefill(clover_ctx* ctx, int32_t seq, const int32_t* tokens, int32_t n,
                             int32_t* first_token);

/* One speculate-and-verify step (Sec. 2.1, 3) for each listed active sequence:
 * draft a candidate tree with the Clover heads, truncate it to tree_tokens, verify
 * it in one tree-masked forward, accept the longest path matching the target's
 * greedy tokens and commit its KV entries.  out_tokens: host [n_seqs][n_spec_heads+1];
 * out_count[s] = number of tokens emitted for seqs[s] (accepted speculated tokens plus
 * the bonus token, 1..n_spec_heads+1).  Errors: INVALID_ARG, STATE (inactive seq),
 * CAPACITY (a sequence would exceed max_context).  Blocks until done. */
clover_status clover_step(clover_ctx* ctx, const int32_t* seqs, int32_t n_seqs,
                          int32_t* out_tokens, int32_t* out_count);

/* Verify a caller-supplied tree instead of drafting (test hook for forcing
 * acceptance).  tokens/parents: host arrays of T entries, tokens[0] must be the
 * sequence's pending token, parents[0] = -1, 0 <= parents[i] < i.  T <= tree_tokens.
 * Accepts, commits and emits like clover_step.  Errors: BAD_TREE, plus those of
 * clover_step. */
clover_status clover_verify_tree(clover_ctx* ctx, int32_t seq, const int32_t* tokens,
                                 const int32_t* parents, int32_t T, int32_t* out_tokens,
                                 int32_t* out_count);

/* Deactivate a sequence slot and free its KV pages. */
clover_status clover_release(clover_ctx* ctx, int32_t seq);

/* Committed length of a sequence (host mirror), or -1 if inactive. */
int32_t clover_seq_len(const clover_ctx* ctx, int32_t seq);

/* ---- inspection (test hooks; not on the hot path) ------------------------------------ */

/* Copy a named device buffer of the last prefill/step to host memory (synchronous).
 * Names: "cand_token","cand_parent","cand_depth","cand_lp" (per sequence slot
 * [max_batch][n_candidates+1]); "tree_token","tree_parent","tree_depth","tree_pos"
 * ([max_batch][T]); "tree_mask" (u64 [max_batch][T][ceil(T/64)]); "target"
 * ([max_batch][T]); "acc" ([max_batch][H+1]); "acc_len" ([max_batch]); "h0"
 * (f32 [max_batch][d]); "t0" ([max_batch]); "verify_logits" (f32 [max_batch*T][V],
 * rows of the last verify); "draft_logits{j}" (f32 [max_batch*F_j][V], frontier rows of
 * depth j = 1..H); "x_last" (f32 [max_batch*T][d], residual after the last target
 * layer); "ab_out" (f32 [max_batch*T][d], Augmenting Block output over the tree).
 * Rows are in batch order of the last call (sequence list order).
 * *written receives the bytes copied (at most bytes). */
clover_status clover_debug_read(clover_ctx* ctx, const char* name, void* host_dst, size_t bytes,
                                size_t* written);

/* Read one committed K or V row of a layer (layer = n_layers selects the Augmenting
 * Block) at position pos of seq into host f32 [n_kv_heads*head_dim]. */
clover_status clover_debug_kv(clover_ctx* ctx, int32_t seq, int32_t layer, int32_t pos,
                              int32_t which_v, float* host_out);

/* Residual-stream trace (test hook for layer-by-layer parity).  While dev_buf is set, every
 * prefill chunk, step and planted-tree verify of rows rows writes f32 [n_layers + 2][rows]
 * [d_model] into dev_buf (device, caller-owned): slot l < n_layers holds the residual stream
 * entering target layer l (embedding for l = 0), slot n_layers the residual after the last
 * layer (x_N) and slot n_layers + 1 the Augmenting Block's output (x_N without one).  Rows
 * are those of the launch (batch order, tree nodes in order).  Traced calls launch eagerly
 * and fail with CAPACITY (state unchanged) when (n_layers + 2) * rows * d_model * 4 exceeds
 * bytes.  dev_buf NULL switches the trace off. */
clover_status clover_debug_trace(clover_ctx* ctx, float* dev_buf, size_t bytes);

typedef struct {
  float draft_ms, verify_ms, accept_ms, total_ms; /* last step, measured with HIP events */
  int32_t steps;
} clover_timings;
clover_status clover_get_timings(clover_ctx* ctx, clover_timings* out);

/* Per-kernel-class statistics accumulated over steps while CLOVER_FLAG_PROFILE is
 * set: launches, summed launch durations (HIP events on the context's stream) and the
 * algorithmic bytes and flops those launches must move and compute (each weight,
 * activation and output byte counted once).  Classes: */
enum {
  CLOVER_KSTAT_GEMM_VERIFY = 0, /* streaming GEMMs of the verify forward (layers, AB, LM head) */
  CLOVER_KSTAT_GEMM_DRAFT = 1,  /* streaming GEMMs of the Clover heads */
  CLOVER_KSTAT_ATTENTION = 2,   /* tree attention of the verify forward */
  CLOVER_KSTAT_OTHER = 3,       /* norms, embeddings, reductions, tree, acceptance */
  CLOVER_KSTAT_COUNT = 4
};
typedef struct {
  int64_t launches;
  double total_ms;
  double bytes;
  double flops;
} clover_kernel_stats;
clover_status clover_kernel_stats_get(clover_ctx* ctx, int32_t kind, clover_kernel_stats* out);
clover_status clover_kernel_stats_reset(clover_ctx* ctx);
/* Replace the context's CLOVER_FLAG_* bits (e.g. switch per-launch profiling on for a
 * measured pass and off again for graph replay). */
clover_status clover_set_flags(clover_ctx* ctx, int32_t flags);

/* ---- single-kernel entry points (parity tests at full size) ---------------------------
 * Each runs one hot-path kernel on caller buffers.  scratch: device memory of at least
 * scratch_bytes bytes (clover_op_scratch_bytes gives a sufficient size).  dtype is
 * clover_dtype of the storage-type operands.  All enqueue on hip_stream. */

size_t clover_op_scratch_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K);

/* Y[M][N] (f32, device) = X[M][K] (storage, device, row-major) * W^T, W packed from a
 * row-major [N][K] matrix by clover_pack_matrix. */
clover_status clover_op_linear(int32_t dtype, const void* X, int32_t M, int32_t K, const void* Wp,
                               int32_t N, float* Y, void* scratch, size_t scratch_bytes,
                               void* hip_stream);
size_t clover_packed_matrix_bytes(int32_t dtype, int32_t rows, int32_t cols);
clover_status clover_pack_matrix(int32_t dtype, const void* src, int32_t rows, int32_t cols,
                                 void* dst, void* hip_stream);

/* clover_op_linear for callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that forbid allocation): the same kernels, with the split-K
 * partials in a 16 MiB device array the library owns (one per GPU, kept until the process
 * ends) instead of a caller scratch buffer.  The call allocates nothing.  Shapes whose
 * partials need more than clover_op_linear_noalloc_max_bytes() bytes (clover_op_scratch_bytes)
 * are rejected with CLOVER_ERR_CAPACITY before anything is enqueued.  Every call on one GPU
 * shares that GPU's array, so calls that overlap in time on one GPU (other streams, other
 * threads) race; calls ordered on one stream do not.  Errors: INVALID_ARG, CAPACITY, DEVICE. */
size_t clover_op_linear_noalloc_max_bytes(void);
clover_status clover_op_linear_noalloc(int32_t dtype, const void* X, int32_t M, int32_t K, const void* Wp,
                                       int32_t N, float* Y, void* hip_stream);

/* The target layer's gated MLP activation (the SwiGLU feed-forward of the pre-norm decoder
 * whose forward the verify runs, Sec. 2.1): act[M][F] (storage, device, row-major) =
 * silu(X W_gate^T) * (X W_up^T), each product in fp32, the result rounded once to the storage
 * type.  X: [M][K] storage (device, row-major); Wg_p, Wu_p: [F][K] matrices packed by
 * clover_pack_matrix (F a multiple of 16, K of 32 for bf16 and 16 for f32).  Uses the
 * kernel and plan the verify's MLP takes for M rows.  Needs no scratch; returns
 * CLOVER_ERR_INVALID_ARG for bad sizes or null pointers, CLOVER_ERR_DEVICE if the launch
 * fails. */
clover_status clover_op_swiglu(int32_t dtype, const void* X, int32_t M, int32_t K, const void* Wg_p,
                               const void* Wu_p, int32_t F, void* act, void* hip_stream);

/* Tree attention (Sec. 2.2) for one sequence: queries Q[T][n_heads][head_dim] at
 * positions L + depth attend to prefix keys 0..L-1 and to tree keys j with
 * mask[i][j] (ancestor-or-self of i, from parents).  Kpre/Vpre: [L][n_kv][hd] and
 * Ktree/Vtree: [T][n_kv][hd] (storage, device, already rotated) are written into a
 * paged cache inside scratch, then attended.  O: [T][n_heads][hd] storage (device).
 * parents: host [T].  causal != 0 ignores parents and uses a causal tail. */
size_t clover_op_attention_scratch_bytes(int32_t dtype, int32_t L, int32_t T, int32_t n_heads,
                                         int32_t n_kv, int32_t head_dim);
clover_status clover_op_attention(int32_t dtype, const void* Q, const void* Kpre,
                                  const void* Vpre, const void* Ktree, const void* Vtree,
                                  int32_t L, int32_t T, const int32_t* parents, int32_t causal,
                                  int32_t n_heads, int32_t n_kv, int32_t head_dim, void* O,
                                  void* scratch, size_t scratch_bytes, void* hip_stream);

/* Per-row argmax (lowest index on ties) of f32 logits [M][V] -> out[M] int32 (device).
 * scratch: device memory of at least 8*M bytes. */
clover_status clover_op_argmax(const float* logits, int32_t M, int32_t V, int32_t* out, void* scratch,
                               void* hip_stream);
/* Per-row top-k by (value desc, index asc) and log-softmax: tok[M][k] int32,
 * logp[M][k] f32 = logits - logsumexp(row) (device); scratch of
 * clover_op_topk_scratch_bytes(M, V, k) bytes (0 = invalid arguments). */
size_t clover_op_topk_scratch_bytes(int32_t M, int32_t V, int32_t k);
clover_status clover_op_topk(const float* logits, int32_t M, int32_t V, int32_t k, int32_t* tok,
                             float* logp, void* scratch, void* hip_stream);

/* Tree truncation (device arrays for one sequence): keep the T-1 best non-root
 * candidates by (lp desc, depth asc, index asc), list root + kept in creation
 * order; write tokens/parent/depth [T], pos [T] = L + depth and the ancestor mask
 * u64 [T][ceil(T/64)].  n_cand includes the root (index 0). */
clover_status clover_op_tree_build(const int32_t* cand_token, const int32_t* cand_parent,
                                   const int32_t* cand_depth, const float* cand_lp, int32_t n_cand,
                                   int32_t T, int32_t L, int32_t* tokens, int32_t* parent,
                                   int32_t* depth, int32_t* pos, uint64_t* mask, void* hip_stream);
/* Greedy acceptance (Sec. 2.1) on device arrays of one tree: acc[max_depth+1],
 * *acc_len, *bonus (device int32). */
clover_status clover_op_accept(const int32_t* tokens, const int32_t* parent, const int32_t* target,
                               int32_t T, int32_t max_depth, int32_t* acc, int32_t* acc_len,
                               int32_t* bonus, void* hip_stream);

/* KV compaction after acceptance (the step's commit; Sec. 2.1 keeps only the accepted
 * path): for every layer, the K and V rows of tree slot L + acc[j] move to slot L + j,
 * j = 0..A-1.  A destination may be an earlier source (acc[j] >= j), so every source is
 * read before any destination is written; slots other than L..L+A-1 are untouched.
 * kcache / vcache: device pools [n_layers][n_blocks][n_kv][16 * head_dim] in the library's
 * paged layout (storage dtype); block_table: host [n_table] physical block of each 16-slot
 * page of the sequence, each in [0, n_blocks); acc: host [A], 1 <= A <= 9, every
 * L + max(acc[j], j) < 16 * n_table.  scratch: device memory of at least 4 * (n_table + A)
 * bytes the call stages the two arrays in.  Synchronises hip_stream before returning.
 * Errors: INVALID_ARG (any bound above), CAPACITY (scratch too small), DEVICE. */
clover_status clover_op_compact(int32_t dtype, void* kcache, void* vcache, int32_t n_layers, int32_t n_blocks,
                                int32_t n_kv, int32_t head_dim, const int32_t* block_table, int32_t n_table,
                                int32_t L, const int32_t* acc, int32_t A, void* scratch, size_t scratch_bytes,
                                void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* CLOVER_H */
