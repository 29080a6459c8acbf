// C ABI of the Clover library: configuration queries, weight packing, context
// lifetime, prefill, the speculate-and-verify step and test hooks.
//
// The host side validates every call before enqueuing work, keeps the paged-KV
// allocator and a mirror of each sequence's committed length, and orchestrates the
// kernels of one step on the context's stream:
//   draft  (Sec. 3): per depth j, Attention Decoder (Eq. 1-2) on the frontier, head MLP,
//          shared LM head, top-k -> candidate tree;  truncation -> verify tree
//   verify (Sec. 2.1, 2.2): one tree-masked forward of all layers, final norm, LM head,
//          greedy argmax per node; the Augmenting Block (Sec. 3.3) runs as one extra
//          layer over the tree with its own KV cache
//   accept: longest path matching the greedy tokens, bonus token, KV compaction of every
//          layer, h_0 for the next draft = Augmenting Block output at the last accepted node
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/clover.h"
#include "kernels.h"

using namespace clover;

namespace {

thread_local std::string g_err;

void set_global_err(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
}

}  // namespace

namespace clover {
void set_last_error(const char* msg) { set_global_err("%s", msg); }
}  // namespace clover

namespace {

constexpr size_t ALIGN = 256;
constexpr int GEMM_MAX_SPLITS = 8;
constexpr int QKV_MAX_SPLITS = 2;  // Q|K|V may be split when the plan prefers it (fix-up pass)
size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

int es_of(int dtype) { return dtype == CLOVER_BF16 ? 2 : 4; }
bool is_medusa(const clover_config& c) { return c.draft_mode == CLOVER_DRAFT_MEDUSA; }
bool mlp_regressive(const clover_config& c) { return !is_medusa(c) && c.regressive == CLOVER_REGRESSIVE_MLP; }
bool per_head_lm(const clover_config& c) { return is_medusa(c) && c.medusa_lm_heads == 1; }
int ab_mode(const clover_config& c) {
  if (c.ab_mode != CLOVER_AB_DEFAULT) return c.ab_mode;
  return is_medusa(c) ? CLOVER_AB_NONE : CLOVER_AB_FULL;
}
bool ab_attn(const clover_config& c) { return ab_mode(c) == CLOVER_AB_FULL || ab_mode(c) == CLOVER_AB_ATTN; }
bool ab_mlp(const clover_config& c) { return ab_mode(c) == CLOVER_AB_FULL || ab_mode(c) == CLOVER_AB_MLP; }
bool has_ab(const clover_config& c) { return ab_attn(c) || ab_mlp(c); }
// layers with a KV cache: the target's, plus the Augmenting Block's when it has attention
int kv_layers(const clover_config& c) { return c.n_layers + (ab_attn(c) ? 1 : 0); }
int kc_of(int dtype) { return dtype == CLOVER_BF16 ? 32 : 16; }

// ---- canonical weights ----------------------------------------------------------------
const char* kLayer[9] = {"attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down"};

struct WSpec {
  std::string name;
  int64_t rows, cols;  // cols == 0: vector of rows elements
  bool matrix;
};

// attn / mlp: include the attention half (attn_norm .. wo) / the MLP half (mlp_norm .. w_down)
void layer_specs(const clover_config& c, const std::string& pre, std::vector<WSpec>& out,
                 bool attn = true, bool mlp = true) {
  const int64_t d = c.d_model, F = c.ffn_dim, qd = (int64_t)c.n_heads * c.head_dim,
                kvd = (int64_t)c.n_kv_heads * c.head_dim;
  const int64_t shp[9][2] = {{d, 0}, {qd, d}, {kvd, d}, {kvd, d}, {d, qd}, {d, 0}, {F, d}, {F, d}, {d, F}};
  for (int i = 0; i < 9; ++i)
    if (i < 5 ? attn : mlp) out.push_back({pre + "." + kLayer[i], shp[i][0], shp[i][1], shp[i][1] != 0});
}

std::vector<WSpec> weight_specs(const clover_config& c) {
  std::vector<WSpec> s;
  const int64_t d = c.d_model, V = c.vocab, qd = (int64_t)c.n_heads * c.head_dim;
  s.push_back({"emb", V, d, false});  // gathered by rows, kept row-major
  for (int l = 0; l < c.n_layers; ++l) layer_specs(c, "layer" + std::to_string(l), s);
  s.push_back({"final_norm", d, 0, false});
  s.push_back({"lm_head", V, d, true});
  if (has_ab(c)) layer_specs(c, "ab", s, ab_attn(c), ab_mlp(c));
  if (mlp_regressive(c)) {  // the MLP regressive block over [RMSNorm(h); e]
    s.push_back({"rb.norm", d, 0, false});
    s.push_back({"rb.w", d, 2 * d, true});
    s.push_back({"rb.b", d, 0, false});
  } else if (!is_medusa(c)) {  // ad.* shared, or ad{j}.* per head
    for (int j = 0; j < (c.ad_per_head ? c.n_spec_heads : 1); ++j) {
      const std::string pre = c.ad_per_head ? "ad" + std::to_string(j) : std::string("ad");
      s.push_back({pre + ".norm", d, 0, false});
      s.push_back({pre + ".wq", qd, d, true});
      s.push_back({pre + ".wk", qd, d, true});
      s.push_back({pre + ".wv", qd, d, true});
      s.push_back({pre + ".wo", d, qd, true});
    }
  }
  for (int j = 0; j < c.n_spec_heads; ++j) {
    s.push_back({"head" + std::to_string(j) + ".w1", d, d, true});
    s.push_back({"head" + std::to_string(j) + ".b1", d, 0, false});
    if (per_head_lm(c)) s.push_back({"head" + std::to_string(j) + ".lm", V, d, true});
  }
  return s;
}

int n_candidates(const clover_config& c) {  // root excluded
  int total = 0, width = 1;
  for (int j = 0; j < c.n_spec_heads; ++j) {
    width *= c.topk[j];
    total += width;
  }
  return total;
}
int frontier(const clover_config& c, int j) {  // rows expanded at depth j (1-based)
  int w = 1;
  for (int i = 0; i < j - 1; ++i) w *= c.topk[i];
  return w;
}
int depth_base(const clover_config& c, int depth) {  // first candidate index of a depth
  int base = 0, w = 1;
  for (int i = 0; i < depth; ++i) {
    base += w;
    w *= c.topk[i];
  }
  return base;
}
int prefill_chunk(const clover_config& c) { return c.prefill_chunk > 0 ? c.prefill_chunk : 256; }

bool check_config(const clover_config* c, std::string& why) {
  char buf[256];
  auto fail = [&](const char* m) { why = m; return false; };
  if (!c) return fail("config is null");
  if (c->dtype != CLOVER_F32 && c->dtype != CLOVER_BF16) return fail("dtype must be F32 or BF16");
  if (c->draft_mode != CLOVER_DRAFT_CLOVER && c->draft_mode != CLOVER_DRAFT_MEDUSA)
    return fail("draft_mode must be CLOVER_DRAFT_CLOVER or CLOVER_DRAFT_MEDUSA");
  if (c->ab_mode < CLOVER_AB_DEFAULT || c->ab_mode > CLOVER_AB_NONE) return fail("ab_mode out of range");
  if (c->ad_keys < CLOVER_AD_KEYS_SINGLE || c->ad_keys > CLOVER_AD_KEYS_PATH) return fail("ad_keys out of range");
  if (c->ad_per_head != 0 && c->ad_per_head != 1) return fail("ad_per_head must be 0 or 1");
  if (c->regressive != CLOVER_REGRESSIVE_ATTENTION && c->regressive != CLOVER_REGRESSIVE_MLP)
    return fail("regressive must be CLOVER_REGRESSIVE_ATTENTION or CLOVER_REGRESSIVE_MLP");
  if (c->medusa_lm_heads != 0 && c->medusa_lm_heads != 1) return fail("medusa_lm_heads must be 0 or 1");
  if (c->medusa_lm_heads == 1 && c->draft_mode != CLOVER_DRAFT_MEDUSA)
    return fail("per-head LM heads belong to the Medusa draft (the Clover heads share the LM head)");
  if (c->regressive == CLOVER_REGRESSIVE_MLP && (c->ad_keys != CLOVER_AD_KEYS_SINGLE || c->ad_per_head))
    return fail("the MLP regressive block takes no Attention Decoder key set or per-head decoders");
  if (!(c->temperature >= 0.f) || c->temperature > 1e30f) return fail("temperature must be finite and >= 0");
  const int kc = kc_of(c->dtype);
  if (c->n_layers < 1 || c->n_layers > 1024) return fail("n_layers out of range");
  if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128) return fail("head_dim must be 32, 64 or 128");
  if (c->n_heads < 1 || c->n_kv_heads < 1 || c->n_heads % c->n_kv_heads) return fail("n_kv_heads must divide n_heads");
  if (c->d_model < kc || c->d_model % kc || c->d_model % 16) return fail("d_model must be a multiple of 16 (fp32) or 32 (bf16)");
  if (((int64_t)c->n_heads * c->head_dim) % kc) return fail("n_heads*head_dim must be a multiple of the K chunk");
  if (c->ffn_dim < 16 || c->ffn_dim % 16 || c->ffn_dim % kc) return fail("ffn_dim must be a multiple of 16 (fp32) or 32 (bf16)");
  if (c->vocab < 16 || c->vocab % 16) return fail("vocab must be a positive multiple of 16");
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f)) return fail("rms_eps/rope_theta invalid");
  if (c->n_spec_heads < 1 || c->n_spec_heads > CLOVER_MAX_HEADS) return fail("n_spec_heads must be 1..8");
  for (int j = 0; j < c->n_spec_heads; ++j)
    if (c->topk[j] < 1 || c->topk[j] > 16) return fail("topk entries must be 1..16");
  if (c->tree_tokens < 1 || c->tree_tokens > 128) return fail("tree_tokens must be 1..128");
  const int64_t nc = n_candidates(*c);
  if (nc + 1 < c->tree_tokens) return fail("the full candidate tree has fewer nodes than tree_tokens");
  if (nc + 1 > 1024) return fail("candidate tree larger than 1024 nodes");
  if (c->max_batch < 1 || c->max_batch > 256) return fail("max_batch must be 1..256");
  if (c->kv_block != 16) return fail("kv_block must be 16");
  if (c->max_context < c->tree_tokens + 1) return fail("max_context must exceed tree_tokens");
  if (c->max_context > 65536) return fail("max_context must be at most 65536");
  if (c->prefill_chunk < 0 || c->prefill_chunk % 64) return fail("prefill_chunk must be a multiple of 64");
  if ((int64_t)c->max_batch * frontier(*c, c->n_spec_heads) > 4096) return fail("draft frontier too large");
  (void)buf;
  return true;
}

// ---- workspace layout ------------------------------------------------------------------
struct Layout {
  int es, T, W, H, NC, Mv, Mp, Mmax, Fsum, Fmaxrows, mbps, nblocks;
  size_t pool_bytes;
  size_t kpool, vpool, pool_ptrs, block_table, seq_len, seq_ids;
  size_t x, xa, xab, xn, qbuf, obuf, act, vlogits, row_tok, row_pos, row_slot, row_seq, row_kb, amax;
  size_t sample_step;  // per slot: speculate-and-verify steps done since its prefill (sampling counters)
  size_t rope_cs;  // [Mmax][hd/2] (cos, sin) of the current rows' positions
  size_t h0, t0, cand_token, cand_parent, cand_depth, cand_lp;
  size_t tree_token, tree_parent, tree_depth, tree_pos, tree_mask, target, acc, acc_len, out_tokens;
  size_t dstate[CLOVER_MAX_HEADS], dlogits[CLOVER_MAX_HEADS];
  size_t d_hin, d_a, d_e, d_q, d_kv, d_o, d_sst, d_r, d_rn;
  size_t d_kvpath;  // path key set: fp32 keys/values of every drafted depth's nodes
  size_t m_tok, m_logp;  // Medusa draft: per-(head, sequence) top-k tokens and log-probs
  size_t gpart, gpart2, amax_part, topk_scratch;
  size_t apart, apart_floats;  // attention split partials
  size_t gpart_floats, gpart2_floats;
  size_t total;
};

Layout make_layout(const clover_config& c) {
  Layout L{};
  L.es = es_of(c.dtype);
  L.T = c.tree_tokens;
  L.W = (L.T + 63) / 64;
  L.H = c.n_spec_heads;
  L.NC = n_candidates(c) + 1;
  L.Mv = c.max_batch * L.T;
  L.Mp = prefill_chunk(c);
  L.Mmax = std::max(L.Mv, L.Mp);
  L.Fsum = 0;
  L.Fmaxrows = 0;
  for (int j = 1; j <= L.H; ++j) {
    L.Fsum += c.max_batch * frontier(c, j);
    L.Fmaxrows = std::max(L.Fmaxrows, c.max_batch * frontier(c, j));
  }
  if (is_medusa(c)) L.Fmaxrows = std::max(L.Fmaxrows, c.max_batch * L.H);  // all heads' rows at once
  L.mbps = (c.max_context + 15) / 16;
  L.nblocks = c.max_batch * L.mbps;
  const int64_t d = c.d_model, V = c.vocab, F = c.ffn_dim, hd = c.head_dim;
  const int64_t qd = c.n_heads * hd, kvd = c.n_kv_heads * hd;
  const int NL = kv_layers(c);  // base layers (+ Augmenting Block)
  L.pool_bytes = align_up((size_t)L.nblocks * kvd * 16 * L.es);
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + std::max<size_t>(bytes, 1)); return o; };
  L.kpool = take(L.pool_bytes * NL);
  L.vpool = take(L.pool_bytes * NL);
  L.pool_ptrs = take(sizeof(void*) * 2 * NL);
  L.block_table = take(sizeof(int) * (size_t)c.max_batch * L.mbps);
  L.seq_len = take(sizeof(int) * c.max_batch);
  L.seq_ids = take(sizeof(int) * c.max_batch);
  L.sample_step = take(sizeof(int) * c.max_batch);  // zeroed at init with the state
  L.x = take(4 * (size_t)L.Mmax * d);
  L.xa = take(4 * (size_t)L.Mmax * d);
  L.xab = take(4 * (size_t)c.max_batch * (L.H + 1) * d);  // commit-time Augmenting Block rows
  L.xn = take((size_t)L.es * L.Mmax * d);
  L.qbuf = take((size_t)L.es * L.Mmax * qd);
  L.obuf = take((size_t)L.es * L.Mmax * qd);
  L.act = take((size_t)L.es * L.Mmax * F);
  L.vlogits = take(4 * (size_t)L.Mv * V);
  L.row_tok = take(4 * (size_t)L.Mmax);
  L.row_pos = take(4 * (size_t)L.Mmax);
  L.row_slot = take(4 * (size_t)L.Mmax);
  L.row_seq = take(4 * (size_t)L.Mmax);
  L.row_kb = take(4 * (size_t)L.Mmax);
  L.rope_cs = take(4 * (size_t)L.Mmax * c.head_dim);
  L.amax = take(4 * (size_t)L.Mv);
  L.h0 = take(4 * (size_t)c.max_batch * d);
  L.t0 = take(4 * (size_t)c.max_batch);
  const size_t ncand = (size_t)c.max_batch * L.NC;
  L.cand_token = take(4 * ncand);
  L.cand_parent = take(4 * ncand);
  L.cand_depth = take(4 * ncand);
  L.cand_lp = take(4 * ncand);
  const size_t nt = (size_t)c.max_batch * L.T;
  L.tree_token = take(4 * nt);
  L.tree_parent = take(4 * nt);
  L.tree_depth = take(4 * nt);
  L.tree_pos = take(4 * nt);
  L.tree_mask = take(8 * nt * L.W);
  L.target = take(4 * nt);
  L.acc = take(4 * (size_t)c.max_batch * (L.H + 1));
  L.acc_len = take(4 * (size_t)c.max_batch);
  L.out_tokens = take(4 * (size_t)c.max_batch * (L.H + 1));
  if (is_medusa(c)) {
    // one LM-head pass over every head's rows: logits [H][batch][V], head after head
    const size_t all = take(4 * (size_t)L.H * c.max_batch * V);
    for (int j = 1; j <= L.H; ++j) L.dlogits[j - 1] = all;
    L.m_tok = take(4 * (size_t)L.H * c.max_batch * 16);
    L.m_logp = take(4 * (size_t)L.H * c.max_batch * 16);
  } else {
    for (int j = 1; j <= L.H; ++j) {
      const size_t rows = (size_t)c.max_batch * frontier(c, j);
      L.dstate[j - 1] = take(4 * rows * d);
      L.dlogits[j - 1] = take(4 * rows * V);
    }
  }
  const size_t fr = L.Fmaxrows;
  L.d_hin = take(4 * fr * d);
  L.d_a = take((size_t)L.es * 2 * fr * d);  // normalised states, then embeddings (two-token keys)
  L.d_e = take((size_t)L.es * fr * d);
  L.d_q = take(4 * fr * qd);
  L.d_kv = take(4 * fr * 2 * qd);
  L.d_o = take((size_t)L.es * fr * qd);
  L.d_sst = take((size_t)L.es * fr * d);
  L.d_r = take(4 * fr * d);
  L.d_rn = take((size_t)L.es * fr * d);
  L.d_kvpath = take(c.ad_keys == CLOVER_AD_KEYS_PATH ? 4 * (size_t)L.Fsum * 2 * qd : 0);
  // split-K partials [S][M][N] of the residual-type GEMMs (at most GEMM_MAX_SPLITS)
  const size_t maxM = std::max<size_t>({(size_t)L.Mv, (size_t)L.Mp, (size_t)L.Fmaxrows});
  const size_t maxN = std::max<size_t>({(size_t)d, (size_t)qd});
  L.gpart_floats = std::max((size_t)GEMM_MAX_SPLITS * maxM * maxN,
                            (size_t)QKV_MAX_SPLITS * maxM * (size_t)(qd + 2 * c.n_kv_heads * c.head_dim));
  L.gpart2_floats = (size_t)GEMM_MAX_SPLITS * 2 * L.Fmaxrows * 2 * qd;  // Attention Decoder keys/values
  L.gpart = take(4 * L.gpart_floats);
  L.gpart2 = take(4 * L.gpart2_floats);
  // per-(column group, row) argmax keys of the LM-head epilogue: a group holds at least
  // two 16-column tiles in every plan
  L.amax_part = take(8 * ((size_t)V / 32 + 1) * (size_t)L.Mv);
  L.topk_scratch = take(4 * topk_scratch_floats(L.Fmaxrows, (int)V, 16));
  // attention split partials: the largest of the verify launches (every batch size) and
  // the prefill chunks (every chunk length)
  {
    AttnParams a{};
    a.n_heads = c.n_heads; a.n_kv = c.n_kv_heads; a.hd = c.head_dim;
    size_t af = 0;
    for (int b = 1; b <= c.max_batch; ++b) {
      a.nbatch = b; a.nq = L.T;
      af = std::max(af, attention_part_floats(a));
      a.nq = L.H + 1;  // the Augmenting Block at commit
      af = std::max(af, attention_part_floats(a));
    }
    a.nbatch = 1;
    for (int rows = 16; rows < L.Mp + 16; rows += 16) {
      a.nq = std::min(rows, L.Mp);
      af = std::max(af, attention_part_floats(a));
    }
    L.apart_floats = af;
    L.apart = take(4 * std::max<size_t>(af, 1));
  }
  L.total = off;
  return L;
}

}  // namespace

// ---- context -----------------------------------------------------------------------------

struct LayerPtrs {
  const void *attn_norm, *wq, *wk, *wv, *wo, *mlp_norm, *wg, *wu, *wd;
};

struct clover_ctx {
  clover_config cfg;
  Layout L;
  hipStream_t st;
  char* ws;
  std::vector<const void*> w;
  std::vector<LayerPtrs> layers;  // n_layers (+ Augmenting Block last, Clover draft)
  const void *emb, *final_norm, *lm_head;
  struct AdPtrs { const void *norm, *wq, *wk, *wv, *wo; };
  std::vector<AdPtrs> ad;  // one Attention Decoder shared by the heads, or one per head
  const void *rb_norm = nullptr, *rb_w = nullptr, *rb_b = nullptr;  // MLP regressive block
  std::vector<const void*> head_w1, head_b1;
  std::vector<const void*> head_lm;  // Medusa heads' own LM heads (medusa_lm_heads)
  // host state
  std::vector<int> seq_len;                  // -1 inactive
  std::vector<std::vector<int>> seq_blocks;  // physical KV blocks per slot
  std::vector<int> free_blocks;
  int* bt_host = nullptr;  // pinned host copy of the block table [max_batch][mbps]: the step's
                           // block-table updates are copied from it like the other pinned staging
  std::vector<int> host_ids, host_len;
  int* pin_ids = nullptr;   // pinned host staging of the step's sequence ids [max_batch]
  int* pin_len = nullptr;   // ... and of the committed lengths [max_batch]
  int* pin_out = nullptr;   // ... and of the emitted tokens [max_batch][H+1]
  std::string err;
  bool dead = false;
  hipEvent_t ev[4] = {};
  clover_timings tim{};
  int last_nbatch = 0;
  // per-launch profiling (CLOVER_FLAG_PROFILE)
  bool profile = false, in_step = false;
  int phase = CLOVER_KSTAT_GEMM_VERIFY;
  std::vector<hipEvent_t> pev;
  struct Pending { int kind; size_t ev; double bytes, flops; };
  std::vector<Pending> pend;
  clover_kernel_stats kst[CLOVER_KSTAT_COUNT]{};
  // captured step phases per batch size
  struct StepGraphs { hipGraphExec_t draft = nullptr, verify = nullptr, accept = nullptr; };
  std::vector<StepGraphs> graphs;
  bool use_graphs = true;
  float* trace = nullptr;  // residual-stream trace (clover_debug_trace): [n_layers + 2][rows][d]
  size_t trace_bytes = 0;
  hipStream_t cap_st = nullptr;  // private stream the phases are captured on (the caller's
                                 // stream may be the legacy default stream, which cannot be)

  template <typename T> T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
};

namespace {

clover_status ctx_fail(clover_ctx* c, clover_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  c->err = buf;
  return s;
}

// ---- per-launch timing ---------------------------------------------------------------
// Marker events around the scope's launches; with `kernel_events` the scope holds a single
// launch that records the pair itself from the kernel's own start and end (see timing()).
struct ProfScope {
  clover_ctx* c;
  bool on, kev;
  LaunchTiming lt{};
  ProfScope(clover_ctx* c_, int kind, double bytes, double flops, bool kernel_events = false)
      : c(c_), on(c_->profile && c_->in_step), kev(kernel_events) {
    if (!on) return;
    const size_t i = c->pend.size() * 2;
    while (c->pev.size() < i + 2) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) { on = false; return; }
      c->pev.push_back(e);
    }
    lt = {c->pev[i], c->pev[i + 1]};
    if (!kev) (void)hipEventRecord(lt.start, c->st);
    c->pend.push_back({kind, i, bytes, flops});
  }
  const LaunchTiming* timing() const { return on && kev ? &lt : nullptr; }
  ~ProfScope() {
    if (on && !kev) (void)hipEventRecord(lt.stop, c->st);
  }
};

void prof_collect(clover_ctx* c) {  // after a stream sync
  for (auto& p : c->pend) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, c->pev[p.ev], c->pev[p.ev + 1]) != hipSuccess) continue;
    auto& k = c->kst[p.kind];
    k.launches += 1;
    k.total_ms += ms;
    k.bytes += p.bytes;
    k.flops += p.flops;
  }
  c->pend.clear();
}

#define HIPCK(ctx, expr)                                                                  \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess) {                                                               \
      (ctx)->dead = true;                                                                 \
      return ctx_fail((ctx), CLOVER_ERR_DEVICE, "%s failed: %s", #expr, hipGetErrorString(e_)); \
    }                                                                                     \
  } while (0)

// Y = X W^T through the streaming GEMM.  EP_PARTIAL writes [S][M][N] fp32 partials to
// `part` (S <= max_splits; the consumer sums them) and returns S through *splits.
hipError_t run_gemm(clover_ctx* c, GemmParams p, int M, int K,
                    std::initializer_list<std::pair<const void*, int>> segs, int* splits = nullptr,
                    int* groups = nullptr) {
  p.M = M;
  p.K = K;
  p.nchunks = K / kc_of(c->cfg.dtype);
  p.nseg = 0;
  p.ntiles = 0;
  for (auto& s : segs) {
    p.seg[p.nseg++] = GemmSeg{s.first, s.second / 16};
    p.ntiles += s.second / 16;
  }
  if (p.mode != EP_SWIGLU) p.N = p.ntiles * 16;
  const double es = es_of(c->cfg.dtype);
  const double rows = p.ntiles * 16.0;
  const double ybytes = (p.mode == EP_PARTIAL ? 4.0 : es) * M * p.N;
  hipError_t e;
  {
    ProfScope ps(c, c->phase, rows * K * es + es * M * K + ybytes, 2.0 * M * rows * K, true);
    e = launch_gemm(c->cfg.dtype, p, c->st, ps.timing());
  }
  if (splits) *splits = p.S;
  if (groups) *groups = p.ngroups;
  return e;
}

// Per-row tables of a forward over M rows (rotary factors, KV append slots) from row_pos,
// row_seq, row_slot and the block table, once before its layers.
hipError_t row_tables(clover_ctx* c, int M) {
  const Layout& L = c->L;
  return launch_rope_table(c->at<int>(L.row_pos), M, c->cfg.head_dim, c->cfg.rope_theta, c->at<float>(L.rope_cs),
                           c->st, c->at<int>(L.row_seq), c->at<int>(L.row_slot), c->at<int>(L.block_table), L.mbps,
                           c->at<int>(L.row_kb));
}

// Residual-stream trace: copy the M rows of x into trace slot `idx` (clover_debug_trace).
hipError_t trace_rows(clover_ctx* c, int idx, const float* x, int M) {
  if (!c->trace) return hipSuccess;
  const size_t n = (size_t)M * c->cfg.d_model;
  return hipMemcpyAsync(c->trace + (size_t)idx * n, x, 4 * n, hipMemcpyDeviceToDevice, c->st);
}

// resid_norm: x += sum of pending partials; xn = RMSNorm(x) * gain (storage)
hipError_t run_rowfix(clover_ctx* c, RowFixParams rp) {
  ProfScope ps(c, CLOVER_KSTAT_OTHER, 0, 0);
  return launch_rowfix(c->cfg.dtype, rp, c->st);
}

// The attention half of a layer on the normalised rows in xn: Q|K|V with rotary and paged
// KV append, tree-masked (or causal) attention, output projection into split-K partials in
// gpart, whose split count it returns through *splits.
hipError_t run_attention_half(clover_ctx* c, const LayerPtrs& lw, int layer_idx, int M, AttnParams att,
                              int max_keys, int* splits) {
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  const int d = cf.d_model, hd = cf.head_dim, qd = cf.n_heads * hd, kvd = cf.n_kv_heads * hd;
  void* xn = c->at<void>(L.xn);
  float* part = c->at<float>(L.gpart);
  void* kp = c->ws + L.kpool + L.pool_bytes * layer_idx;
  void* vp = c->ws + L.vpool + L.pool_bytes * layer_idx;
  hipError_t e;
  GemmParams g{};
  g.X = xn; g.ldx = d; g.mode = EP_QKV;
  g.qbuf = c->at<void>(L.qbuf); g.ldq = qd;
  g.kcache = kp; g.vcache = vp;
  g.row_kb = c->at<int>(L.row_kb);
  g.n_heads = cf.n_heads; g.n_kv = cf.n_kv_heads; g.hd = hd; g.rope_cs = c->at<float>(L.rope_cs);
  const int qkv_tiles = (qd + 2 * kvd) / 16, kc = kc_of(cf.dtype);
  const int qkv_seg[3] = {qd / 16, kvd / 16, kvd / 16};
  if (plan_gemm(cf.dtype, M, qkv_tiles, d / kc, false, QKV_MAX_SPLITS, EP_QKV, qkv_seg, 3).S > 1) {
    // K-split Q|K|V: partials, then the fix-up pass (sums, rotary, stores)
    g.mode = EP_PARTIAL; g.max_splits = QKV_MAX_SPLITS; g.part = part;
    int sq = 1;
    if ((e = run_gemm(c, g, M, d, {{lw.wq, qd}, {lw.wk, kvd}, {lw.wv, kvd}}, &sq))) return e;
    g.M = M;
    ProfScope ps(c, CLOVER_KSTAT_OTHER, 0, 0);
    if ((e = launch_qkv_fix(cf.dtype, g, part, sq, c->st))) return e;
  } else if ((e = run_gemm(c, g, M, d, {{lw.wq, qd}, {lw.wk, kvd}, {lw.wv, kvd}}))) {
    return e;
  }
  att.Q = c->at<void>(L.qbuf); att.ldq = qd;
  att.O = c->at<void>(L.obuf); att.ldo = qd;
  att.kcache = kp; att.vcache = vp;
  att.block_table = c->at<int>(L.block_table); att.max_blocks = L.mbps;
  att.n_heads = cf.n_heads; att.n_kv = cf.n_kv_heads; att.hd = hd;
  {
    const double es = L.es;
    const double keys = (double)max_keys;  // upper bound over the batch
    ProfScope ps(c, CLOVER_KSTAT_ATTENTION,
                 att.nbatch * (2.0 * keys * kvd * es + 2.0 * att.nq * qd * es),
                 att.nbatch * 4.0 * att.nq * keys * hd * cf.n_heads, true);
    if ((e = launch_attention(cf.dtype, att, max_keys, c->st, ps.timing()))) return e;
  }
  GemmParams o{};
  o.X = c->at<void>(L.obuf); o.ldx = qd; o.mode = EP_PARTIAL; o.max_splits = GEMM_MAX_SPLITS; o.part = part;
  return run_gemm(c, o, M, qd, {{lw.wo, d}}, splits);
}

// One pre-norm decoder layer over M rows of the residual `x` (in place).  `pend` is the
// split count of the previous down-projection partials in gpart still to be added to
// x (0: none); returns through *pend_out the split count of this layer's last
// partials (down projection, or the output projection without the MLP half), which the
// caller's next row kernel adds.  attn / mlp: run the attention / MLP half (Augmenting
// Block variants; target layers run both).
hipError_t run_layer(clover_ctx* c, const LayerPtrs& lw, int layer_idx, float* x, int M,
                     AttnParams att, int max_keys, int pend, int* pend_out, bool attn = true,
                     bool mlp = true) {
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  const int d = cf.d_model;
  void* xn = c->at<void>(L.xn);
  float* part = c->at<float>(L.gpart);
  hipError_t e;
  RowFixParams rf{};
  rf.M = M; rf.d = d; rf.part = part; rf.S = pend; rf.ldp = d;
  rf.resid = x; rf.ldr = d; rf.out_f = x; rf.ldo = d;
  rf.gain = attn ? lw.attn_norm : lw.mlp_norm; rf.eps = cf.rms_eps; rf.out_norm = xn; rf.ldn = d;
  if ((e = run_rowfix(c, rf))) return e;
  if (layer_idx < cf.n_layers && (e = trace_rows(c, layer_idx, x, M))) return e;  // the layer's input
  if (attn) {
    if ((e = run_attention_half(c, lw, layer_idx, M, att, max_keys, pend_out))) return e;
    if (!mlp) return hipSuccess;
    rf.S = *pend_out; rf.gain = lw.mlp_norm;
    if ((e = run_rowfix(c, rf))) return e;
  }
  GemmParams gu{};
  gu.X = xn; gu.ldx = d; gu.mode = EP_SWIGLU;
  gu.out_s = c->at<void>(L.act); gu.ldos = cf.ffn_dim; gu.N = cf.ffn_dim;
  if ((e = run_gemm(c, gu, M, d, {{lw.wg, cf.ffn_dim}, {lw.wu, cf.ffn_dim}}))) return e;
  GemmParams dn{};
  dn.X = c->at<void>(L.act); dn.ldx = cf.ffn_dim; dn.mode = EP_PARTIAL; dn.max_splits = GEMM_MAX_SPLITS;
  dn.part = c->at<float>(L.gpart);
  return run_gemm(c, dn, M, cf.ffn_dim, {{lw.wd, d}}, pend_out);
}


clover_status ensure_blocks(clover_ctx* c, int slot, int upto) {
  const int need = (upto + 15) / 16;
  auto& bl = c->seq_blocks[slot];
  if (need > c->L.mbps) return ctx_fail(c, CLOVER_ERR_CAPACITY, "sequence %d needs %d KV blocks > %d", slot, need, c->L.mbps);
  if ((int)bl.size() >= need) return CLOVER_OK;
  if ((int)c->free_blocks.size() < need - (int)bl.size())
    return ctx_fail(c, CLOVER_ERR_CAPACITY, "KV pool exhausted");
  const int first = (int)bl.size();
  while ((int)bl.size() < need) {
    bl.push_back(c->free_blocks.back());
    c->free_blocks.pop_back();
  }
  int* row = c->bt_host + (size_t)slot * c->L.mbps;
  for (int i = first; i < need; ++i) row[i] = bl[i];
  HIPCK(c, hipMemcpyAsync(c->at<int>(c->L.block_table) + (size_t)slot * c->L.mbps + first,
                          row + first, sizeof(int) * (need - first), hipMemcpyHostToDevice, c->st));
  return CLOVER_OK;
}

#define HE(expr)                        \
  do {                                  \
    hipError_t e_ = (expr);             \
    if (e_ != hipSuccess) return e_;    \
  } while (0)

// The verify and prefill LM heads write their fp32 logits only on request; the target's
// choices need only the argmax keys of the epilogue.
bool keep_logits(const clover_ctx* c) { return (c->cfg.flags & CLOVER_FLAG_KEEP_LOGITS) != 0; }

// Where the Augmenting Block runs (Sec. 3.3: it extends the committed rows).  Over the whole
// tree as layer N+1 of the verify, its KV compacted with the others, when the verify's rows
// are few: its weights stream once either way.  At commit, over the <= H+1 accepted rows of
// each sequence, when the verify has enough rows (B*T >= 129, the matrix-bound regime) that
// running the block over every tree row would cost compute the commit does not.
constexpr int AB_COMMIT_MIN_ROWS = 129;
bool ab_at_commit(const clover_ctx* c, int B) {
  return has_ab(c->cfg) &&
         ((c->cfg.flags & CLOVER_FLAG_AB_COMMIT) || B * c->L.T >= AB_COMMIT_MIN_ROWS);
}

// LM-head argmax keys of the target's choices: plain argmax (greedy), or with temperature a
// Gumbel-max sample per row (GemmParams::inv_temp).  domain 0: tree nodes (row m is node
// m % rows_per_seq of sequence slot_of_row[m]); 1: the token after the prompt.
void set_sampling(clover_ctx* c, GemmParams& lm, uint32_t domain, const int* slot_of_row, int rows_per_seq) {
  const clover_config& cf = c->cfg;
  if (!(cf.temperature > 0.f)) return;
  lm.inv_temp = 1.0f / cf.temperature;
  lm.samp_seed = cf.sample_seed;
  lm.samp_domain = domain;
  lm.samp_slot = slot_of_row;
  lm.samp_step = c->at<int>(c->L.sample_step);
  lm.samp_rows = rows_per_seq;
}

// Verify forward for the batch in seq_ids (tree already in device buffers): all target
// layers over the tree, final norm, LM head, greedy argmax, then the Augmenting Block
// over the tree.
hipError_t enq_verify(clover_ctx* c, int B, int max_keys) {
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  const int T = L.T, M = B * T, d = cf.d_model;
  float* x = c->at<float>(L.x);
  float* xa = c->at<float>(L.xa);
  HE(launch_embed(cf.dtype, c->emb, c->at<int>(L.row_tok), M, d, x, c->st));
  HE(row_tables(c, M));
  AttnParams att{};
  att.seq_ids = c->at<int>(L.seq_ids);
  att.prefix_dev = c->at<int>(L.seq_len);
  att.rows_per_seq = T; att.nq = T; att.n_tail = T; att.causal = 0;
  att.mask = c->at<uint64_t>(L.tree_mask); att.mask_words = L.W; att.mask_seq_stride = T * L.W;
  att.nbatch = B;
  att.part = c->at<float>(L.apart); att.part_cap = L.apart_floats;
  int pend = 0;
  for (int l = 0; l < cf.n_layers; ++l) HE(run_layer(c, c->layers[l], l, x, M, att, max_keys, pend, &pend));
  // x_N = x + last partials; kept in xa for the Augmenting Block; final norm; LM head; argmax
  RowFixParams rf{};
  rf.M = M; rf.d = d; rf.part = c->at<float>(L.gpart); rf.S = pend; rf.ldp = d;
  rf.resid = x; rf.ldr = d; rf.out_f = x; rf.ldo = d; rf.out_copy_f = xa;
  rf.gain = c->final_norm; rf.eps = cf.rms_eps; rf.out_norm = c->at<void>(L.xn); rf.ldn = d;
  HE(run_rowfix(c, rf));
  HE(trace_rows(c, cf.n_layers, x, M));
  // LM head; its epilogue leaves per-(column group, row) argmax keys, reduced per row
  GemmParams lm{};
  lm.X = c->at<void>(L.xn); lm.ldx = d; lm.mode = EP_PARTIAL; lm.max_splits = 1;
  lm.part = keep_logits(c) ? c->at<float>(L.vlogits) : nullptr;  // argmax keys only otherwise
  lm.amax_part = c->at<unsigned long long>(L.amax_part);
  set_sampling(c, lm, 0, c->at<int>(L.row_seq), T);
  int lm_groups = 0;
  HE(run_gemm(c, lm, M, d, {{c->lm_head, cf.vocab}}, nullptr, &lm_groups));
  {
    ProfScope ps(c, CLOVER_KSTAT_OTHER, 0, 0);
    HE(launch_argmax_groups(c->at<unsigned long long>(L.amax_part), lm_groups, M, c->at<int>(L.target), c->st));
  }
  // xa keeps x_N: the next draft reads it (no block), or the block runs at commit
  if (!has_ab(cf) || ab_at_commit(c, B)) return trace_rows(c, cf.n_layers + 1, xa, M);
  // Augmenting Block over the tree (tree mask, its own KV cache)
  HE(run_layer(c, c->layers[cf.n_layers], cf.n_layers, xa, M, att, max_keys, 0, &pend, ab_attn(cf), ab_mlp(cf)));
  RowFixParams ra{};
  ra.M = M; ra.d = d; ra.part = c->at<float>(L.gpart); ra.S = pend; ra.ldp = d;
  ra.resid = xa; ra.ldr = d; ra.out_f = xa; ra.ldo = d;
  HE(run_rowfix(c, ra));
  return trace_rows(c, cf.n_layers + 1, xa, M);
}

// Greedy acceptance, bonus token, KV compaction of every layer, h_0 for the next draft (the
// Augmenting Block's output at the last accepted node: from the tree, or from the block run
// here over the accepted rows).
hipError_t enq_accept(clover_ctx* c, int B, int max_keys) {
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  const int T = L.T, d = cf.d_model, H = L.H;
  const bool commit = ab_at_commit(c, B);
  AcceptParams ap{};
  ap.seq_ids = c->at<int>(L.seq_ids); ap.nbatch = B; ap.T = T; ap.H = H;
  ap.tree_token = c->at<int>(L.tree_token); ap.tree_parent = c->at<int>(L.tree_parent);
  ap.target = c->at<int>(L.target);
  ap.acc = c->at<int>(L.acc); ap.acc_len = c->at<int>(L.acc_len);
  ap.out_tokens = c->at<int>(L.out_tokens); ap.t0 = c->at<int>(L.t0);
  ap.ab_out = c->at<float>(L.xa); ap.d = d; ap.h0 = commit ? nullptr : c->at<float>(L.h0);
  ap.step_ctr = c->at<int>(L.sample_step);
  {
    ProfScope ps(c, CLOVER_KSTAT_OTHER, 0, 0);
    HE(launch_accept(ap, c->st));
  }
  CompactParams cp{};
  cp.seq_ids = c->at<int>(L.seq_ids); cp.nbatch = B; cp.H = H;
  cp.acc = c->at<int>(L.acc); cp.acc_len = c->at<int>(L.acc_len); cp.seq_len = c->at<int>(L.seq_len);
  cp.kpools = c->at<void*>(L.pool_ptrs); cp.vpools = c->at<void*>(L.pool_ptrs) + kv_layers(cf);
  cp.nlayers = commit ? cf.n_layers : kv_layers(cf);  // at commit the block writes its own KV
  cp.block_table = c->at<int>(L.block_table); cp.max_blocks = L.mbps;
  cp.n_kv = cf.n_kv_heads; cp.hd = cf.head_dim;
  {
    ProfScope ps(c, CLOVER_KSTAT_OTHER, 0, 0);
    HE(launch_compact(cf.dtype, cp, c->st));
  }
  if (!commit) return hipSuccess;
  // the Augmenting Block over each sequence's accepted rows (x_N), causal against its cache
  const int Mab = B * (H + 1);
  float* xr = c->at<float>(L.xab);  // x keeps the verify's last rows
  HE(launch_ab_commit_rows(c->at<int>(L.seq_ids), B, T, H, c->at<int>(L.acc), c->at<int>(L.acc_len),
                           c->at<int>(L.seq_len), c->at<float>(L.xa), d, xr, c->at<int>(L.row_pos),
                           c->at<int>(L.row_slot), c->at<int>(L.row_seq), c->st));
  HE(row_tables(c, Mab));
  AttnParams att{};
  att.seq_ids = c->at<int>(L.seq_ids);
  att.prefix_dev = c->at<int>(L.seq_len);
  att.rows_per_seq = H + 1; att.nq = H + 1; att.n_tail = H + 1; att.causal = 1;
  att.nbatch = B;
  att.part = c->at<float>(L.apart); att.part_cap = L.apart_floats;
  int pend = 0;
  HE(run_layer(c, c->layers[cf.n_layers], cf.n_layers, xr, Mab, att, max_keys, 0, &pend, ab_attn(cf), ab_mlp(cf)));
  RowFixParams ra{};
  ra.M = Mab; ra.d = d; ra.part = c->at<float>(L.gpart); ra.S = pend; ra.ldp = d;
  ra.resid = xr; ra.ldr = d; ra.out_f = xr; ra.ldo = d;
  HE(run_rowfix(c, ra));
  return launch_ab_commit_h0(c->at<int>(L.seq_ids), B, H, c->at<int>(L.acc_len), xr, d, c->at<float>(L.h0), c->st);
}

// Emitted tokens to the host, one stream sync, host mirrors and phase timings.
clover_status finish_step(clover_ctx* c, int B, int* out_tokens, int* out_count) {
  const Layout& L = c->L;
  const int H = L.H;
  HIPCK(c, hipMemcpyAsync(c->pin_out, c->at<int>(L.out_tokens), sizeof(int) * B * (H + 1),
                          hipMemcpyDeviceToHost, c->st));
  HIPCK(c, hipEventRecord(c->ev[3], c->st));
  // poll rather than block: the step's end is the latency the caller sees
  for (;;) {
    const hipError_t q = hipEventQuery(c->ev[3]);
    if (q == hipSuccess) break;
    if (q != hipErrorNotReady) HIPCK(c, q);
  }
  prof_collect(c);
  for (int b = 0; b < B; ++b) {
    int n = 0;
    for (int i = 0; i <= H; ++i) {
      const int t = c->pin_out[(size_t)b * (H + 1) + i];
      out_tokens[(size_t)b * (H + 1) + i] = t;
      if (t >= 0) ++n;
    }
    out_count[b] = n;
    c->seq_len[c->host_ids[b]] += n;
  }
  float ms;
  if (hipEventElapsedTime(&ms, c->ev[0], c->ev[1]) == hipSuccess) c->tim.draft_ms = ms;
  if (hipEventElapsedTime(&ms, c->ev[1], c->ev[2]) == hipSuccess) c->tim.verify_ms = ms;
  if (hipEventElapsedTime(&ms, c->ev[2], c->ev[3]) == hipSuccess) c->tim.accept_ms = ms;
  if (hipEventElapsedTime(&ms, c->ev[0], c->ev[3]) == hipSuccess) c->tim.total_ms = ms;
  c->tim.steps++;
  return CLOVER_OK;
}

// Run one phase of the step: eagerly, or through a HIP graph captured on first use for
// this batch size (the phase's launches depend only on the batch size; everything that
// changes between steps is read from device memory).
template <typename Fn>
hipError_t run_phase(clover_ctx* c, hipGraphExec_t* slot, bool graph, Fn&& fn) {
  if (!graph) return fn();
  if (!*slot) {
    hipError_t e = hipStreamBeginCapture(c->cap_st, hipStreamCaptureModeRelaxed);
    if (e != hipSuccess) return e;
    hipStream_t user = c->st;
    c->st = c->cap_st;  // the phase enqueues on c->st
    const hipError_t e2 = fn();
    c->st = user;
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(c->cap_st, &g);
    if (e2 != hipSuccess || e != hipSuccess) {
      if (g) (void)hipGraphDestroy(g);
      return e2 != hipSuccess ? e2 : e;
    }
    e = hipGraphInstantiate(slot, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (e != hipSuccess) {
      *slot = nullptr;
      return e;
    }
  }
  return hipGraphLaunch(*slot, c->st);
}

hipError_t enq_tree(clover_ctx* c, int B);

// Medusa draft (the paper's baseline, Sec. 2.3): every head reads the state h_0 of the last
// committed token -- x_N, or the Augmenting Block's output when one is configured; head j:
// r = h + SiLU(W1_j h + b1_j), logits = W_lm RMSNorm_f(r) -- the Clover head block without
// Attention Decoder and Regressive Connection (Sec. 4.3).  The heads' rows share one
// LM-head pass; their top-k lists span the candidate tree as a Cartesian product.
hipError_t enq_draft_medusa(clover_ctx* c, int B) {
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  const int d = cf.d_model, H = L.H;
  int* ids = c->at<int>(L.seq_ids);
  int *ct = c->at<int>(L.cand_token), *cpar = c->at<int>(L.cand_parent), *cd = c->at<int>(L.cand_depth);
  float* clp = c->at<float>(L.cand_lp);
  HE(launch_set_root(ids, B, c->at<int>(L.t0), ct, cpar, cd, clp, L.NC, c->st));
  HE(launch_gather_state(cf.dtype, ids, B, c->at<float>(L.h0), d, c->at<float>(L.d_hin), c->at<void>(L.d_a), c->st));
  float* part = c->at<float>(L.gpart);
  char* rn = c->at<char>(L.d_rn);
  for (int j = 1; j <= H; ++j) {
    int sh = 0;
    GemmParams hm{};
    hm.X = c->at<void>(L.d_a); hm.ldx = d; hm.mode = EP_PARTIAL; hm.max_splits = GEMM_MAX_SPLITS; hm.part = part;
    HE(run_gemm(c, hm, B, d, {{c->head_w1[j - 1], d}}, &sh));
    RowFixParams rh{};  // r = x + SiLU(W1 x + b1), then the shared final norm into head j's rows
    rh.M = B; rh.d = d; rh.part = part; rh.S = sh; rh.ldp = d;
    rh.resid = c->at<float>(L.d_hin); rh.ldr = d; rh.act = 1; rh.bias = c->head_b1[j - 1];
    rh.gain = c->final_norm; rh.eps = cf.rms_eps;
    rh.out_norm = rn + (size_t)(j - 1) * B * d * L.es; rh.ldn = d;
    HE(run_rowfix(c, rh));
  }
  if (per_head_lm(cf)) {
    // the original Medusa's heads each carry an LM head (Sec. 3.4): one pass per head
    for (int j = 0; j < H; ++j) {
      GemmParams lm{};
      lm.X = rn + (size_t)j * B * d * L.es; lm.ldx = d; lm.mode = EP_PARTIAL; lm.max_splits = 1;
      lm.part = c->at<float>(L.dlogits[0]) + (size_t)j * B * cf.vocab;
      HE(run_gemm(c, lm, B, d, {{c->head_lm[j], cf.vocab}}));
    }
  } else {
    GemmParams lm{};
    lm.X = rn; lm.ldx = d; lm.mode = EP_PARTIAL; lm.max_splits = 1;
    lm.part = c->at<float>(L.dlogits[0]);
    HE(run_gemm(c, lm, H * B, d, {{c->lm_head, cf.vocab}}));
  }
  int kmax = 1;
  for (int j = 0; j < H; ++j) kmax = std::max(kmax, cf.topk[j]);
  TopkParams tp{};  // the top-k_j of head j are the first k_j of its top-kmax
  tp.logits = c->at<float>(L.dlogits[0]); tp.M = H * B; tp.V = cf.vocab; tp.k = kmax;
  tp.tok = c->at<int>(L.m_tok); tp.logp = c->at<float>(L.m_logp);
  tp.scratch = c->at<float>(L.topk_scratch);
  HE(launch_topk(tp, c->st));
  MedusaExpandParams mx{};
  mx.seq_ids = ids; mx.nbatch = B; mx.H = H; mx.kmax = kmax;
  for (int j = 0; j < H; ++j) mx.topk[j] = cf.topk[j];
  mx.tok = c->at<int>(L.m_tok); mx.logp = c->at<float>(L.m_logp);
  mx.cand_token = ct; mx.cand_parent = cpar; mx.cand_depth = cd; mx.cand_lp = clp; mx.cand_stride = L.NC;
  {
    ProfScope ps(c, CLOVER_KSTAT_OTHER, 0, 0);
    HE(launch_medusa_expand(mx, c->st));
  }
  return enq_tree(c, B);
}

// Draft (Sec. 3): per depth, the regressive block on the frontier (the Attention Decoder,
// Eq. 1-2, or the MLP of the Sec. 4.3 ablation), head MLP, shared final norm + LM head,
// top-k children; then truncation into the verify tree.
hipError_t enq_draft(clover_ctx* c, int B) {
  if (is_medusa(c->cfg)) return enq_draft_medusa(c, B);
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  const int d = cf.d_model, qd = cf.n_heads * cf.head_dim, H = L.H;
  int* ids = c->at<int>(L.seq_ids);
  int *ct = c->at<int>(L.cand_token), *cpar = c->at<int>(L.cand_parent), *cd = c->at<int>(L.cand_depth);
  float* clp = c->at<float>(L.cand_lp);
  HE(launch_set_root(ids, B, c->at<int>(L.t0), ct, cpar, cd, clp, L.NC, c->st));
  for (int j = 1; j <= H; ++j) {
    const int F = frontier(cf, j), M = B * F;
    AdPrepParams ap{};
    ap.use_slot_state = (j == 1);
    ap.prev = (j == 1) ? c->at<float>(L.h0) : c->at<float>(L.dstate[j - 2]);
    ap.Fprev = (j == 1) ? 1 : frontier(cf, j - 1);
    ap.kprev = (j == 1) ? 1 : cf.topk[j - 2];
    ap.seq_ids = ids; ap.nbatch = B; ap.F = F;
    ap.cand_token = ct; ap.cand_stride = L.NC; ap.base_node = depth_base(cf, j - 1);
    ap.lm_packed = c->lm_head; ap.lm_nchunks = d / kc_of(cf.dtype);
    float* part = c->at<float>(L.gpart);
    if (mlp_regressive(cf)) {
      // MLP regressive block: one [M][2d] row per frontier node, RMSNorm_r(h) then e, so a
      // single GEMM with K = 2d applies W_r to the concatenation
      ap.ad_norm = c->rb_norm; ap.eps = cf.rms_eps; ap.d = d; ap.ld_out = 2 * d;
      ap.hin = c->at<float>(L.d_hin); ap.a_out = c->at<void>(L.d_a);
      ap.e_out = c->at<char>(L.d_a) + (size_t)d * L.es;
      HE(launch_ad_prep(cf.dtype, ap, c->st));
      GemmParams rg{};
      rg.X = c->at<void>(L.d_a); rg.ldx = 2 * d; rg.mode = EP_PARTIAL; rg.max_splits = GEMM_MAX_SPLITS; rg.part = part;
      int sr = 0;
      HE(run_gemm(c, rg, M, 2 * d, {{c->rb_w, d}}, &sr));
      RowFixParams rr{};  // s = h + SiLU(W_r [RMSNorm_r(h); e] + b_r): fp32 state and storage copy
      rr.M = M; rr.d = d; rr.part = part; rr.S = sr; rr.ldp = d;
      rr.resid = c->at<float>(L.d_hin); rr.ldr = d; rr.act = 1; rr.bias = c->rb_b;
      rr.out_f = c->at<float>(L.dstate[j - 1]); rr.ldo = d; rr.out_copy_s = c->at<void>(L.d_sst);
      HE(run_rowfix(c, rr));
    } else {
      const clover_ctx::AdPtrs& adw = c->ad[cf.ad_per_head ? j - 1 : 0];
      ap.ad_norm = adw.norm; ap.eps = cf.rms_eps; ap.d = d;
      // with the two-token key set the embeddings follow the normalised states in one [2M][d]
      // block, so one K|V GEMM projects both
      const bool two = cf.ad_keys == CLOVER_AD_KEYS_TWO;
      ap.hin = c->at<float>(L.d_hin); ap.a_out = c->at<void>(L.d_a);
      ap.e_out = two ? (void*)(c->at<char>(L.d_a) + (size_t)M * d * L.es) : c->at<void>(L.d_e);
      HE(launch_ad_prep(cf.dtype, ap, c->st));
      float* part2 = c->at<float>(L.gpart2);
      int sq = 0, skv = 0, so = 0;
      // With the single key (Eq. 1 read literally) the softmax weight is exactly 1, so the
      // decoder's output is W_V e: the Q and K projections cannot change it and are skipped.
      const bool values_only = cf.ad_keys == CLOVER_AD_KEYS_SINGLE;
      if (!values_only) {
        GemmParams q{};
        q.X = c->at<void>(L.d_a); q.ldx = d; q.mode = EP_PARTIAL; q.max_splits = GEMM_MAX_SPLITS; q.part = part;
        HE(run_gemm(c, q, M, d, {{adw.wq, qd}}, &sq));
      }
      GemmParams kv{};
      kv.X = two ? c->at<void>(L.d_a) : c->at<void>(L.d_e); kv.ldx = d; kv.mode = EP_PARTIAL;
      kv.max_splits = GEMM_MAX_SPLITS; kv.part = part2;
      if (values_only)
        HE(run_gemm(c, kv, M, d, {{adw.wv, qd}}, &skv));
      else
        HE(run_gemm(c, kv, two ? 2 * M : M, d, {{adw.wk, qd}, {adw.wv, qd}}, &skv));
      AdAttnParams aa{};
      aa.q = part; aa.Sq = sq; aa.kv = part2; aa.Skv = skv; aa.values_only = values_only;
      aa.M = M; aa.F = F; aa.n_heads = cf.n_heads; aa.hd = cf.head_dim;
      aa.keys = cf.ad_keys; aa.depth = j - 1; aa.out = c->at<void>(L.d_o);
      if (cf.ad_keys == CLOVER_AD_KEYS_PATH) {
        // key/value rows of every depth's nodes, depth after depth; an ancestor at depth dd of
        // a depth-(j-1) node fl has index fl / (k_dd * ... * k_{j-2}) among its depth's nodes
        aa.kv_path = c->at<float>(L.d_kvpath);
        int off = 0;
        for (int dd = 0; dd < j; ++dd) {
          aa.kv_path_off[dd] = off;
          aa.path_nodes[dd] = frontier(cf, dd + 1);
          off += B * frontier(cf, dd + 1);
          int div = 1;
          for (int t = dd; t < j - 1; ++t) div *= cf.topk[t];
          aa.anc_div[dd] = div;
        }
      }
      HE(launch_ad_attn(cf.dtype, aa, c->st));
      GemmParams o{};
      o.X = c->at<void>(L.d_o); o.ldx = qd; o.mode = EP_PARTIAL; o.max_splits = GEMM_MAX_SPLITS; o.part = part;
      HE(run_gemm(c, o, M, qd, {{adw.wo, d}}, &so));
      RowFixParams rs{};  // s = h + W_O attn (Eq. 2): fp32 state and storage copy for the MLP
      rs.M = M; rs.d = d; rs.part = part; rs.S = so; rs.ldp = d;
      rs.resid = c->at<float>(L.d_hin); rs.ldr = d;
      rs.out_f = c->at<float>(L.dstate[j - 1]); rs.ldo = d; rs.out_copy_s = c->at<void>(L.d_sst);
      HE(run_rowfix(c, rs));
    }
    int sh = 0;
    GemmParams hm{};
    hm.X = c->at<void>(L.d_sst); hm.ldx = d; hm.mode = EP_PARTIAL; hm.max_splits = GEMM_MAX_SPLITS; hm.part = part;
    HE(run_gemm(c, hm, M, d, {{c->head_w1[j - 1], d}}, &sh));
    RowFixParams rh{};  // r = s + SiLU(W1 s + b1), then the shared final norm
    rh.M = M; rh.d = d; rh.part = part; rh.S = sh; rh.ldp = d;
    rh.resid = c->at<float>(L.dstate[j - 1]); rh.ldr = d; rh.act = 1; rh.bias = c->head_b1[j - 1];
    rh.out_f = c->at<float>(L.d_r); rh.ldo = d;
    rh.gain = c->final_norm; rh.eps = cf.rms_eps; rh.out_norm = c->at<void>(L.d_rn); rh.ldn = d;
    HE(run_rowfix(c, rh));
    GemmParams lm{};
    lm.X = c->at<void>(L.d_rn); lm.ldx = d; lm.mode = EP_PARTIAL; lm.max_splits = 1;
    lm.part = c->at<float>(L.dlogits[j - 1]);
    HE(run_gemm(c, lm, M, d, {{c->lm_head, cf.vocab}}));
    TopkParams tp{};
    tp.logits = c->at<float>(L.dlogits[j - 1]); tp.M = M; tp.V = cf.vocab; tp.k = cf.topk[j - 1];
    tp.seq_ids = ids; tp.F = F;
    tp.cand_token = ct; tp.cand_parent = cpar; tp.cand_depth = cd; tp.cand_lp = clp; tp.cand_stride = L.NC;
    tp.base_parent = depth_base(cf, j - 1); tp.base_child = depth_base(cf, j); tp.depth = j;
    tp.scratch = c->at<float>(L.topk_scratch);
    HE(launch_topk(tp, c->st));
  }
  return enq_tree(c, B);
}

// Truncation of every listed sequence's candidates into its verify tree and verify rows.
hipError_t enq_tree(clover_ctx* c, int B) {
  const Layout& L = c->L;
  TreeParams tr{};
  tr.seq_ids = c->at<int>(L.seq_ids); tr.nbatch = B;
  tr.cand_token = c->at<int>(L.cand_token); tr.cand_parent = c->at<int>(L.cand_parent);
  tr.cand_depth = c->at<int>(L.cand_depth); tr.cand_lp = c->at<float>(L.cand_lp);
  tr.cand_stride = L.NC; tr.n_cand = L.NC; tr.T = L.T; tr.mask_words = L.W;
  tr.seq_len = c->at<int>(L.seq_len);
  tr.tree_token = c->at<int>(L.tree_token); tr.tree_parent = c->at<int>(L.tree_parent);
  tr.tree_depth = c->at<int>(L.tree_depth); tr.tree_pos = c->at<int>(L.tree_pos);
  tr.tree_mask = c->at<uint64_t>(L.tree_mask);
  tr.row_tok = c->at<int>(L.row_tok); tr.row_pos = c->at<int>(L.row_pos);
  tr.row_slot = c->at<int>(L.row_slot); tr.row_seq = c->at<int>(L.row_seq);
  HE(launch_tree_build(tr, c->st));
  return hipSuccess;
}

clover_status check_ctx(clover_ctx* c) {
  if (!c) {
    set_global_err("context is null");
    return CLOVER_ERR_INVALID_ARG;
  }
  if (c->dead) return ctx_fail(c, CLOVER_ERR_DEVICE, "context unusable after a device error");
  return CLOVER_OK;
}

// upload batch ids and committed lengths; make KV room for L + T
clover_status begin_batch(clover_ctx* c, const int32_t* seqs, int B, int& max_keys) {
  const Layout& L = c->L;
  c->host_ids.assign(seqs, seqs + B);
  max_keys = 0;
  for (int b = 0; b < B; ++b) {
    const int s = seqs[b];
    clover_status st = ensure_blocks(c, s, c->seq_len[s] + L.T);
    if (st != CLOVER_OK) return st;
    max_keys = std::max(max_keys, c->seq_len[s] + L.T);
  }
  // pinned staging: the previous step has completed (finish_step waited for it), so the
  // buffers are free to overwrite
  for (int b = 0; b < B; ++b) c->pin_ids[b] = seqs[b];
  for (int i = 0; i < c->cfg.max_batch; ++i) c->pin_len[i] = std::max(c->seq_len[i], 0);
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.seq_ids), c->pin_ids, sizeof(int) * B, hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.seq_len), c->pin_len, sizeof(int) * c->cfg.max_batch,
                          hipMemcpyHostToDevice, c->st));
  return CLOVER_OK;
}

clover_status check_seqs(clover_ctx* c, const int32_t* seqs, int n) {
  if (!seqs || n < 1 || n > c->cfg.max_batch) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "bad sequence list");
  for (int i = 0; i < n; ++i) {
    const int s = seqs[i];
    if (s < 0 || s >= c->cfg.max_batch) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "sequence %d out of range", s);
    for (int j = 0; j < i; ++j)
      if (seqs[j] == s) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "sequence %d listed twice", s);
    if (c->seq_len[s] < 0) return ctx_fail(c, CLOVER_ERR_STATE, "sequence %d is not active", s);
    if (c->seq_len[s] + c->L.T > c->cfg.max_context)
      return ctx_fail(c, CLOVER_ERR_CAPACITY, "sequence %d would exceed max_context", s);
  }
  return CLOVER_OK;
}

}  // namespace

extern "C" {

clover_status clover_check_config(const clover_config* cfg) {
  std::string why;
  if (!check_config(cfg, why)) {
    set_global_err("invalid config: %s", why.c_str());
    return CLOVER_ERR_INVALID_ARG;
  }
  return CLOVER_OK;
}

size_t clover_weight_count(const clover_config* cfg) {
  if (clover_check_config(cfg) != CLOVER_OK) return 0;
  return weight_specs(*cfg).size();
}

int clover_weight_name(const clover_config* cfg, size_t i, char* buf, size_t buflen) {
  if (clover_check_config(cfg) != CLOVER_OK) return -1;
  auto s = weight_specs(*cfg);
  if (i >= s.size() || !buf || buflen == 0) return -1;
  snprintf(buf, buflen, "%s", s[i].name.c_str());
  return (int)s[i].name.size();
}

int clover_weight_shape(const clover_config* cfg, size_t i, int64_t out[2]) {
  if (clover_check_config(cfg) != CLOVER_OK) return -1;
  auto s = weight_specs(*cfg);
  if (i >= s.size() || !out) return -1;
  out[0] = s[i].rows;
  out[1] = s[i].cols;
  return s[i].cols ? 2 : 1;
}

size_t clover_packed_bytes(const clover_config* cfg, size_t i) {
  if (clover_check_config(cfg) != CLOVER_OK) return 0;
  auto s = weight_specs(*cfg);
  if (i >= s.size()) return 0;
  return (size_t)s[i].rows * std::max<int64_t>(s[i].cols, 1) * es_of(cfg->dtype);
}

size_t clover_workspace_bytes(const clover_config* cfg) {
  if (clover_check_config(cfg) != CLOVER_OK) return 0;
  return make_layout(*cfg).total;
}

clover_status clover_pack_weight(const clover_config* cfg, size_t i, const void* src, void* dst,
                                 void* hip_stream) {
  if (clover_check_config(cfg) != CLOVER_OK) return CLOVER_ERR_INVALID_ARG;
  auto s = weight_specs(*cfg);
  if (i >= s.size() || !src || !dst) {
    set_global_err("pack: bad index or null pointer");
    return CLOVER_ERR_INVALID_ARG;
  }
  hipStream_t st = (hipStream_t)hip_stream;
  hipError_t e;
  const std::string& nm = s[i].name;
  // Q/K projections of the target and Augmenting Block layers carry rotary (tile-local
  // rotary packing); the Attention Decoder's (ad.* or ad{j}.*) do not
  const bool decoder = nm.size() > 3 && nm.compare(0, 2, "ad") == 0 &&
                       (nm[2] == '.' || (nm[2] >= '0' && nm[2] <= '9'));
  const bool qk = !decoder && nm.size() > 3 &&
                  (nm.compare(nm.size() - 3, 3, ".wq") == 0 || nm.compare(nm.size() - 3, 3, ".wk") == 0);
  if (s[i].matrix)
    e = launch_pack(cfg->dtype, src, (int)s[i].rows, (int)s[i].cols, dst, qk ? cfg->head_dim : 0, st);
  else
    e = hipMemcpyAsync(dst, src, clover_packed_bytes(cfg, i), hipMemcpyDeviceToDevice, st);
  if (e != hipSuccess) {
    set_global_err("pack: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

const char* clover_last_error(const clover_ctx* ctx) { return ctx ? ctx->err.c_str() : g_err.c_str(); }

clover_status clover_init(const clover_config* cfg, void* const* weights, void* workspace,
                          size_t ws_bytes, void* hip_stream, clover_ctx** out) {
  if (!out) {
    set_global_err("out is null");
    return CLOVER_ERR_INVALID_ARG;
  }
  *out = nullptr;
  if (clover_check_config(cfg) != CLOVER_OK) return CLOVER_ERR_INVALID_ARG;
  if (!weights || !workspace) {
    set_global_err("weights or workspace is null");
    return CLOVER_ERR_INVALID_ARG;
  }
  auto specs = weight_specs(*cfg);
  for (size_t i = 0; i < specs.size(); ++i)
    if (!weights[i]) {
      set_global_err("weight %zu (%s) is null", i, specs[i].name.c_str());
      return CLOVER_ERR_INVALID_ARG;
    }
  Layout L = make_layout(*cfg);
  if (ws_bytes < L.total) {
    set_global_err("workspace too small: %zu < %zu bytes", ws_bytes, L.total);
    return CLOVER_ERR_CAPACITY;
  }
  clover_ctx* c = new clover_ctx();
  c->cfg = *cfg;
  c->L = L;
  c->st = (hipStream_t)hip_stream;
  c->ws = (char*)workspace;
  c->w.assign(weights, weights + specs.size());
  size_t k = 0;
  c->emb = c->w[k++];
  auto take_layer = [&]() {
    LayerPtrs p;
    p.attn_norm = c->w[k++]; p.wq = c->w[k++]; p.wk = c->w[k++]; p.wv = c->w[k++]; p.wo = c->w[k++];
    p.mlp_norm = c->w[k++]; p.wg = c->w[k++]; p.wu = c->w[k++]; p.wd = c->w[k++];
    return p;
  };
  for (int l = 0; l < cfg->n_layers; ++l) c->layers.push_back(take_layer());
  c->final_norm = c->w[k++];
  c->lm_head = c->w[k++];
  if (has_ab(*cfg)) {  // the Augmenting Block's halves in weight-list order
    LayerPtrs p{};
    if (ab_attn(*cfg)) { p.attn_norm = c->w[k++]; p.wq = c->w[k++]; p.wk = c->w[k++]; p.wv = c->w[k++]; p.wo = c->w[k++]; }
    if (ab_mlp(*cfg)) { p.mlp_norm = c->w[k++]; p.wg = c->w[k++]; p.wu = c->w[k++]; p.wd = c->w[k++]; }
    c->layers.push_back(p);
  }
  if (mlp_regressive(*cfg)) {
    c->rb_norm = c->w[k++]; c->rb_w = c->w[k++]; c->rb_b = c->w[k++];
  } else if (!is_medusa(*cfg)) {
    for (int j = 0; j < (cfg->ad_per_head ? cfg->n_spec_heads : 1); ++j) {
      clover_ctx::AdPtrs a;
      a.norm = c->w[k++]; a.wq = c->w[k++]; a.wk = c->w[k++]; a.wv = c->w[k++]; a.wo = c->w[k++];
      c->ad.push_back(a);
    }
  }
  for (int j = 0; j < cfg->n_spec_heads; ++j) {
    c->head_w1.push_back(c->w[k++]);
    c->head_b1.push_back(c->w[k++]);
    if (per_head_lm(*cfg)) c->head_lm.push_back(c->w[k++]);
  }
  c->profile = (cfg->flags & CLOVER_FLAG_PROFILE) != 0;
  c->use_graphs = !c->profile && !(cfg->flags & CLOVER_FLAG_EAGER);
  c->graphs.resize(cfg->max_batch + 1);
  c->seq_len.assign(cfg->max_batch, -1);
  c->seq_blocks.assign(cfg->max_batch, {});
  for (int b = L.nblocks - 1; b >= 0; --b) c->free_blocks.push_back(b);
  auto fail = [&](hipError_t e, const char* what) {
    set_global_err("init: %s: %s", what, hipGetErrorString(e));
    clover_destroy(c);  // releases whatever was created so far
    return CLOVER_ERR_DEVICE;
  };
  hipError_t e;
  for (int i = 0; i < 4; ++i)
    if ((e = hipEventCreate(&c->ev[i])) != hipSuccess) return fail(e, "event");
  if ((e = hipStreamCreateWithFlags(&c->cap_st, hipStreamNonBlocking)) != hipSuccess) return fail(e, "capture stream");
  const size_t H1 = (size_t)c->L.H + 1;
  if ((e = hipHostMalloc((void**)&c->pin_ids, sizeof(int) * cfg->max_batch, hipHostMallocDefault)) != hipSuccess ||
      (e = hipHostMalloc((void**)&c->pin_len, sizeof(int) * cfg->max_batch, hipHostMallocDefault)) != hipSuccess ||
      (e = hipHostMalloc((void**)&c->pin_out, sizeof(int) * cfg->max_batch * H1, hipHostMallocDefault)) != hipSuccess ||
      (e = hipHostMalloc((void**)&c->bt_host, sizeof(int) * (size_t)cfg->max_batch * L.mbps, hipHostMallocDefault)) != hipSuccess)
    return fail(e, "pinned staging");
  std::memset(c->bt_host, 0, sizeof(int) * (size_t)cfg->max_batch * L.mbps);
  // zero the KV pools (attention reads whole 16-key blocks), counters and state
  if ((e = hipMemsetAsync(c->ws, 0, L.pool_ptrs, c->st)) != hipSuccess) return fail(e, "memset pools");
  if ((e = hipMemsetAsync(c->ws + L.block_table, 0, L.x - L.block_table, c->st)) != hipSuccess) return fail(e, "memset state");
  const int NL = kv_layers(*cfg);
  std::vector<void*> pools(2 * NL);
  for (int l = 0; l < NL; ++l) {
    pools[l] = c->ws + L.kpool + L.pool_bytes * l;
    pools[NL + l] = c->ws + L.vpool + L.pool_bytes * l;
  }
  if ((e = hipMemcpyAsync(c->ws + L.pool_ptrs, pools.data(), sizeof(void*) * pools.size(),
                          hipMemcpyHostToDevice, c->st)) != hipSuccess)
    return fail(e, "pool table");
  if ((e = hipStreamSynchronize(c->st)) != hipSuccess) return fail(e, "sync");
  *out = c;
  return CLOVER_OK;
}

void clover_destroy(clover_ctx* ctx) {
  if (!ctx) return;
  (void)hipStreamSynchronize(ctx->st);
  for (int i = 0; i < 4; ++i)
    if (ctx->ev[i]) (void)hipEventDestroy(ctx->ev[i]);
  for (auto e : ctx->pev) (void)hipEventDestroy(e);
  for (auto& g : ctx->graphs)
    for (hipGraphExec_t x : {g.draft, g.verify, g.accept})
      if (x) (void)hipGraphExecDestroy(x);
  if (ctx->cap_st) (void)hipStreamDestroy(ctx->cap_st);
  for (int* p : {ctx->pin_ids, ctx->pin_len, ctx->pin_out, ctx->bt_host})
    if (p) (void)hipHostFree(p);
  delete ctx;
}

int32_t clover_seq_len(const clover_ctx* ctx, int32_t seq) {
  if (!ctx || seq < 0 || seq >= ctx->cfg.max_batch) return -1;
  return ctx->seq_len[seq];
}

clover_status clover_release(clover_ctx* c, int32_t seq) {
  clover_status s = check_ctx(c);
  if (s) return s;
  if (seq < 0 || seq >= c->cfg.max_batch) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "sequence out of range");
  if (c->seq_len[seq] < 0) return ctx_fail(c, CLOVER_ERR_STATE, "sequence %d is not active", seq);
  for (int b : c->seq_blocks[seq]) c->free_blocks.push_back(b);
  c->seq_blocks[seq].clear();
  c->seq_len[seq] = -1;
  return CLOVER_OK;
}

clover_status clover_prefill(clover_ctx* c, int32_t seq, const int32_t* tokens, int32_t n,
                             int32_t* first_token) {
  clover_status s = check_ctx(c);
  if (s) return s;
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  if (seq < 0 || seq >= cf.max_batch) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "sequence %d out of range", seq);
  if (!tokens || n < 1 || !first_token) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "bad prompt");
  if (c->seq_len[seq] >= 0) return ctx_fail(c, CLOVER_ERR_STATE, "sequence %d is already active", seq);
  if ((int64_t)n + L.T > cf.max_context) return ctx_fail(c, CLOVER_ERR_CAPACITY, "prompt of %d tokens exceeds max_context", n);
  for (int i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= cf.vocab) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "token %d out of range", tokens[i]);
  if (c->trace && (size_t)(cf.n_layers + 2) * std::min(n, L.Mp) * cf.d_model * 4 > c->trace_bytes)
    return ctx_fail(c, CLOVER_ERR_CAPACITY, "trace buffer too small for a %d-row prefill chunk", std::min(n, L.Mp));
  if ((s = ensure_blocks(c, seq, n + L.T))) return s;
  const int d = cf.d_model, C = L.Mp;
  float* x = c->at<float>(L.x);
  float* xa = c->at<float>(L.xa);
  std::vector<int> meta(4 * (size_t)C);
  c->host_ids.assign(1, seq);
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.seq_ids), c->host_ids.data(), sizeof(int), hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemsetAsync(c->at<int>(L.sample_step) + seq, 0, sizeof(int), c->st));  // a new sequence's draws
  for (int c0 = 0; c0 < n; c0 += C) {
    const int rows = std::min(C, n - c0);
    for (int i = 0; i < rows; ++i) {
      meta[i] = tokens[c0 + i];
      meta[C + i] = c0 + i;      // position
      meta[2 * C + i] = c0 + i;  // slot
      meta[3 * C + i] = seq;
    }
    HIPCK(c, hipMemcpyAsync(c->at<int>(L.row_tok), meta.data(), sizeof(int) * rows, hipMemcpyHostToDevice, c->st));
    HIPCK(c, hipMemcpyAsync(c->at<int>(L.row_pos), meta.data() + C, sizeof(int) * rows, hipMemcpyHostToDevice, c->st));
    HIPCK(c, hipMemcpyAsync(c->at<int>(L.row_slot), meta.data() + 2 * C, sizeof(int) * rows, hipMemcpyHostToDevice, c->st));
    HIPCK(c, hipMemcpyAsync(c->at<int>(L.row_seq), meta.data() + 3 * C, sizeof(int) * rows, hipMemcpyHostToDevice, c->st));
    HIPCK(c, launch_embed(cf.dtype, c->emb, c->at<int>(L.row_tok), rows, d, x, c->st));
    HIPCK(c, row_tables(c, rows));
    AttnParams att{};
    att.seq_ids = c->at<int>(L.seq_ids);
    att.prefix_dev = nullptr; att.prefix_host = c0;
    att.rows_per_seq = rows; att.nq = rows; att.n_tail = rows; att.causal = 1;
    att.nbatch = 1;
    att.part = c->at<float>(L.apart); att.part_cap = L.apart_floats;
    int pend = 0;
    for (int l = 0; l < cf.n_layers; ++l)
      HIPCK(c, run_layer(c, c->layers[l], l, x, rows, att, c0 + rows, pend, &pend));
    RowFixParams rf{};
    rf.M = rows; rf.d = d; rf.part = c->at<float>(L.gpart); rf.S = pend; rf.ldp = d;
    rf.resid = x; rf.ldr = d; rf.out_f = x; rf.ldo = d; rf.out_copy_f = xa;
    rf.gain = c->final_norm; rf.eps = cf.rms_eps; rf.out_norm = c->at<void>(L.xn); rf.ldn = d;
    HIPCK(c, run_rowfix(c, rf));
    HIPCK(c, trace_rows(c, cf.n_layers, x, rows));
    if (c0 + rows == n) {
      GemmParams lm{};
      lm.X = (const char*)c->at<char>(L.xn) + (size_t)(rows - 1) * d * L.es; lm.ldx = d;
      lm.mode = EP_PARTIAL; lm.max_splits = 1;
      lm.part = keep_logits(c) ? c->at<float>(L.vlogits) : nullptr;
      lm.amax_part = c->at<unsigned long long>(L.amax_part);
      set_sampling(c, lm, 1, c->at<int>(L.seq_ids), 1);  // the first token: row 0 is sequence seq
      int lm_groups = 0;
      HIPCK(c, run_gemm(c, lm, 1, d, {{c->lm_head, cf.vocab}}, nullptr, &lm_groups));
      HIPCK(c, launch_argmax_groups(c->at<unsigned long long>(L.amax_part), lm_groups, 1, c->at<int>(L.amax), c->st));
    }
    if (has_ab(cf)) {  // Augmenting Block over the chunk; without it xa keeps x_N
      HIPCK(c, run_layer(c, c->layers[cf.n_layers], cf.n_layers, xa, rows, att, c0 + rows, 0, &pend,
                         ab_attn(cf), ab_mlp(cf)));
      RowFixParams ra{};
      ra.M = rows; ra.d = d; ra.part = c->at<float>(L.gpart); ra.S = pend; ra.ldp = d;
      ra.resid = xa; ra.ldr = d; ra.out_f = xa; ra.ldo = d;
      HIPCK(c, run_rowfix(c, ra));
    }
    HIPCK(c, trace_rows(c, cf.n_layers + 1, xa, rows));
    if (c0 + rows == n)
      HIPCK(c, launch_finish_prefill(seq, c->at<int>(L.amax), xa + (size_t)(rows - 1) * d, d,
                                     c->at<int>(L.t0), c->at<float>(L.h0), c->st));
    HIPCK(c, hipStreamSynchronize(c->st));  // meta is reused by the next chunk
  }
  int t0 = -1;
  HIPCK(c, hipMemcpyAsync(&t0, c->at<int>(L.t0) + seq, sizeof(int), hipMemcpyDeviceToHost, c->st));
  HIPCK(c, hipStreamSynchronize(c->st));
  c->seq_len[seq] = n;
  *first_token = t0;
  return CLOVER_OK;
}

clover_status clover_step(clover_ctx* c, const int32_t* seqs, int32_t n_seqs, int32_t* out_tokens,
                          int32_t* out_count) {
  clover_status s = check_ctx(c);
  if (s) return s;
  if (!out_tokens || !out_count) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "null output");
  if ((s = check_seqs(c, seqs, n_seqs))) return s;
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  const int B = n_seqs, d = cf.d_model, qd = cf.n_heads * cf.head_dim, H = L.H;
  if (c->trace && (size_t)(cf.n_layers + 2) * B * L.T * d * 4 > c->trace_bytes)
    return ctx_fail(c, CLOVER_ERR_CAPACITY, "trace buffer too small for %d verify rows", B * L.T);
  int max_keys = 0;
  if ((s = begin_batch(c, seqs, B, max_keys))) return s;
  const bool graph = c->use_graphs && !c->trace;  // a traced step runs its launches eagerly
  HIPCK(c, hipEventRecord(c->ev[0], c->st));
  c->in_step = true;
  c->phase = CLOVER_KSTAT_GEMM_DRAFT;
  HIPCK(c, run_phase(c, &c->graphs[B].draft, graph, [&] { return enq_draft(c, B); }));
  HIPCK(c, hipEventRecord(c->ev[1], c->st));
  c->phase = CLOVER_KSTAT_GEMM_VERIFY;
  HIPCK(c, run_phase(c, &c->graphs[B].verify, graph, [&] { return enq_verify(c, B, max_keys); }));
  HIPCK(c, hipEventRecord(c->ev[2], c->st));
  HIPCK(c, run_phase(c, &c->graphs[B].accept, graph, [&] { return enq_accept(c, B, max_keys); }));
  c->last_nbatch = B;
  s = finish_step(c, B, out_tokens, out_count);
  c->in_step = false;
  return s;
}

clover_status clover_verify_tree(clover_ctx* c, int32_t seq, const int32_t* tokens,
                                 const int32_t* parents, int32_t T, int32_t* out_tokens,
                                 int32_t* out_count) {
  clover_status s = check_ctx(c);
  if (s) return s;
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  if (!tokens || !parents || !out_tokens || !out_count) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "null argument");
  if ((s = check_seqs(c, &seq, 1))) return s;
  if (T < 1 || T > L.T) return ctx_fail(c, CLOVER_ERR_BAD_TREE, "tree of %d tokens (max %d)", T, L.T);
  if (parents[0] != -1) return ctx_fail(c, CLOVER_ERR_BAD_TREE, "parents[0] must be -1");
  if (c->trace && (size_t)(cf.n_layers + 2) * L.T * cf.d_model * 4 > c->trace_bytes)
    return ctx_fail(c, CLOVER_ERR_CAPACITY, "trace buffer too small for %d verify rows", L.T);
  std::vector<int> depth(L.T, 0), tok(L.T, 0), par(L.T, -1);
  for (int i = 0; i < T; ++i) {
    if (tokens[i] < 0 || tokens[i] >= cf.vocab) return ctx_fail(c, CLOVER_ERR_BAD_TREE, "token %d out of range", tokens[i]);
    if (i > 0 && (parents[i] < 0 || parents[i] >= i)) return ctx_fail(c, CLOVER_ERR_BAD_TREE, "parents[%d] = %d", i, parents[i]);
    tok[i] = tokens[i];
    par[i] = parents[i];
    if (i > 0) depth[i] = depth[parents[i]] + 1;
    if (depth[i] > L.H) return ctx_fail(c, CLOVER_ERR_BAD_TREE, "tree deeper than %d", L.H);
  }
  // Pad to the configured size: padding nodes have parent -2, which no accepted node
  // index equals, and see only themselves (plus the committed prefix) in attention.
  for (int i = T; i < L.T; ++i) {
    tok[i] = tokens[0];
    par[i] = -2;
    depth[i] = 1;
  }
  int max_keys = 0;
  if ((s = begin_batch(c, &seq, 1, max_keys))) return s;
  const int Ln = c->seq_len[seq];
  // tree arrays and verify rows for slot `seq`
  std::vector<int> meta(8 * (size_t)L.T);
  std::vector<uint64_t> mask((size_t)L.T * L.W, 0);
  for (int i = 0; i < L.T; ++i) {
    if (i < T)
      for (int j = i; j >= 0; j = par[j]) mask[(size_t)i * L.W + j / 64] |= 1ull << (j % 64);
    else
      mask[(size_t)i * L.W + i / 64] |= 1ull << (i % 64);
    meta[i] = tok[i];
    meta[L.T + i] = par[i];
    meta[2 * L.T + i] = depth[i];
    meta[3 * L.T + i] = Ln + depth[i];
    meta[4 * L.T + i] = tok[i];          // row_tok
    meta[5 * L.T + i] = Ln + depth[i];   // row_pos
    meta[6 * L.T + i] = Ln + i;          // row_slot
    meta[7 * L.T + i] = seq;             // row_seq
  }
  const size_t tb = (size_t)seq * L.T;
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.tree_token) + tb, meta.data(), 4 * L.T, hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.tree_parent) + tb, meta.data() + L.T, 4 * L.T, hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.tree_depth) + tb, meta.data() + 2 * L.T, 4 * L.T, hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.tree_pos) + tb, meta.data() + 3 * L.T, 4 * L.T, hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemcpyAsync(c->at<uint64_t>(L.tree_mask) + tb * L.W, mask.data(), 8 * mask.size(), hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.row_tok), meta.data() + 4 * L.T, 4 * L.T, hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.row_pos), meta.data() + 5 * L.T, 4 * L.T, hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.row_slot), meta.data() + 6 * L.T, 4 * L.T, hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipMemcpyAsync(c->at<int>(L.row_seq), meta.data() + 7 * L.T, 4 * L.T, hipMemcpyHostToDevice, c->st));
  HIPCK(c, hipEventRecord(c->ev[0], c->st));
  HIPCK(c, hipEventRecord(c->ev[1], c->st));
  c->last_nbatch = 1;
  c->in_step = true;
  c->phase = CLOVER_KSTAT_GEMM_VERIFY;
  HIPCK(c, enq_verify(c, 1, max_keys));
  HIPCK(c, hipEventRecord(c->ev[2], c->st));
  HIPCK(c, enq_accept(c, 1, max_keys));
  s = finish_step(c, 1, out_tokens, out_count);
  c->in_step = false;
  return s;
}

clover_status clover_debug_read(clover_ctx* c, const char* name, void* host_dst, size_t bytes,
                                size_t* written) {
  clover_status s = check_ctx(c);
  if (s) return s;
  if (!name || !host_dst) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "null argument");
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  const size_t B = cf.max_batch, T = L.T, NC = L.NC, H = L.H;
  struct Item { const char* n; size_t off, bytes; };
  std::vector<Item> items = {
      {"cand_token", L.cand_token, 4 * B * NC}, {"cand_parent", L.cand_parent, 4 * B * NC},
      {"cand_depth", L.cand_depth, 4 * B * NC}, {"cand_lp", L.cand_lp, 4 * B * NC},
      {"tree_token", L.tree_token, 4 * B * T}, {"tree_parent", L.tree_parent, 4 * B * T},
      {"tree_depth", L.tree_depth, 4 * B * T}, {"tree_pos", L.tree_pos, 4 * B * T},
      {"tree_mask", L.tree_mask, 8 * B * T * L.W}, {"target", L.target, 4 * B * T},
      {"acc", L.acc, 4 * B * (H + 1)}, {"acc_len", L.acc_len, 4 * B}, {"h0", L.h0, 4 * B * cf.d_model},
      {"t0", L.t0, 4 * B}, {"sample_step", L.sample_step, 4 * B},
      {"verify_logits", L.vlogits, 4 * B * T * (size_t)cf.vocab},
      {"x_last", L.x, 4 * B * T * (size_t)cf.d_model}, {"ab_out", L.xa, 4 * B * T * (size_t)cf.d_model}};
  std::vector<std::string> dn;
  for (int j = 1; j <= L.H; ++j) dn.push_back("draft_logits" + std::to_string(j));
  for (int j = 1; j <= L.H; ++j) {
    if (is_medusa(cf))  // head j's rows of the last step's batch
      items.push_back({dn[j - 1].c_str(), L.dlogits[0] + 4 * (size_t)(j - 1) * c->last_nbatch * cf.vocab,
                       4 * (size_t)c->last_nbatch * cf.vocab});
    else
      items.push_back({dn[j - 1].c_str(), L.dlogits[j - 1], 4 * B * frontier(cf, j) * (size_t)cf.vocab});
  }
  for (auto& it : items) {
    if (strcmp(it.n, name)) continue;
    const size_t n = std::min(bytes, it.bytes);
    HIPCK(c, hipStreamSynchronize(c->st));
    HIPCK(c, hipMemcpy(host_dst, c->ws + it.off, n, hipMemcpyDeviceToHost));
    if (written) *written = n;
    return CLOVER_OK;
  }
  return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "unknown debug buffer '%s'", name);
}

clover_status clover_debug_kv(clover_ctx* c, int32_t seq, int32_t layer, int32_t pos, int32_t which_v,
                              float* host_out) {
  clover_status s = check_ctx(c);
  if (s) return s;
  const clover_config& cf = c->cfg;
  const Layout& L = c->L;
  if (seq < 0 || seq >= cf.max_batch || layer < 0 || layer >= kv_layers(cf) || !host_out)
    return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "bad argument");
  if (pos < 0 || pos >= (int)c->seq_blocks[seq].size() * 16) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "position not allocated");
  const int hd = cf.head_dim, nkv = cf.n_kv_heads, EPL = 16 / L.es, KC = 4 * EPL;
  const int blk = c->seq_blocks[seq][pos / 16], key = pos % 16;
  std::vector<char> buf((size_t)nkv * 16 * hd * L.es);
  const size_t off = (which_v ? L.vpool : L.kpool) + L.pool_bytes * layer + (size_t)blk * nkv * 16 * hd * L.es;
  HIPCK(c, hipStreamSynchronize(c->st));
  HIPCK(c, hipMemcpy(buf.data(), c->ws + off, buf.size(), hipMemcpyDeviceToHost));
  for (int h = 0; h < nkv; ++h)
    for (int dd = 0; dd < hd; ++dd) {
      int idx;
      if (!which_v) {
        const int cc = dd / KC, q = dd % KC;
        idx = (cc * 64 + key + 16 * (q / EPL)) * EPL + (q % EPL);
      } else {
        idx = (((dd >> 4) * 4 + (key >> 2)) * 16 + (dd & 15)) * 4 + (key & 3);
      }
      const size_t e = (size_t)h * 16 * hd + idx;
      float v;
      if (L.es == 2) {
        uint32_t u = (uint32_t)(*(uint16_t*)(buf.data() + 2 * e)) << 16;
        memcpy(&v, &u, 4);
      } else {
        memcpy(&v, buf.data() + 4 * e, 4);
      }
      host_out[h * hd + dd] = v;
    }
  return CLOVER_OK;
}

clover_status clover_debug_trace(clover_ctx* c, float* dev_buf, size_t bytes) {
  clover_status s = check_ctx(c);
  if (s) return s;
  if (dev_buf && bytes < (size_t)(c->cfg.n_layers + 2) * c->cfg.d_model * 4)
    return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "trace buffer smaller than one row per slot");
  c->trace = dev_buf;
  c->trace_bytes = dev_buf ? bytes : 0;
  return CLOVER_OK;
}

clover_status clover_get_timings(clover_ctx* c, clover_timings* out) {
  clover_status s = check_ctx(c);
  if (s) return s;
  if (!out) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "null output");
  *out = c->tim;
  return CLOVER_OK;
}

clover_status clover_kernel_stats_get(clover_ctx* c, int32_t kind, clover_kernel_stats* out) {
  clover_status s = check_ctx(c);
  if (s) return s;
  if (!out || kind < 0 || kind >= CLOVER_KSTAT_COUNT) return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "bad kernel class");
  *out = c->kst[kind];
  return CLOVER_OK;
}

clover_status clover_set_flags(clover_ctx* c, int32_t flags) {
  clover_status s = check_ctx(c);
  if (s) return s;
  if (flags & ~(CLOVER_FLAG_KEEP_LOGITS | CLOVER_FLAG_PROFILE | CLOVER_FLAG_EAGER | CLOVER_FLAG_AB_COMMIT))
    return ctx_fail(c, CLOVER_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
  if ((flags ^ c->cfg.flags) & (CLOVER_FLAG_KEEP_LOGITS | CLOVER_FLAG_AB_COMMIT)) {
    // the captured phases bake in whether the LM head stores its logits and where the
    // Augmenting Block runs
    (void)hipStreamSynchronize(c->st);
    for (auto& g : c->graphs)
      for (hipGraphExec_t* x : {&g.draft, &g.verify, &g.accept})
        if (*x) {
          (void)hipGraphExecDestroy(*x);
          *x = nullptr;
        }
  }
  c->cfg.flags = flags;
  c->profile = (flags & CLOVER_FLAG_PROFILE) != 0;
  c->use_graphs = !c->profile && !(flags & CLOVER_FLAG_EAGER);
  return CLOVER_OK;
}

clover_status clover_kernel_stats_reset(clover_ctx* c) {
  clover_status s = check_ctx(c);
  if (s) return s;
  for (auto& k : c->kst) k = clover_kernel_stats{};
  return CLOVER_OK;
}

// ---- single-kernel entry points --------------------------------------------------------

// N <= 8192: split-K partials reduced by the row kernel (the path residual GEMMs take);
// wider outputs: one unsplit launch (the LM-head path)
static int op_linear_splits(int N) { return N <= 8192 ? GEMM_MAX_SPLITS : 1; }

size_t clover_op_scratch_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K) {
  if ((dtype != 0 && dtype != 1) || M < 1 || N < 16 || N % 16 || K < 1 || K % kc_of(dtype)) return 0;
  GemmPlan pl = plan_gemm(dtype, M, N / 16, K / kc_of(dtype), false, op_linear_splits(N));
  return align_up(4 * pl.part_floats) + ALIGN;
}

size_t clover_packed_matrix_bytes(int32_t dtype, int32_t rows, int32_t cols) {
  if ((dtype != 0 && dtype != 1) || rows < 16 || rows % 16 || cols < 1 || cols % kc_of(dtype)) return 0;
  return packed_matrix_bytes(dtype, rows, cols);
}

clover_status clover_pack_matrix(int32_t dtype, const void* src, int32_t rows, int32_t cols, void* dst,
                                 void* hip_stream) {
  if (!clover_packed_matrix_bytes(dtype, rows, cols) || !src || !dst) {
    set_global_err("pack_matrix: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  hipError_t e = launch_pack(dtype, src, rows, cols, dst, 0, (hipStream_t)hip_stream);
  if (e != hipSuccess) {
    set_global_err("pack_matrix: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

clover_status clover_op_linear(int32_t dtype, const void* X, int32_t M, int32_t K, const void* Wp,
                               int32_t N, float* Y, void* scratch, size_t scratch_bytes,
                               void* hip_stream) {
  const size_t need = clover_op_scratch_bytes(dtype, M, N, K);
  if (!need || !X || !Wp || !Y || !scratch) {
    set_global_err("op_linear: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  if (scratch_bytes < need) {
    set_global_err("op_linear: scratch %zu < %zu bytes", scratch_bytes, need);
    return CLOVER_ERR_CAPACITY;
  }
  hipStream_t st = (hipStream_t)hip_stream;
  GemmParams p{};
  p.X = X; p.ldx = K; p.M = M; p.K = K; p.nchunks = K / kc_of(dtype);
  p.seg[0] = GemmSeg{Wp, N / 16}; p.nseg = 1; p.ntiles = N / 16; p.N = N;
  p.mode = EP_PARTIAL;
  p.max_splits = op_linear_splits(N);
  p.part = p.max_splits == 1 ? Y : (float*)scratch;
  hipError_t e = launch_gemm(dtype, p, st);
  if (e == hipSuccess && p.max_splits > 1) {
    RowFixParams rf{};
    rf.M = M; rf.d = N; rf.part = (float*)scratch; rf.S = p.S; rf.ldp = N;
    rf.out_f = Y; rf.ldo = N;
    e = launch_rowfix(dtype, rf, st);
  }
  if (e != hipSuccess) {
    set_global_err("op_linear: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

clover_status clover_op_swiglu(int32_t dtype, const void* X, int32_t M, int32_t K, const void* Wg_p,
                               const void* Wu_p, int32_t F, void* act, void* hip_stream) {
  // the sizes a model's ffn_dim and d_model may take (clover_config)
  const int fq = dtype == 1 ? 32 : 16;
  if ((dtype != 0 && dtype != 1) || M < 1 || K < 1 || K % kc_of(dtype) || F < fq || F % fq || !X || !Wg_p ||
      !Wu_p || !act) {
    set_global_err("op_swiglu: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  GemmParams p{};
  p.X = X; p.ldx = K; p.M = M; p.K = K; p.nchunks = K / kc_of(dtype);
  p.seg[0] = GemmSeg{Wg_p, F / 16}; p.seg[1] = GemmSeg{Wu_p, F / 16}; p.nseg = 2; p.ntiles = 2 * (F / 16);
  p.N = F; p.mode = EP_SWIGLU; p.out_s = act; p.ldos = F;
  const hipError_t e = launch_gemm(dtype, p, (hipStream_t)hip_stream);
  if (e != hipSuccess) {
    set_global_err("op_swiglu: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

size_t clover_op_attention_scratch_bytes(int32_t dtype, int32_t L, int32_t T, int32_t n_heads,
                                         int32_t n_kv, int32_t head_dim) {
  if ((dtype != 0 && dtype != 1) || L < 0 || T < 1 || L + T > 65536 || n_heads < 1 || n_kv < 1 || n_heads % n_kv ||
      (head_dim != 32 && head_dim != 64 && head_dim != 128))
    return 0;
  const int nblocks = (L + T + 15) / 16;
  AttnParams a{};
  a.nbatch = 1; a.nq = T; a.n_heads = n_heads; a.n_kv = n_kv; a.hd = head_dim;
  size_t b = 0;
  b += align_up(4 * attention_part_floats(a));                                 // split partials
  b += align_up((size_t)nblocks * n_kv * 16 * head_dim * es_of(dtype)) * 2;  // K and V pools
  b += align_up(4 * (size_t)nblocks);                                          // block table
  b += align_up(8 * (size_t)T * ((T + 63) / 64));                              // mask
  b += align_up(4 * 2);                                                        // seq id
  return b;
}

clover_status clover_op_attention(int32_t dtype, const void* Q, const void* Kpre, const void* Vpre,
                                  const void* Ktree, const void* Vtree, int32_t L, int32_t T,
                                  const int32_t* parents, int32_t causal, int32_t n_heads,
                                  int32_t n_kv, int32_t head_dim, void* O, void* scratch,
                                  size_t scratch_bytes, void* hip_stream) {
  const size_t need = clover_op_attention_scratch_bytes(dtype, L, T, n_heads, n_kv, head_dim);
  if (!need || !Q || !Ktree || !Vtree || !O || !scratch || (L > 0 && (!Kpre || !Vpre)) ||
      (!causal && (!parents || T > 128))) {
    set_global_err("op_attention: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  if (scratch_bytes < need) {
    set_global_err("op_attention: scratch too small");
    return CLOVER_ERR_CAPACITY;
  }
  hipStream_t st = (hipStream_t)hip_stream;
  const int nblocks = (L + T + 15) / 16, W = (T + 63) / 64;
  const int es = es_of(dtype);
  char* p = (char*)scratch;
  AttnParams a{};
  a.nbatch = 1; a.nq = T; a.n_heads = n_heads; a.n_kv = n_kv; a.hd = head_dim;
  a.part_cap = attention_part_floats(a);
  a.part = (float*)p; p += align_up(4 * a.part_cap);
  char* kp = p; p += align_up((size_t)nblocks * n_kv * 16 * head_dim * es);
  char* vp = p; p += align_up((size_t)nblocks * n_kv * 16 * head_dim * es);
  int* bt = (int*)p; p += align_up(4 * (size_t)nblocks);
  uint64_t* mask = (uint64_t*)p; p += align_up(8 * (size_t)T * W);
  int* ids = (int*)p; p += align_up(8);
  std::vector<int> hbt(nblocks);
  for (int i = 0; i < nblocks; ++i) hbt[i] = nblocks - 1 - i;  // reversed pages: exercises the table
  std::vector<uint64_t> hm((size_t)T * W, 0);
  if (!causal) {
    for (int i = 0; i < T; ++i) {
      if (i == 0 ? parents[0] != -1 : (parents[i] < 0 || parents[i] >= i)) {
        set_global_err("op_attention: malformed parents");
        return CLOVER_ERR_BAD_TREE;
      }
      for (int j = i; j >= 0; j = parents[j]) hm[(size_t)i * W + j / 64] |= 1ull << (j % 64);
    }
  }
  int zero = 0;
  hipError_t e = hipSuccess;
  if (!e) e = hipMemsetAsync(kp, 0, (size_t)nblocks * n_kv * 16 * head_dim * es, st);
  if (!e) e = hipMemsetAsync(vp, 0, (size_t)nblocks * n_kv * 16 * head_dim * es, st);
  if (!e) e = hipMemcpyAsync(bt, hbt.data(), 4 * nblocks, hipMemcpyHostToDevice, st);
  if (!e) e = hipMemcpyAsync(mask, hm.data(), 8 * hm.size(), hipMemcpyHostToDevice, st);
  if (!e) e = hipMemcpyAsync(ids, &zero, 4, hipMemcpyHostToDevice, st);
  if (!e && L > 0) e = launch_kv_write(dtype, Kpre, Vpre, L, 0, 0, kp, vp, bt, nblocks, n_kv, head_dim, st);
  if (!e) e = launch_kv_write(dtype, Ktree, Vtree, T, L, 0, kp, vp, bt, nblocks, n_kv, head_dim, st);
  a.Q = Q; a.ldq = n_heads * head_dim; a.O = O; a.ldo = n_heads * head_dim;
  a.kcache = kp; a.vcache = vp; a.block_table = bt; a.max_blocks = nblocks;
  a.seq_ids = ids; a.prefix_dev = nullptr; a.prefix_host = L;
  a.rows_per_seq = T; a.n_tail = T; a.causal = causal ? 1 : 0;
  a.mask = mask; a.mask_words = W; a.mask_seq_stride = T * W;
  a.n_kv = n_kv; a.hd = head_dim;
  if (!e) e = launch_attention(dtype, a, L + T, st);
  if (!e) e = hipStreamSynchronize(st);  // host staging vectors die with this call
  if (e != hipSuccess) {
    set_global_err("op_attention: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

clover_status clover_op_argmax(const float* logits, int32_t M, int32_t V, int32_t* out, void* scratch,
                               void* hip_stream) {
  if (!logits || !out || !scratch || M < 1 || V < 1) {
    set_global_err("op_argmax: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  hipError_t e = launch_argmax(logits, M, V, out, (unsigned long long*)scratch, false, (hipStream_t)hip_stream);
  if (e != hipSuccess) {
    set_global_err("op_argmax: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

size_t clover_op_topk_scratch_bytes(int32_t M, int32_t V, int32_t k) {
  if (M < 1 || V < 1 || k < 1 || k > 16 || V < k) return 0;
  return 4 * topk_scratch_floats(M, V, k);
}

clover_status clover_op_topk(const float* logits, int32_t M, int32_t V, int32_t k, int32_t* tok,
                             float* logp, void* scratch, void* hip_stream) {
  if (!logits || !tok || !logp || !scratch || !clover_op_topk_scratch_bytes(M, V, k)) {
    set_global_err("op_topk: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  TopkParams p{};
  p.logits = logits; p.M = M; p.V = V; p.k = k; p.tok = tok; p.logp = logp;
  p.scratch = (float*)scratch;
  hipError_t e = launch_topk(p, (hipStream_t)hip_stream);
  if (e != hipSuccess) {
    set_global_err("op_topk: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

clover_status clover_op_tree_build(const int32_t* cand_token, const int32_t* cand_parent,
                                   const int32_t* cand_depth, const float* cand_lp, int32_t n_cand,
                                   int32_t T, int32_t L, int32_t* tokens, int32_t* parent,
                                   int32_t* depth, int32_t* pos, uint64_t* mask, void* hip_stream) {
  if (!cand_token || !cand_parent || !cand_depth || !cand_lp || !tokens || !parent || !depth || !pos ||
      !mask || T < 1 || T > 128 || n_cand < T || n_cand > 1024 || L < 0) {
    set_global_err("op_tree_build: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  TreeParams p{};
  p.seq_ids = nullptr; p.nbatch = 1;
  p.cand_token = cand_token; p.cand_parent = cand_parent; p.cand_depth = cand_depth; p.cand_lp = cand_lp;
  p.cand_stride = n_cand; p.n_cand = n_cand; p.T = T; p.mask_words = (T + 63) / 64;
  p.seq_len = nullptr; p.seq_len_host = L;
  p.tree_token = tokens; p.tree_parent = parent; p.tree_depth = depth; p.tree_pos = pos; p.tree_mask = mask;
  hipError_t e = launch_tree_build(p, (hipStream_t)hip_stream);
  if (e != hipSuccess) {
    set_global_err("op_tree_build: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

clover_status clover_op_accept(const int32_t* tokens, const int32_t* parent, const int32_t* target,
                               int32_t T, int32_t max_depth, int32_t* acc, int32_t* acc_len,
                               int32_t* bonus, void* hip_stream) {
  if (!tokens || !parent || !target || !acc || !acc_len || !bonus || T < 1 || T > 1024 ||
      max_depth < 0 || max_depth > 15) {
    set_global_err("op_accept: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  AcceptParams p{};
  p.seq_ids = nullptr; p.nbatch = 1; p.T = T; p.H = max_depth;
  p.tree_token = tokens; p.tree_parent = parent; p.target = target;
  p.acc = acc; p.acc_len = acc_len; p.out_tokens = nullptr; p.t0 = bonus;
  p.ab_out = nullptr; p.d = 0; p.h0 = nullptr;
  hipError_t e = launch_accept(p, (hipStream_t)hip_stream);
  if (e != hipSuccess) {
    set_global_err("op_accept: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

clover_status clover_op_compact(int32_t dtype, void* kcache, void* vcache, int32_t n_layers, int32_t n_blocks,
                                int32_t n_kv, int32_t head_dim, const int32_t* block_table, int32_t n_table,
                                int32_t L, const int32_t* acc, int32_t A, void* scratch, size_t scratch_bytes,
                                void* hip_stream) {
  if ((dtype != CLOVER_F32 && dtype != CLOVER_BF16) || !kcache || !vcache || !block_table || !acc ||
      !scratch || n_layers < 1 || n_blocks < 1 || n_table < 1 || n_kv < 1 ||
      (head_dim != 32 && head_dim != 64 && head_dim != 128) || L < 0 || A < 1 || A > 9) {
    set_global_err("op_compact: bad arguments");
    return CLOVER_ERR_INVALID_ARG;
  }
  if (scratch_bytes < sizeof(int32_t) * (size_t)(n_table + A)) {
    set_global_err("op_compact: scratch needs 4 * (n_table + A) bytes");
    return CLOVER_ERR_CAPACITY;
  }
  for (int i = 0; i < n_table; ++i)
    if (block_table[i] < 0 || block_table[i] >= n_blocks) {
      set_global_err("op_compact: block_table[%d] = %d outside [0, %d)", i, block_table[i], n_blocks);
      return CLOVER_ERR_INVALID_ARG;
    }
  for (int k = 0; k < A; ++k)
    if (acc[k] < 0 || (int64_t)L + std::max(acc[k], k) >= (int64_t)n_table * 16) {
      set_global_err("op_compact: slot L + acc[%d] or L + %d outside the block table", k, k);
      return CLOVER_ERR_INVALID_ARG;
    }
  hipStream_t st = (hipStream_t)hip_stream;
  int32_t* dev = (int32_t*)scratch;  // [block table][acc]
  hipError_t e = hipMemcpyAsync(dev, block_table, sizeof(int32_t) * n_table, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipMemcpyAsync(dev + n_table, acc, sizeof(int32_t) * A, hipMemcpyHostToDevice, st);
  CompactParams cp{};
  cp.seq_ids = nullptr; cp.nbatch = 1; cp.H = A - 1;
  cp.acc = dev + n_table; cp.acc_len = nullptr; cp.seq_len = nullptr; cp.A_host = A; cp.L_host = L;
  cp.kpools = nullptr; cp.vpools = nullptr; cp.nlayers = n_layers;
  cp.kbase = kcache; cp.vbase = vcache; cp.layer_elems = (size_t)n_blocks * n_kv * 16 * head_dim;
  cp.block_table = dev; cp.max_blocks = n_table;
  cp.n_kv = n_kv; cp.hd = head_dim;
  if (e == hipSuccess) e = launch_compact(dtype, cp, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);  // the host arrays may go once this returns
  if (e != hipSuccess) {
    set_global_err("op_compact: %s", hipGetErrorString(e));
    return CLOVER_ERR_DEVICE;
  }
  return CLOVER_OK;
}

}  // extern "C"
