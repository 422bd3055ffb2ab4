// Host runtime of the drafting library: context, step-indexed weight arena,
// workspace, the per-pass launch sequence, and HIP-graph capture of the
// chain and the tree.  Implements include/prism_draft.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "prism_draft.h"
#include "internal.h"

using namespace prism;

namespace {

struct Set {
  bool loaded = false;
  int F = 0;
  TiledMat fc, qkv, o, gu, down;
  void *g1 = nullptr, *g2 = nullptr;
  void *arena = nullptr;
  // embedding half of the fusion FC for every token, W_fc[:, :H] E[v]
  // (fp32 [V, H]); valid once both this set and the shared tensors are loaded
  float *tab = nullptr;
  bool tab_ready = false;
};

struct Pass {            // one forward pass: where its inputs and outputs live
  int set, R, F, topk;
  int grp;                // > 1: attention over groups of grp rows of one sequence (tree levels)
  int rps;                // > 0 (with grp): rows in runs of rps rows of one tree (tree scoring)
  RowsIn in;
  TokFromLm lm_in;        // tokens from the previous pass's LM partials (pval != NULL)
  bool defer_merge;       // leave the LM partials to the next pass (chain, top-1)
  // stochastic drafting (u != NULL): draw from softmax(logits * inv_temp)
  const float *u; int ld_u;
  float inv_temp;
  float *logp_out; int ld_logp;
  float *hid_out; int ld_hid;
  float *logits; long ld_logits;
  int *ids; float *logp;
  int *tok_a; int *tok_b; int ld_b;
  // chain steps: this pass's FC takes its feature operand from the previous
  // pass's down product and its tokens in its own K-split kernel (no prep
  // pass); this pass's down product writes that operand for the next pass
  bool op_in, op_out;
  // tree scoring (lm_rows_x.hi != NULL): no LM head in the pass; its
  // operand rows and row scales go here, for the caller's LM head over them
  ActOut lm_rows_x;
  float *lm_rows_scale;
};

std::string g_create_error;

}  // namespace

void prism::set_global_error(const char *msg) { g_create_error = msg; }

struct prism_ctx {
  prism_config cfg{};
  bool bf16 = true;
  size_t esz = 2;
  int dev = 0;
  int H = 0, nq = 0, nkv = 0, d = 0, I = 0, V = 0, QKV = 0;
  int rows_max = 0, max_slots = 0, kmax = 1, n_wg_lm = 0, Cmax = 0;
  // rows of the largest pass: tree scoring (bf16) runs whole trees in passes
  // of up to LMR_MAX_ROWS rows (the row-group products and one LM head per
  // pass); other passes take at most rows_max
  int pass_max = 0;
  int score_grp = 1;                // tree scoring: rows per attention workgroup
  int feat_max = 0;
  // passes take the fusion FC's embedding half from a per-set table (bf16)
  bool use_tab = false;
  int32_t *tab_tok = nullptr;       // batched FC rows' tokens for the table term [R]

  void *embed = nullptr, *gf = nullptr, *shared_arena = nullptr;
  TiledMat lm;
  bool shared_loaded = false;
  std::vector<Set> sets;
  std::vector<int> fmap;

  // workspace
  void *ws = nullptr;
  ActOut xfc;                       // FC operand planes [R, H + feat_max]
  float *u = nullptr, *r1 = nullptr;  // residual stream rows [R, H]
  ActOut ug, r1g, hg;               // (x * gain) operand planes [R, H]
  ActOut lmr_x;                     // bf16: LM-head operand rows of a tree-scoring pass [LMR_MAX_ROWS, H]
  float *lmr_scale = nullptr;       // and their row scales
  float *ss_u = nullptr, *ss_r1 = nullptr, *ss_h = nullptr;  // [parts <= H/16][R]
  float *sc_u = nullptr, *sc_r1 = nullptr, *sc_h = nullptr;  // row scales [R]
  float *q = nullptr;               // [R, nq*d] fp32
  float *pm = nullptr, *pl = nullptr, *po = nullptr;         // attention partials
  ActOut o;                         // attention output planes [R, nq*d]
  ActOut z;                         // SwiGLU planes [R, I]
  float *hid[2] = {nullptr, nullptr};
  float *part = nullptr;            // batched products: K-slice partial sums
  float *lm_max = nullptr, *lm_sum = nullptr, *lm_val = nullptr, *logp = nullptr;
  int *lm_id = nullptr, *ids = nullptr, *tokbuf = nullptr;
  int32_t *c_seq = nullptr, *c_pos = nullptr, *c_tok0 = nullptr;
  int32_t *t_ctok = nullptr, *t_cpar = nullptr, *t_front = nullptr;
  float *t_fscore = nullptr;
  float *t_cscore = nullptr;
  int32_t *t_tok = nullptr, *t_frow = nullptr, *t_seq = nullptr, *t_pos = nullptr, *t_slot = nullptr;
  uint64_t *t_bits[2] = {nullptr, nullptr};
  int att_grp = 1;                  // tree levels: rows per attention workgroup
  int lm_nwg_last = 0;              // LM-head partial count of the pass last enqueued
  int new_max = 0;                  // catch-up rows capacity
  int front_max = 0;                // rows of one catch-up front chunk
  int32_t *c_rseq = nullptr, *c_rpos = nullptr, *c_last = nullptr;   // catch-up rows
  // tree scoring: the rows of every tree, [max_batch * (MAX_SCORE_NODES + 1)]
  int32_t *s_tok = nullptr, *s_seq = nullptr, *s_pos = nullptr, *s_slot = nullptr;
  uint64_t *s_bits = nullptr;
  int score_rows = 0;
  float *q2 = nullptr, *u2 = nullptr;   // q and u of each sequence's last accepted row
  float *samp_logits = nullptr;     // [rows, V] fp32 logits kept for the sampler
  void *vstats = nullptr;           // verification: per-slice statistics of logits rows
  int vrows_max = 0;
  size_t lds_limit = 65536;         // LDS bytes one workgroup may use
  uint32_t *err = nullptr;
  double *inv_freq = nullptr;

  hipStream_t cap = nullptr;
  bool use_graph = true;
  bool enq_bad = false;             // a product plan was refused while enqueueing
  // measurement: event pairs around LM-head launches
  bool profile = false;
  int prof_what = 0;        // PRISM_PROFILE_* bits
  std::vector<hipEvent_t> prof_ev;
  int prof_used = 0;        // pairs recorded by the enqueue in progress
  int prof_last = 0;        // pairs of the last chain/tree call
  // captured graphs by key, each with the call count of its last use
  struct Graph {
    hipGraphExec_t exec;
    uint64_t used;
  };
  std::map<std::vector<uintptr_t>, Graph> graphs;
  uint64_t graph_calls = 0;
  std::string msg;
};

// ------------------------------------------------------------------ helpers
static prism_status fail(prism_ctx *c, prism_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->msg = buf;
  else g_create_error = buf;
  return st;
}

#define HIPCHK(c, call)                                                                  \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail((c), PRISM_ERR_HIP, "%s failed: %s", #call, hipGetErrorString(e_));    \
  } while (0)

static TiledMat make_tiled(int N, int K, bool bf16) {
  TiledMat t;
  t.N = N;
  t.K = K;
  t.n_tiles = N / 16;
  t.nkb = K / (bf16 ? 32 : 16);
  return t;
}
static size_t tiled_bytes(const TiledMat &t) { return (size_t)t.n_tiles * t.nkb * 1024; }

static void carve(char *&p, void **dst, size_t bytes) {
  *dst = p;
  p += (bytes + 255) & ~(size_t)255;
}

// ------------------------------------------------------------------ C ABI
extern "C" {

const char *prism_last_error(const prism_ctx *ctx) {
  return ctx ? ctx->msg.c_str() : g_create_error.c_str();
}

prism_status prism_create(const prism_config *cfg, prism_ctx **out) {
  if (!out) return fail(nullptr, PRISM_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!cfg) return fail(nullptr, PRISM_ERR_INVALID_ARG, "cfg is NULL");
  const prism_config &k = *cfg;
  if (k.dtype != PRISM_F32 && k.dtype != PRISM_BF16)
    return fail(nullptr, PRISM_ERR_INVALID_ARG, "dtype %d", k.dtype);
  if (k.hidden <= 0 || k.n_q_heads <= 0 || k.n_kv_heads <= 0 || k.head_dim <= 0 || k.ffn <= 0 ||
      k.vocab <= 0 || k.n_sets <= 0 || k.max_steps <= 0 || k.feat_width <= 0 ||
      k.kv_block_size <= 0 || k.max_batch <= 0 || k.max_blocks_per_seq <= 0 || k.tree_width < 0 ||
      k.tree_nodes < 0 || !(k.rms_eps >= 0.f) || !(k.rope_theta > 0.f))
    return fail(nullptr, PRISM_ERR_INVALID_ARG, "non-positive size in config");
  const bool bf16 = k.dtype == PRISM_BF16;
  const int kq = bf16 ? 32 : 16;
  if (k.n_q_heads % k.n_kv_heads) return fail(nullptr, PRISM_ERR_SHAPE, "n_q_heads %% n_kv_heads != 0");
  if (k.n_q_heads / k.n_kv_heads > 8) return fail(nullptr, PRISM_ERR_SHAPE, "more than 8 query heads per KV head");
  if (k.head_dim < 32 || k.head_dim > 256 || (k.head_dim & (k.head_dim - 1)))
    return fail(nullptr, PRISM_ERR_SHAPE, "head_dim %d must be a power of two in 32..256", k.head_dim);
  if ((k.n_q_heads / k.n_kv_heads) * k.head_dim > 1024)
    return fail(nullptr, PRISM_ERR_SHAPE, "query heads per KV head x head_dim > 1024");
  if (k.hidden % kq || k.ffn % kq || (k.n_q_heads * k.head_dim) % kq || k.feat_width % kq)
    return fail(nullptr, PRISM_ERR_SHAPE, "H, I, n_q*d and F_t must be multiples of %d", kq);
  if (k.vocab % 16) return fail(nullptr, PRISM_ERR_SHAPE, "vocab must be a multiple of 16");
  if (k.hidden > 16384) return fail(nullptr, PRISM_ERR_SHAPE, "hidden > 16384");
  if (((k.n_q_heads + 2 * k.n_kv_heads) * k.head_dim + k.head_dim) > 16384)
    return fail(nullptr, PRISM_ERR_SHAPE, "q/k/v width too large");
  if (k.max_steps > 63) return fail(nullptr, PRISM_ERR_SHAPE, "max_steps > 63");
  if (k.max_new_rows < 0 || k.max_new_rows > MAX_NEW_ROWS)
    return fail(nullptr, PRISM_ERR_SHAPE, "max_new_rows %d out of 0..%d", k.max_new_rows,
                MAX_NEW_ROWS);
  const int w = k.tree_width;
  const int rows = k.max_batch * (w > 1 ? w : 1);
  if (rows > MAX_ROWS) return fail(nullptr, PRISM_ERR_SHAPE, "rows per pass %d > %d", rows, MAX_ROWS);
  int Cmax = 0;
  if (w > 0) {
    if (w > MAX_TOPK) return fail(nullptr, PRISM_ERR_SHAPE, "tree_width > %d", MAX_TOPK);
    Cmax = w + (k.max_steps - 1) * w * w;
    if (Cmax > MAX_TREE_CAND) return fail(nullptr, PRISM_ERR_SHAPE, "too many tree candidates");
    if (1 + (k.max_steps - 1) * w > 64) return fail(nullptr, PRISM_ERR_SHAPE, "tree uses more than 64 draft slots");
    if (k.tree_nodes < 1 || k.tree_nodes > 64)
      return fail(nullptr, PRISM_ERR_SHAPE, "tree_nodes must be in 1..64");
    if (w > k.vocab) return fail(nullptr, PRISM_ERR_SHAPE, "tree_width > vocab");
  }

  prism_ctx *c = new prism_ctx();
  c->cfg = k;
  c->bf16 = bf16;
  c->esz = bf16 ? 2 : 4;
  (void)hipGetDevice(&c->dev);
  {
    int lds = 0;
    if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, c->dev) == hipSuccess &&
        lds > 0)
      c->lds_limit = (size_t)lds;
  }
  c->H = k.hidden; c->nq = k.n_q_heads; c->nkv = k.n_kv_heads; c->d = k.head_dim;
  c->I = k.ffn; c->V = k.vocab; c->QKV = (c->nq + 2 * c->nkv) * c->d;
  c->rows_max = rows;
  c->max_slots = k.max_blocks_per_seq * k.kv_block_size;
  // attention partials: rows x chunks of the largest pass (chunks per pass
  // from its row count); tree levels group att_grp rows of one sequence
  c->att_grp = w > 1 ? attention_group(bf16, k.n_q_heads, k.n_kv_heads, k.head_dim, w) : 1;
  c->pass_max = bf16 && rows < LMR_MAX_ROWS ? LMR_MAX_ROWS : rows;
  c->score_grp = score_attention_group(bf16, k.n_q_heads, k.n_kv_heads, k.head_dim);
  int max_chunks = 0;
  const long part_rc = attention_partial_rows(c->pass_max, c->att_grp, c->score_grp, k.n_kv_heads,
                                              c->max_slots, max_chunks);
  if (max_chunks > ATT_MAX_CHUNKS) {
    delete c;
    return fail(nullptr, PRISM_ERR_SHAPE, "KV capacity per sequence too large for the attention merge");
  }
  c->kmax = w > 1 ? w : 1;
  c->Cmax = Cmax;
  c->feat_max = k.feat_width > k.hidden ? k.feat_width : k.hidden;
  c->use_tab = bf16 && k.hidden % 64 == 0;
  c->sets.resize(k.n_sets);
  c->fmap.resize(k.max_steps);
  for (int i = 0; i < k.max_steps; ++i) c->fmap[i] = i < k.n_sets ? i : k.n_sets - 1;
  c->lm = make_tiled(c->V, c->H, bf16);
  c->n_wg_lm = lm_workgroups(c->lm.n_tiles, 1);
  if (const char *e = getenv("PRISM_NO_GRAPH")) c->use_graph = !(e[0] == '1');

  // rows of a drafting pass (R), of any pass (RP: tree scoring), and of one
  // chunk of the fusion FC / QKV front of a catch-up step too (RF: the
  // accepted tokens, at most MAX_ROWS per chunk)
  const size_t R = rows, RP = c->pass_max, es = c->esz;
  const int front_rows = k.max_new_rows < MAX_ROWS ? k.max_new_rows : MAX_ROWS;
  const size_t RF = (int)RP > front_rows ? RP : front_rows;
  c->new_max = k.max_new_rows;
  c->front_max = (int)RF;
  size_t total = 0;
  std::vector<std::pair<void **, size_t>> L;
  auto add = [&](void **p, size_t b) { L.push_back({p, b}); total += (b + 255) & ~(size_t)255; };
  auto planes = [&](ActOut &a, size_t n) {   // hi (and lo for bf16) planes of n values
    add(&a.hi, n * es);
    if (bf16) add(&a.lo, n * es);
  };
  const size_t nth = (size_t)c->H / 16;
  planes(c->xfc, RF * (c->H + c->feat_max));
  add((void **)&c->u, RF * c->H * 4);
  add((void **)&c->r1, RP * c->H * 4);
  planes(c->ug, RF * c->H);
  planes(c->r1g, RP * c->H);
  planes(c->hg, RP * c->H);
  if (bf16) {
    planes(c->lmr_x, (size_t)LMR_MAX_ROWS * c->H);
    add((void **)&c->lmr_scale, LMR_MAX_ROWS * 4);
  }
  add((void **)&c->ss_u, nth * RF * 4);
  add((void **)&c->ss_r1, nth * RP * 4);
  add((void **)&c->ss_h, nth * RP * 4);
  add((void **)&c->sc_u, RF * 4);
  add((void **)&c->sc_r1, RP * 4);
  add((void **)&c->sc_h, RP * 4);
  add((void **)&c->q, RF * c->nq * c->d * 4);
  add((void **)&c->pm, part_rc * c->nq * 4);
  add((void **)&c->pl, part_rc * c->nq * 4);
  add((void **)&c->po, part_rc * c->nq * c->d * 4);
  planes(c->o, RP * c->nq * c->d);
  planes(c->z, RP * c->I);
  add((void **)&c->hid[0], RP * c->H * 4);
  add((void **)&c->hid[1], R * c->H * 4);
  if ((int)RF > GEMV_MAX_ROWS) {   // batched products: K-slice partial sums [split][rows][N]
    size_t pn = 0;
    auto upd = [&](int N, int K) {
      const TiledMat t = make_tiled(N, K, bf16);
      pn = std::max(pn, product_partial_floats(t.n_tiles, t.nkb, t.K, (int)RF));
    };
    upd(c->H, c->H + k.feat_width);
    upd(c->H, 2 * c->H);
    upd(c->QKV, c->H);
    upd(c->H, c->nq * c->d);
    upd(2 * c->I, c->H);
    upd(c->H, c->I);
    add((void **)&c->part, pn * 4);
  }
  add((void **)&c->lm_max, R * c->n_wg_lm * 4);
  add((void **)&c->lm_sum, R * c->n_wg_lm * 4);
  add((void **)&c->lm_val, R * c->n_wg_lm * c->kmax * 4);
  add((void **)&c->lm_id, R * c->n_wg_lm * c->kmax * 4);
  add((void **)&c->ids, R * c->kmax * 4);
  add((void **)&c->logp, R * c->kmax * 4);
  add((void **)&c->tokbuf, R * 4);
  add((void **)&c->tab_tok, RF * 4);
  add((void **)&c->samp_logits, R * c->V * 4);
  {   // verification rows: target and draft rows of a chain, or every node of a tree
    const int chain_rows = k.max_batch * (2 * k.max_steps + 1);
    const int tree_rows = k.max_batch * (MAX_VERIFY_NODES + 1);
    c->vrows_max = chain_rows > tree_rows ? chain_rows : tree_rows;
    add(&c->vstats, verify_stats_bytes(c->vrows_max));
  }
  add((void **)&c->c_seq, (size_t)k.max_batch * 4);
  add((void **)&c->c_pos, (size_t)k.max_batch * k.max_steps * 4);
  add((void **)&c->c_tok0, (size_t)k.max_batch * 4);
  if (k.max_new_rows > 0) {   // catch-up: accepted rows and each sequence's last one
    add((void **)&c->c_rseq, (size_t)k.max_new_rows * 4);
    add((void **)&c->c_rpos, (size_t)k.max_new_rows * 4);
    add((void **)&c->c_last, (size_t)k.max_batch * 4);
    add((void **)&c->q2, (size_t)k.max_batch * c->nq * c->d * 4);
    add((void **)&c->u2, (size_t)k.max_batch * c->H * 4);
  }
  const size_t tb = (size_t)k.max_batch * (Cmax > 0 ? Cmax : 1);
  add((void **)&c->t_ctok, tb * 4);
  add((void **)&c->t_cpar, tb * 4);
  add((void **)&c->t_cscore, tb * 4);
  add((void **)&c->t_front, (size_t)k.max_batch * (k.max_steps > 1 ? k.max_steps - 1 : 1) * (w > 0 ? w : 1) * 4);
  add((void **)&c->t_fscore, (size_t)k.max_batch * (k.max_steps > 1 ? k.max_steps - 1 : 1) * (w > 0 ? w : 1) * 4);
  add((void **)&c->t_tok, R * 4);
  add((void **)&c->t_frow, R * 4);
  add((void **)&c->t_seq, R * 4);
  add((void **)&c->t_pos, R * 4);
  add((void **)&c->t_slot, R * 4);
  c->score_rows = k.max_batch * (MAX_SCORE_NODES + 1);
  add((void **)&c->s_tok, (size_t)c->score_rows * 4);
  add((void **)&c->s_seq, (size_t)c->score_rows * 4);
  add((void **)&c->s_pos, (size_t)c->score_rows * 4);
  add((void **)&c->s_slot, (size_t)c->score_rows * 4);
  add((void **)&c->s_bits, (size_t)c->score_rows * 8);
  add((void **)&c->t_bits[0], R * 8);
  add((void **)&c->t_bits[1], R * 8);
  add((void **)&c->err, 256);
  add((void **)&c->inv_freq, (size_t)(c->d / 2) * 8);

  if (hipMalloc(&c->ws, total) != hipSuccess) {
    delete c;
    return fail(nullptr, PRISM_ERR_OUT_OF_MEMORY, "workspace of %zu bytes", total);
  }
  char *p = (char *)c->ws;
  for (auto &e : L) carve(p, e.first, e.second);
  (void)hipMemset(c->ws, 0, total);
  std::vector<double> inv(c->d / 2);
  for (int i = 0; i < c->d / 2; ++i) inv[i] = std::pow((double)k.rope_theta, -2.0 * i / c->d);
  (void)hipMemcpy(c->inv_freq, inv.data(), inv.size() * 8, hipMemcpyHostToDevice);
  {   // the static verification scratch of this device, resolved at set-up
    void *vs = nullptr;
    const hipError_t e = verify_scratch(&vs);
    if (e != hipSuccess) {
      (void)hipFree(c->ws);
      delete c;
      return fail(nullptr, PRISM_ERR_HIP, "hipGetSymbolAddress: %s", hipGetErrorString(e));
    }
  }
  if (hipStreamCreateWithFlags(&c->cap, hipStreamNonBlocking) != hipSuccess) {
    (void)hipFree(c->ws);
    delete c;
    return fail(nullptr, PRISM_ERR_HIP, "stream creation failed");
  }
  *out = c;
  return PRISM_OK;
}

static void drop_graphs(prism_ctx *c) {
  if (!c->graphs.empty()) (void)hipDeviceSynchronize();   // none may still run
  for (auto &g : c->graphs) (void)hipGraphExecDestroy(g.second.exec);
  c->graphs.clear();
}

void prism_destroy(prism_ctx *c) {
  if (!c) return;
  (void)hipDeviceSynchronize();
  drop_graphs(c);
  for (auto &s : c->sets)
    if (s.arena) (void)hipFree(s.arena);
  if (c->shared_arena) (void)hipFree(c->shared_arena);
  if (c->ws) (void)hipFree(c->ws);
  if (c->cap) (void)hipStreamDestroy(c->cap);
  for (auto e : c->prof_ev) (void)hipEventDestroy(e);
  delete c;
}

prism_status prism_draft_load_shared(prism_ctx *c, const void *d_embed, const void *d_lm_head,
                                     const void *d_final_norm, void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (!d_embed || !d_lm_head || !d_final_norm)
    return fail(c, PRISM_ERR_INVALID_ARG, "NULL shared tensor");
  hipStream_t s = (hipStream_t)stream;
  drop_graphs(c);
  const size_t eb = (size_t)c->V * c->H * c->esz;
  if (!c->shared_arena) {
    const size_t bytes = ((eb + 255) & ~(size_t)255) + ((tiled_bytes(c->lm) + 255) & ~(size_t)255) +
                         (size_t)c->H * c->esz;
    if (hipMalloc(&c->shared_arena, bytes) != hipSuccess)
      return fail(c, PRISM_ERR_OUT_OF_MEMORY, "shared arena of %zu bytes", bytes);
    char *p = (char *)c->shared_arena;
    carve(p, &c->embed, eb);
    carve(p, &c->lm.w, tiled_bytes(c->lm));
    c->gf = p;
  }
  HIPCHK(c, hipMemcpyAsync(c->embed, d_embed, eb, hipMemcpyDeviceToDevice, s));
  launch_repack(c->bf16, d_lm_head, c->V, c->H, 1, 0, 0, c->d, c->lm, s);
  HIPCHK(c, hipGetLastError());
  HIPCHK(c, hipMemcpyAsync(c->gf, d_final_norm, (size_t)c->H * c->esz, hipMemcpyDeviceToDevice, s));
  for (auto &S : c->sets) {   // embedding tables of the sets already loaded
    if (!S.tab || !S.loaded) continue;
    launch_embed_table(S.fc, c->embed, c->V, c->H, S.tab, s);
    HIPCHK(c, hipGetLastError());
    S.tab_ready = true;
  }
  HIPCHK(c, hipStreamSynchronize(s));
  c->shared_loaded = true;
  return PRISM_OK;
}

prism_status prism_draft_load_params(prism_ctx *c, int32_t set, const prism_param_set *P,
                                     void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (!P) return fail(c, PRISM_ERR_INVALID_ARG, "params is NULL");
  if (set < 0 || set >= c->cfg.n_sets)
    return fail(c, PRISM_ERR_INVALID_ARG, "set %d out of range 0..%d", set, c->cfg.n_sets - 1);
  if (!P->d_w_fc || !P->d_g1 || !P->d_w_q || !P->d_w_k || !P->d_w_v || !P->d_w_o || !P->d_g2 ||
      !P->d_w_gate || !P->d_w_up || !P->d_w_down)
    return fail(c, PRISM_ERR_INVALID_ARG, "NULL weight tensor in set %d", set);
  const int kq = c->bf16 ? 32 : 16;
  if (P->feat_width <= 0 || P->feat_width % kq)
    return fail(c, PRISM_ERR_SHAPE, "feat_width %d must be a positive multiple of %d", P->feat_width, kq);
  if (P->feat_width != c->cfg.feat_width && P->feat_width != c->H)
    return fail(c, PRISM_ERR_SHAPE, "feat_width %d is neither F_t nor H", P->feat_width);
  hipStream_t s = (hipStream_t)stream;
  drop_graphs(c);
  Set &S = c->sets[set];
  const int H = c->H, F = P->feat_width;
  if (S.arena && S.F != F) {
    (void)hipStreamSynchronize(s);
    (void)hipFree(S.arena);
    S.arena = nullptr;
  }
  if (!S.arena) {
    S.fc = make_tiled(H, H + F, c->bf16);
    S.qkv = make_tiled(c->QKV, H, c->bf16);
    S.o = make_tiled(H, c->nq * c->d, c->bf16);
    S.gu = make_tiled(2 * c->I, H, c->bf16);
    S.down = make_tiled(H, c->I, c->bf16);
    const size_t gb = (size_t)H * c->esz;
    const size_t tb = c->use_tab ? (size_t)c->V * H * 4 : 0;
    const size_t bytes = tiled_bytes(S.fc) + tiled_bytes(S.qkv) + tiled_bytes(S.o) +
                         tiled_bytes(S.gu) + tiled_bytes(S.down) + 2 * ((gb + 255) & ~(size_t)255) +
                         tb + 7 * 256;
    if (hipMalloc(&S.arena, bytes) != hipSuccess)
      return fail(c, PRISM_ERR_OUT_OF_MEMORY, "arena of set %d (%zu bytes)", set, bytes);
    char *p = (char *)S.arena;
    carve(p, &S.fc.w, tiled_bytes(S.fc));
    carve(p, &S.qkv.w, tiled_bytes(S.qkv));
    carve(p, &S.o.w, tiled_bytes(S.o));
    carve(p, &S.gu.w, tiled_bytes(S.gu));
    carve(p, &S.down.w, tiled_bytes(S.down));
    carve(p, &S.g1, gb);
    carve(p, &S.g2, gb);
    if (tb) carve(p, (void **)&S.tab, tb);
    S.F = F;
  }
  S.loaded = false;
  S.tab_ready = false;
  launch_repack(c->bf16, P->d_w_fc, H, H + F, 1, 0, 0, c->d, S.fc, s);
  // q, k, v rows stacked into one product; q and k heads pair-permuted for RoPE
  TiledMat qv = S.qkv;
  const int rot = (c->nq + c->nkv) * c->d;
  launch_repack(c->bf16, P->d_w_q, c->nq * c->d, H, 1, 0, rot, c->d, qv, s);
  launch_repack(c->bf16, P->d_w_k, c->nkv * c->d, H, 1, c->nq * c->d, rot, c->d, qv, s);
  launch_repack(c->bf16, P->d_w_v, c->nkv * c->d, H, 1, rot, rot, c->d, qv, s);
  launch_repack(c->bf16, P->d_w_o, H, c->nq * c->d, 1, 0, 0, c->d, S.o, s);
  // gate/up interleaved row by row: gate c -> 2c, up c -> 2c + 1
  launch_repack(c->bf16, P->d_w_gate, c->I, H, 2, 0, 0, c->d, S.gu, s);
  launch_repack(c->bf16, P->d_w_up, c->I, H, 2, 1, 0, c->d, S.gu, s);
  launch_repack(c->bf16, P->d_w_down, H, c->I, 1, 0, 0, c->d, S.down, s);
  HIPCHK(c, hipGetLastError());
  HIPCHK(c, hipMemcpyAsync(S.g1, P->d_g1, (size_t)H * c->esz, hipMemcpyDeviceToDevice, s));
  HIPCHK(c, hipMemcpyAsync(S.g2, P->d_g2, (size_t)H * c->esz, hipMemcpyDeviceToDevice, s));
  if (S.tab && c->shared_loaded) {
    launch_embed_table(S.fc, c->embed, c->V, H, S.tab, s);
    HIPCHK(c, hipGetLastError());
  }
  HIPCHK(c, hipStreamSynchronize(s));
  S.loaded = true;
  S.tab_ready = S.tab && c->shared_loaded;
  return PRISM_OK;
}

prism_status prism_set_step_map(prism_ctx *c, const int32_t *f_map, int32_t K) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (!f_map) return fail(c, PRISM_ERR_INVALID_ARG, "f_map is NULL");
  if (K < 1 || K > c->cfg.max_steps) return fail(c, PRISM_ERR_INVALID_ARG, "K %d out of 1..%d", K, c->cfg.max_steps);
  for (int i = 0; i < K; ++i)
    if (f_map[i] < 0 || f_map[i] >= c->cfg.n_sets)
      return fail(c, PRISM_ERR_INVALID_ARG, "f_map[%d] = %d out of range", i, f_map[i]);
  drop_graphs(c);
  c->fmap.assign(f_map, f_map + K);
  return PRISM_OK;
}

}  // extern "C"

// ------------------------------------------------------------------ passes
static KvArgs kv_of(const prism_ctx *c, const prism_batch *b) {
  KvArgs kv;
  kv.k_pool = b->d_k_pool;
  kv.v_pool = b->d_v_pool;
  kv.block_table = b->d_block_table;
  kv.ctx_lens = b->d_ctx_lens;
  kv.mbps = c->cfg.max_blocks_per_seq;
  kv.bs = c->cfg.kv_block_size;
  kv.n_blocks = b->n_pool_blocks;
  kv.n_seq = b->batch;
  return kv;
}

static Act act_of(const ActOut &o, int ld) {
  Act a;
  a.hi = o.hi;
  a.lo = o.lo;
  a.ld = ld;
  return a;
}

// RMSNorm row scales for a consumer: reduced by the consumer itself from the
// producer's n_parts partials per row when it can hold them all (own), else
// by a small kernel first.
static RowNorm norm_for(prism_ctx *c, const float *ss, int n_parts, bool own, float *scale, int R,
                        hipStream_t s) {
  RowNorm n;
  n.n_parts = n_parts;
  n.n = c->H;
  n.eps = c->cfg.rms_eps;
  if (own) {
    n.ss = ss;
  } else {
    launch_rowscale(R, ss, n_parts, c->H, n.eps, scale, s);
    n.scale = scale;
  }
  return n;
}

// kb_lo: the product covers k-blocks [kb_lo, nkb) of m (the fusion FC's
// feature columns when its embedding half comes from the table)
static GemmLaunch gemm_of(const prism_ctx *c, const TiledMat &m, const Act &x, int R, int epi,
                          int kb_lo = 0) {
  GemmLaunch g{};
  g.m = m;
  g.x = x;
  g.R = R;
  g.epi = epi;
  g.kb_lo = kb_lo;
  const int nkb = m.nkb - kb_lo, K = m.K - kb_lo * (c->bf16 ? 32 : 16);
  const ProductPlan pl =
      plan_product(m.n_tiles, nkb, K, m.K, R, epi == EPI_QKV, c->bf16, c->lds_limit);
  g.kw = pl.kw;
  g.nt = pl.nt;
  g.split = pl.split;
  g.gemv = pl.gemv;
  g.rowgrp = pl.rowgrp;
  if (R > GEMV_MAX_ROWS) g.part = c->part;
  return g;
}

// measurement: an event pair around the next launches of class `what`
// (-1: not profiled, or no event pair left)
static int prof_begin(prism_ctx *c, int what, hipStream_t s) {
  if (!c->profile || !(c->prof_what & what) || 2 * c->prof_used + 1 >= (int)c->prof_ev.size())
    return -1;
  (void)hipEventRecord(c->prof_ev[2 * c->prof_used], s);
  return c->prof_used++;
}
static void prof_end(prism_ctx *c, int pair, hipStream_t s) {
  if (pair >= 0) (void)hipEventRecord(c->prof_ev[2 * pair + 1], s);
}

// launch a planned product; a plan the kernels cannot take fails the call
static void gemm_go(prism_ctx *c, const GemmLaunch &g, hipStream_t s) {
  const int pr = prof_begin(c, PRISM_PROFILE_PRODUCTS, s);
  if (!launch_gemm(c->bf16, g, s)) c->enq_bad = true;
  prof_end(c, pr, s);
}

// Front of a pass: fusion FC and QKV (RoPE, KV append) for p.R rows -> u
// and q in the workspace.
static void enqueue_front(prism_ctx *c, const Pass &p, const KvArgs &kv, hipStream_t s) {
  const Set &S = c->sets[p.set];
  const bool bf = c->bf16;
  const int R = p.R, H = c->H;
  // fusion FC: u = W_fc [E(x) ; f]  ->  u, (u * g1), sums of squares
  ActOut X = c->xfc;
  X.ld = H + p.F;
  // with the set's embedding table the product covers the feature columns
  // only, and its epilogue adds the table row of each row's token
  const int kb_lo = S.tab_ready ? H / (bf ? 32 : 16) : 0;
  GemmLaunch g = gemm_of(c, S.fc, act_of(X, H + p.F), R, EPI_NORM, kb_lo);
  if (S.tab_ready) g.tab = S.tab;
  if (g.gemv) {   // the GEMV stages [E(x) ; f] (or f) itself
    g.gx.embed = c->embed; g.gx.V = c->V; g.gx.H = H; g.gx.in = p.in; g.gx.lm = p.lm_in;
    g.err = c->err;
  } else if (p.op_in) {
    // the feature columns were written by the previous down product; the
    // K-split kernel resolves the tokens for its finish pass
    g.tab_tok = c->tab_tok;
    g.tok_out = c->tab_tok;
    g.gx.V = c->V; g.gx.in = p.in; g.gx.lm = p.lm_in;
    g.err = c->err;
  } else {
    if (S.tab_ready) g.tab_tok = c->tab_tok;
    launch_fc_prep(bf, R, p.in, p.lm_in, c->embed, c->V, H, p.F, X, c->err,
                   S.tab_ready ? c->tab_tok : nullptr, S.tab_ready, s);
  }
  g.y = c->u; g.ldy = H; g.gain = S.g1; g.g = c->ug; g.g.ld = H; g.ss = c->ss_u;
  gemm_go(c, g, s);
  const int parts_u = gemm_ss_parts(g);
  // q, k, v = W_qkv RMSNorm(u; g1);  RoPE;  k, v -> cache slot
  g = gemm_of(c, S.qkv, act_of(c->ug, H), R, EPI_QKV);
  g.norm = norm_for(c, c->ss_u, parts_u, gemm_own_scales(g, parts_u), c->sc_u, R, s);
  g.q = c->q; g.nq = c->nq; g.nkv = c->nkv; g.d = c->d;
  g.rows = p.in; g.kv = kv; g.inv_freq = c->inv_freq; g.err = c->err;
  gemm_go(c, g, s);
}

// Back of a pass, for p.R rows whose q and FC output u are given: attention,
// O, MLP, LM head (and the top-k merge unless deferred).
static void enqueue_back(prism_ctx *c, const Pass &p, const KvArgs &kv, const float *q,
                         const float *u, hipStream_t s) {
  const Set &S = c->sets[p.set];
  const bool bf = c->bf16;
  const int R = p.R, H = c->H;
  // attention over the visible slots -> o
  ActOut o = c->o;
  o.ld = c->nq * c->d;
  launch_attention(bf, R, c->nq, c->nkv, c->d, q, p.in, kv, c->max_slots, p.grp, p.rps, c->pm, c->pl,
                   c->po, o, c->err, s);
  // r1 = u + W_o o  ->  r1, (r1 * g2), sums of squares
  GemmLaunch g = gemm_of(c, S.o, act_of(o, c->nq * c->d), R, EPI_NORM);
  g.res = u; g.ldres = H; g.y = c->r1; g.ldy = H; g.gain = S.g2; g.g = c->r1g; g.g.ld = H;
  g.ss = c->ss_r1;
  gemm_go(c, g, s);
  const int parts_r1 = gemm_ss_parts(g);
  // z = SiLU(W_gate m) * (W_up m),  m = RMSNorm(r1; g2)
  g = gemm_of(c, S.gu, act_of(c->r1g, H), R, EPI_SWIGLU);
  g.norm = norm_for(c, c->ss_r1, parts_r1, gemm_own_scales(g, parts_r1), c->sc_r1, R, s);
  g.z = c->z; g.z.ld = c->I;
  gemm_go(c, g, s);
  // h = r1 + W_down z  ->  h (output), (h * g_final), sums of squares
  g = gemm_of(c, S.down, act_of(c->z, c->I), R, EPI_NORM);
  g.res = c->r1; g.ldres = H; g.y = p.hid_out; g.ldy = p.ld_hid; g.gain = c->gf;
  g.g = p.lm_rows_x.hi ? p.lm_rows_x : c->hg;
  g.g.ld = H; g.ss = c->ss_h;
  if (p.op_out) {   // h as the next pass's FC feature columns (X[:, H:2H])
    g.yx.hi = (bf16_t *)c->xfc.hi + H;
    g.yx.lo = (bf16_t *)c->xfc.lo + H;
    g.yx.ld = 2 * H;
  }
  gemm_go(c, g, s);
  const int parts_h = gemm_ss_parts(g);
  if (p.lm_rows_x.hi) {   // the caller runs the LM head over these rows
    launch_rowscale(R, c->ss_h, parts_h, H, c->cfg.rms_eps, p.lm_rows_scale, s);
    return;
  }
  // logits = LM_head RMSNorm(h; g_final)  ->  top-k partials
  LmLaunch lmg{};
  lmg.m = c->lm;
  lmg.x = act_of(c->hg, H);
  lmg.R = R;
  lmg.V = c->V;
  lmg.topk = p.topk;
  lmg.inv_temp = p.u ? p.inv_temp : 1.f;
  // the GEMV LM head streams whole batches of 16 k-blocks (H a multiple of 512)
  lmg.gemv = (c->bf16 && R <= LM_GEMV_MAX_ROWS && c->lm.nkb % 16 == 0 &&
              gemv_lds_bytes(R, H) + 64 * 1024 <= c->lds_limit) ? 1 : 0;
  lmg.nt = 1;
  // one row: four consecutive vocab tiles per wave when that still gives
  // about four waves per CU (longer weight streams, one round of workgroups)
  if (lmg.gemv && c->lm.n_tiles % 16 == 0 && c->lm.nkb % 16 == 0 && c->lm.n_tiles / 4 >= 1024)
    lmg.nt = 4;
  // batched rows: several vocab tiles per wave share B fragments; 8 up to
  // 32 rows (at 16 rows: 176 -> 166 us against 4 tiles, the B stream being
  // half as large per weight byte), 4 above
  if (!lmg.gemv && R > LM_GEMV_MAX_ROWS) {
    if (c->lm.n_tiles % 8 == 0) lmg.nt = 8;
    else if (c->lm.n_tiles % 4 == 0) lmg.nt = 4;
    else if (c->lm.n_tiles % 2 == 0) lmg.nt = 2;
  }
  lmg.n_wg = lm_workgroups(c->lm.n_tiles, lmg.nt);
  lmg.norm = norm_for(c, c->ss_h, parts_h, lm_own_scales(R, parts_h), c->sc_h, R, s);
  lmg.logits = p.logits;
  lmg.ld_logits = p.ld_logits;
  if (p.u && !lmg.logits) {   // the sampler reads the draw's group back from the logits
    lmg.logits = c->samp_logits;
    lmg.ld_logits = c->V;
  }
  lmg.pmax = c->lm_max; lmg.psum = c->lm_sum; lmg.pval = c->lm_val; lmg.pid = c->lm_id;
  // top-k > 1 on MFMA tiles (tree levels): the LM head stores the logits
  // and a separate pass reduces them to the partials
  const bool topk_pass = !p.u && !lmg.gemv && p.topk > 1 && p.topk <= TK_MAXK;
  if (topk_pass) {
    if (!lmg.logits) {
      lmg.logits = c->samp_logits;
      lmg.ld_logits = c->V;
    }
    lmg.no_part = 1;
  }
  const int pr = prof_begin(c, PRISM_PROFILE_LMHEAD, s);
  launch_lmhead(bf, lmg, s);
  prof_end(c, pr, s);
  if (topk_pass) {
    LmTopkArgs ta{};
    ta.logits = lmg.logits; ta.ld = lmg.ld_logits;
    ta.R = R; ta.V = c->V; ta.topk = p.topk; ta.n_wg = lm_topk_chunks(c->V);
    ta.inv_temp = 1.f;
    ta.pmax = c->lm_max; ta.psum = c->lm_sum; ta.pval = c->lm_val; ta.pid = c->lm_id;
    launch_lm_topk(ta, s);
    lmg.n_wg = ta.n_wg;
  }
  c->lm_nwg_last = lmg.n_wg;
  if (p.u) {
    LmSampleArgs sa{};
    sa.R = R; sa.n_wg = lmg.n_wg; sa.V = c->V; sa.group = 64 * lmg.nt;
    sa.inv_temp = p.inv_temp;
    sa.pmax = c->lm_max; sa.psum = c->lm_sum;
    sa.logits = lmg.logits; sa.ld_logits = lmg.ld_logits;
    sa.u = p.u; sa.ld_u = p.ld_u;
    sa.ids = p.ids; sa.logp = p.logp_out; sa.ld_logp = p.ld_logp;
    sa.tok_a = p.tok_a; sa.tok_b = p.tok_b; sa.ld_b = p.ld_b;
    sa.err = c->err;
    launch_lm_sample(sa, s);
  } else if (!p.defer_merge) {
    launch_lm_combine(R, lmg.n_wg, p.topk, c->V, c->lm_max, c->lm_sum, c->lm_val, c->lm_id, p.ids,
                      p.logp, p.tok_a, p.tok_b, p.ld_b, c->err, s);
  }
}

static void enqueue_pass(prism_ctx *c, const Pass &p, const KvArgs &kv, hipStream_t s) {
  const int pr = prof_begin(c, PRISM_PROFILE_PASSES, s);
  enqueue_front(c, p, kv, s);
  enqueue_back(c, p, kv, c->q, c->u, s);
  prof_end(c, pr, s);
}

static prism_status check_set(prism_ctx *c, int step, int want_F) {
  if (!c->shared_loaded) return fail(c, PRISM_ERR_NOT_LOADED, "shared tensors not loaded");
  if (step < 1 || step > (int)c->fmap.size())
    return fail(c, PRISM_ERR_INVALID_ARG, "step %d beyond the step map (%zu steps)", step, c->fmap.size());
  const int s = c->fmap[step - 1];
  if (!c->sets[s].loaded) return fail(c, PRISM_ERR_NOT_LOADED, "set %d (step %d) not loaded", s, step);
  if (want_F > 0 && c->sets[s].F != want_F)
    return fail(c, PRISM_ERR_UNSUPPORTED,
                "set %d serves step %d, which needs feature width %d, but was loaded with %d", s,
                step, want_F, c->sets[s].F);
  return PRISM_OK;
}

static prism_status check_batch(prism_ctx *c, const prism_batch *b) {
  if (!b) return fail(c, PRISM_ERR_INVALID_ARG, "batch is NULL");
  if (b->batch < 1 || b->batch > c->cfg.max_batch)
    return fail(c, PRISM_ERR_INVALID_ARG, "batch %d out of 1..%d", b->batch, c->cfg.max_batch);
  if (!b->d_tokens || !b->d_features || !b->d_ctx_lens || !b->d_k_pool || !b->d_v_pool ||
      !b->d_block_table)
    return fail(c, PRISM_ERR_INVALID_ARG, "NULL pointer in batch");
  if (b->n_pool_blocks < 1) return fail(c, PRISM_ERR_INVALID_ARG, "n_pool_blocks < 1");
  return PRISM_OK;
}

// Graphs kept per context.  Every distinct key (shape, buffers, step map)
// captures one; past this many the least recently used one is destroyed, so
// callers that pass fresh output buffers on every call do not grow the
// cache without bound.
constexpr size_t GRAPH_CACHE_MAX = 64;

// run `enqueue` directly or through a cached graph keyed by `key`
template <typename F>
static prism_status run_graph(prism_ctx *c, const std::vector<uintptr_t> &key, hipStream_t s,
                              F enqueue) {
  c->enq_bad = false;
  // profiled calls run eagerly: event pairs bracket each LM-head launch on `s`
  if (!c->use_graph || c->profile) {
    c->prof_used = 0;
    enqueue(s);
    c->prof_last = c->prof_used;
    if (c->enq_bad) return fail(c, PRISM_ERR_SHAPE, "a product plan exceeds its kernel's workgroup bound");
    HIPCHK(c, hipGetLastError());
    return PRISM_OK;
  }
  auto it = c->graphs.find(key);
  if (it == c->graphs.end()) {
    hipGraph_t graph;
    HIPCHK(c, hipStreamBeginCapture(c->cap, hipStreamCaptureModeThreadLocal));
    c->prof_used = 0;
    enqueue(c->cap);
    c->prof_last = c->prof_used;
    hipError_t le = hipGetLastError();
    hipError_t ee = hipStreamEndCapture(c->cap, &graph);
    if (ee == hipSuccess && (le != hipSuccess || c->enq_bad)) (void)hipGraphDestroy(graph);
    if (le != hipSuccess) return fail(c, PRISM_ERR_HIP, "launch during capture: %s", hipGetErrorString(le));
    if (ee != hipSuccess) return fail(c, PRISM_ERR_HIP, "hipStreamEndCapture: %s", hipGetErrorString(ee));
    if (c->enq_bad) return fail(c, PRISM_ERR_SHAPE, "a product plan exceeds its kernel's workgroup bound");
    hipGraphExec_t exec;
    hipError_t ie = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (ie != hipSuccess) return fail(c, PRISM_ERR_HIP, "hipGraphInstantiate: %s", hipGetErrorString(ie));
    if (c->graphs.size() >= GRAPH_CACHE_MAX) {
      auto lru = c->graphs.begin();
      for (auto g = c->graphs.begin(); g != c->graphs.end(); ++g)
        if (g->second.used < lru->second.used) lru = g;
      // it may still run on some stream of the caller's
      HIPCHK(c, hipDeviceSynchronize());
      (void)hipGraphExecDestroy(lru->second.exec);
      c->graphs.erase(lru);
    }
    it = c->graphs.emplace(key, prism_ctx::Graph{exec, 0}).first;
  }
  it->second.used = ++c->graph_calls;
  HIPCHK(c, hipGraphLaunch(it->second.exec, s));
  return PRISM_OK;
}

extern "C" {

prism_status prism_draft_step(prism_ctx *c, int32_t k, const prism_step_io *io, void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (!io) return fail(c, PRISM_ERR_INVALID_ARG, "io is NULL");
  prism_status st = check_set(c, k, 0);
  if (st) return st;
  if (io->rows < 1 || io->rows > c->rows_max)
    return fail(c, PRISM_ERR_INVALID_ARG, "rows %d out of 1..%d", io->rows, c->rows_max);
  if (io->topk < 1 || io->topk > c->kmax || io->topk > c->V)
    return fail(c, PRISM_ERR_INVALID_ARG, "topk %d out of 1..%d", io->topk, c->kmax);
  if (!io->d_tokens || !io->d_feat || !io->d_seq || !io->d_pos || !io->d_slot || !io->kv ||
      !io->d_topk_ids)
    return fail(c, PRISM_ERR_INVALID_ARG, "NULL pointer in step io");
  if (io->feat_dtype != PRISM_F32 && io->feat_dtype != PRISM_BF16)
    return fail(c, PRISM_ERR_INVALID_ARG, "feat_dtype %d", io->feat_dtype);
  const prism_batch *b = io->kv;
  if (!b->d_ctx_lens || !b->d_k_pool || !b->d_v_pool || !b->d_block_table || b->n_pool_blocks < 1 ||
      b->batch < 1)
    return fail(c, PRISM_ERR_INVALID_ARG, "incomplete KV description");
  hipStream_t s = (hipStream_t)stream;
  const int set = c->fmap[k - 1];
  Pass p{};
  p.set = set;
  p.R = io->rows;
  p.F = c->sets[set].F;
  p.topk = io->topk;
  p.in.tokens = io->d_tokens;
  p.in.feat = io->d_feat;
  p.in.feat_bf16 = io->feat_dtype == PRISM_BF16;
  p.in.feat_ld = p.F;
  p.in.feat_rows = io->d_feat_rows;
  p.in.seq = io->d_seq;
  p.in.pos = io->d_pos;
  p.in.slot = io->d_slot;
  p.in.bits = io->d_tree_bits;
  p.hid_out = io->d_hidden_out ? io->d_hidden_out : c->hid[0];
  p.ld_hid = c->H;
  p.logits = io->d_logits;
  p.ld_logits = c->V;
  p.ids = io->d_topk_ids;
  p.logp = io->d_topk_logp;
  c->enq_bad = false;
  c->prof_used = 0;
  enqueue_pass(c, p, kv_of(c, b), s);
  c->prof_last = c->prof_used;
  if (c->enq_bad) return fail(c, PRISM_ERR_SHAPE, "a product plan exceeds its kernel's workgroup bound");
  HIPCHK(c, hipGetLastError());
  return PRISM_OK;
}

// K greedy steps for B sequences.  Step 1 fuses each sequence's last
// accepted token with its target feature, or (cu != NULL) is the prefill over
// all accepted rows: the FC / QKV front runs on the T rows (writing their
// KV), then the back of the pass continues from each sequence's last row.
// Step k >= 2 takes its token from the previous LM head's partials.
// With uniforms u [B, K] the tokens are drawn from softmax(logits / T)
// (inv_temp = 1/T) and their log-probabilities go to d_out_logp.
static void enqueue_chain(prism_ctx *c, const prism_batch &b, const KvArgs &kv, int K,
                          const prism_catchup *cu, int32_t *d_out_tokens, float *d_out_logits,
                          float *d_out_hidden, hipStream_t s, const float *u = nullptr,
                          float inv_temp = 1.f, float *d_out_logp = nullptr) {
  const int B = b.batch, H = c->H, V = c->V;
  if (cu)
    launch_catchup_setup(B, cu->total_rows, K, cu->d_offsets, b.d_ctx_lens, c->c_rseq, c->c_rpos,
                         c->c_last, c->c_seq, c->c_pos, c->err, s);
  else
    launch_chain_setup(B, K, b.d_tokens, b.d_ctx_lens, c->c_seq, c->c_pos, c->c_tok0, s);
  // step k >= 2 skips the FC prep pass when its FC is a K-split product over
  // the feature columns (bf16, embedding table) with a workgroup per row
  auto direct = [&](int k) -> bool {
    if (k < 2 || k > K || !c->bf16 || B <= GEMV_MAX_ROWS) return false;
    const Set &S = c->sets[c->fmap[k - 1]];
    if (!S.tab_ready || S.F != H) return false;
    const GemmLaunch g = gemm_of(c, S.fc, Act{}, B, EPI_NORM, H / 32);
    return g.split > 0 && !g.gemv && (long)((S.fc.n_tiles / g.nt + 3) / 4) * g.split >= B;
  };
  const float *prev = nullptr;
  int ld_prev = 0;
  for (int k = 1; k <= K; ++k) {
    Pass p{};
    p.op_in = direct(k);
    p.op_out = direct(k + 1);
    p.set = c->fmap[k - 1];
    p.R = B;
    p.F = k == 1 ? c->cfg.feat_width : H;
    p.topk = 1;
    p.in.tokens = c->c_tok0;      // step 1; later steps take the previous LM partials
    if (u) {                      // drawn tokens: the sampler writes them for the next step
      if (k > 1) p.in.tokens = c->tokbuf;
      p.u = u + (k - 1); p.ld_u = K; p.inv_temp = inv_temp;
      p.logp_out = d_out_logp ? d_out_logp + (k - 1) : nullptr; p.ld_logp = K;
    } else if (k > 1) {
      p.lm_in.pval = c->lm_val; p.lm_in.pid = c->lm_id; p.lm_in.n_wg = c->lm_nwg_last;
      p.lm_in.rec = d_out_tokens + (k - 2); p.lm_in.ld_rec = K;
    }
    p.defer_merge = !u && k < K;
    p.in.feat = k == 1 ? b.d_features : (const void *)prev;
    p.in.feat_bf16 = k == 1 ? (int)c->bf16 : 0;
    p.in.feat_ld = k == 1 ? c->cfg.feat_width : ld_prev;
    p.in.feat_rows = nullptr;
    p.in.seq = c->c_seq;
    p.in.pos = c->c_pos + (size_t)(k - 1) * B;
    p.in.slot = p.in.pos;
    p.in.bits = nullptr;
    p.hid_out = d_out_hidden ? d_out_hidden + (size_t)(k - 1) * H : c->hid[k & 1];
    p.ld_hid = d_out_hidden ? K * H : H;
    p.logits = d_out_logits ? d_out_logits + (size_t)(k - 1) * V : nullptr;
    p.ld_logits = (long)K * V;
    p.ids = c->ids;
    p.logp = nullptr;
    p.tok_a = c->tokbuf;
    p.tok_b = d_out_tokens + (k - 1);
    p.ld_b = K;
    if (k == 1 && cu) {
      const int pr = prof_begin(c, PRISM_PROFILE_PASSES, s);
      // front over every accepted row, in chunks of at most front_max rows:
      // the front (FC, QKV, KV append) of one row depends on no other row,
      // and only each sequence's last row runs the attention, after every
      // chunk has written its KV; that row's q and u are kept as its chunk
      // passes
      const size_t fb = (size_t)c->cfg.feat_width * c->esz;
      for (int r0 = 0; r0 < cu->total_rows; r0 += c->front_max) {
        const int n = cu->total_rows - r0 < c->front_max ? cu->total_rows - r0 : c->front_max;
        Pass f = p;
        f.R = n;
        f.in.tokens = cu->d_tokens + r0;
        f.in.feat = (const char *)cu->d_features + (size_t)r0 * fb;
        f.in.feat_bf16 = (int)c->bf16;
        f.in.feat_ld = c->cfg.feat_width;
        f.in.seq = c->c_rseq + r0;
        f.in.pos = c->c_rpos + r0;
        f.in.slot = c->c_rpos + r0;
        enqueue_front(c, f, kv, s);
        RowsGather rg{};
        rg.idx = c->c_last;
        rg.r0 = r0;
        rg.n_src = n;
        rg.src[0] = c->q; rg.dst[0] = c->q2; rg.n[0] = c->nq * c->d;
        rg.src[1] = c->u; rg.dst[1] = c->u2; rg.n[1] = H;
        launch_rows_gather(B, rg, s);
      }
      enqueue_back(c, p, kv, c->q2, c->u2, s);
      prof_end(c, pr, s);
    } else {
      enqueue_pass(c, p, kv, s);
    }
    prev = p.hid_out;
    ld_prev = p.ld_hid;
  }
}

static prism_status check_chain(prism_ctx *c, const prism_batch *batch, int32_t K,
                                const int32_t *d_out_tokens) {
  prism_status st = check_batch(c, batch);
  if (st) return st;
  if (K < 1 || K > c->cfg.max_steps || K > (int)c->fmap.size())
    return fail(c, PRISM_ERR_INVALID_ARG, "K %d out of 1..%zu", K, c->fmap.size());
  if (!d_out_tokens) return fail(c, PRISM_ERR_INVALID_ARG, "d_out_tokens is NULL");
  for (int k = 1; k <= K; ++k)
    if ((st = check_set(c, k, k == 1 ? c->cfg.feat_width : c->H))) return st;
  return PRISM_OK;
}

static std::vector<uintptr_t> chain_key(prism_ctx *c, uintptr_t kind, const prism_batch &b, int K,
                                        int32_t *d_out_tokens, float *d_out_logits,
                                        float *d_out_hidden) {
  std::vector<uintptr_t> key = {kind, (uintptr_t)b.batch, (uintptr_t)K, (uintptr_t)b.d_tokens,
                                (uintptr_t)b.d_features, (uintptr_t)b.d_ctx_lens,
                                (uintptr_t)b.d_k_pool, (uintptr_t)b.d_v_pool,
                                (uintptr_t)b.d_block_table, (uintptr_t)b.n_pool_blocks,
                                (uintptr_t)d_out_tokens, (uintptr_t)d_out_logits,
                                (uintptr_t)d_out_hidden};
  for (int k = 0; k < K; ++k) key.push_back((uintptr_t)c->fmap[k]);
  return key;
}

prism_status prism_draft_chain(prism_ctx *c, const prism_batch *batch, int32_t K,
                               int32_t *d_out_tokens, float *d_out_logits, float *d_out_hidden,
                               void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  prism_status st = check_chain(c, batch, K, d_out_tokens);
  if (st) return st;
  const prism_batch b = *batch;
  const KvArgs kv = kv_of(c, &b);
  auto key = chain_key(c, 1, b, K, d_out_tokens, d_out_logits, d_out_hidden);
  return run_graph(c, key, (hipStream_t)stream, [&](hipStream_t s) {
    enqueue_chain(c, b, kv, K, nullptr, d_out_tokens, d_out_logits, d_out_hidden, s);
  });
}

prism_status prism_draft_chain_sample(prism_ctx *c, const prism_batch *batch, int32_t K,
                                      float temperature, const float *d_uniforms,
                                      int32_t *d_out_tokens, float *d_out_logp,
                                      float *d_out_logits, float *d_out_hidden, void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  prism_status st = check_chain(c, batch, K, d_out_tokens);
  if (st) return st;
  if (!(temperature > 0.f) || !std::isfinite(1.f / temperature))
    return fail(c, PRISM_ERR_INVALID_ARG, "temperature %g must be positive", (double)temperature);
  if (!d_uniforms) return fail(c, PRISM_ERR_INVALID_ARG, "d_uniforms is NULL");
  // the widest LM-head plan: one tile per wave (most partials), 8 tiles per
  // wave (largest groups)
  if (!lm_sample_fits(c->n_wg_lm, 64 * 8))
    return fail(c, PRISM_ERR_UNSUPPORTED, "vocabulary of %d ids is too large for the sampler", c->V);
  const prism_batch b = *batch;
  const KvArgs kv = kv_of(c, &b);
  const float inv_temp = 1.f / temperature;
  auto key = chain_key(c, 4, b, K, d_out_tokens, d_out_logits, d_out_hidden);
  uint32_t tb;
  std::memcpy(&tb, &inv_temp, 4);
  key.push_back((uintptr_t)tb);
  key.push_back((uintptr_t)d_uniforms);
  key.push_back((uintptr_t)d_out_logp);
  return run_graph(c, key, (hipStream_t)stream, [&](hipStream_t s) {
    enqueue_chain(c, b, kv, K, nullptr, d_out_tokens, d_out_logits, d_out_hidden, s, d_uniforms,
                  inv_temp, d_out_logp);
  });
}

prism_status prism_verify_chain(prism_ctx *c, int32_t batch, int32_t K, float temperature,
                                const float *d_target_logits, const float *d_draft_logits,
                                const int32_t *d_draft_tokens, const float *d_uniforms,
                                int32_t *d_n_accepted, int32_t *d_next_token, void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (batch < 1 || batch > c->cfg.max_batch)
    return fail(c, PRISM_ERR_INVALID_ARG, "batch %d out of 1..%d", batch, c->cfg.max_batch);
  if (K < 1 || K > c->cfg.max_steps)
    return fail(c, PRISM_ERR_INVALID_ARG, "K %d out of 1..%d", K, c->cfg.max_steps);
  if (!(temperature >= 0.f) || (temperature > 0.f && !std::isfinite(1.f / temperature)))
    return fail(c, PRISM_ERR_INVALID_ARG, "temperature %g", (double)temperature);
  const bool sampled = temperature > 0.f;
  if (!d_target_logits || !d_draft_tokens || !d_n_accepted || !d_next_token ||
      (sampled && (!d_draft_logits || !d_uniforms)))
    return fail(c, PRISM_ERR_INVALID_ARG, "NULL pointer");
  hipStream_t s = (hipStream_t)stream;
  launch_verify_chain(batch, K, c->V, sampled ? 1.f / temperature : 0.f, d_target_logits,
                      d_draft_logits, d_draft_tokens, d_uniforms, d_n_accepted, d_next_token,
                      c->vstats, c->err, s);
  HIPCHK(c, hipGetLastError());
  return PRISM_OK;
}

prism_status prism_verify_tree(prism_ctx *c, int32_t batch, int32_t n_nodes,
                               const float *d_target_logits, const int32_t *d_tokens,
                               const int32_t *d_parent, int32_t *d_n_accepted, int32_t *d_path,
                               int32_t *d_next_token, void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (batch < 1 || batch > c->cfg.max_batch)
    return fail(c, PRISM_ERR_INVALID_ARG, "batch %d out of 1..%d", batch, c->cfg.max_batch);
  if (n_nodes < 1 || n_nodes > MAX_VERIFY_NODES)
    return fail(c, PRISM_ERR_INVALID_ARG, "n_nodes %d out of 1..%d", n_nodes, MAX_VERIFY_NODES);
  if (!d_target_logits || !d_tokens || !d_parent || !d_n_accepted || !d_path || !d_next_token)
    return fail(c, PRISM_ERR_INVALID_ARG, "NULL pointer");
  launch_verify_tree(batch, n_nodes, c->V, d_target_logits, d_tokens, d_parent, d_n_accepted,
                     d_path, d_next_token, c->vstats, (hipStream_t)stream);
  HIPCHK(c, hipGetLastError());
  return PRISM_OK;
}

prism_status prism_draft_chain_catchup(prism_ctx *c, const prism_batch *batch,
                                       const prism_catchup *catchup, int32_t K,
                                       int32_t *d_out_tokens, float *d_out_logits,
                                       float *d_out_hidden, void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (!batch) return fail(c, PRISM_ERR_INVALID_ARG, "batch is NULL");
  if (!catchup) return fail(c, PRISM_ERR_INVALID_ARG, "catchup is NULL");
  if (c->new_max < 1) return fail(c, PRISM_ERR_INVALID_ARG, "context was created without max_new_rows");
  // the batch's own tokens and features are not used here
  prism_batch b = *batch;
  if (!b.d_tokens) b.d_tokens = catchup->d_tokens;
  if (!b.d_features) b.d_features = catchup->d_features;
  prism_status st = check_chain(c, &b, K, d_out_tokens);
  if (st) return st;
  const prism_catchup cu = *catchup;
  if (cu.total_rows < b.batch || cu.total_rows > c->new_max)
    return fail(c, PRISM_ERR_INVALID_ARG, "total_rows %d out of %d..%d", cu.total_rows, b.batch,
                c->new_max);
  if (!cu.d_offsets || !cu.d_tokens || !cu.d_features)
    return fail(c, PRISM_ERR_INVALID_ARG, "NULL pointer in catchup");
  const KvArgs kv = kv_of(c, &b);
  auto key = chain_key(c, 3, b, K, d_out_tokens, d_out_logits, d_out_hidden);
  key.push_back((uintptr_t)cu.total_rows);
  key.push_back((uintptr_t)cu.d_offsets);
  key.push_back((uintptr_t)cu.d_tokens);
  key.push_back((uintptr_t)cu.d_features);
  return run_graph(c, key, (hipStream_t)stream, [&](hipStream_t s) {
    enqueue_chain(c, b, kv, K, &cu, d_out_tokens, d_out_logits, d_out_hidden, s);
  });
}

prism_status prism_draft_tree(prism_ctx *c, const prism_batch *batch, int32_t depth,
                              const prism_tree_out *out, void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  prism_status st = check_batch(c, batch);
  if (st) return st;
  const int w = c->cfg.tree_width, v = c->cfg.tree_nodes;
  if (w < 1) return fail(c, PRISM_ERR_INVALID_ARG, "context was created without tree_width");
  if (depth < 1 || depth > c->cfg.max_steps || depth > (int)c->fmap.size())
    return fail(c, PRISM_ERR_INVALID_ARG, "depth %d out of 1..%zu", depth, c->fmap.size());
  if (!out || !out->d_tokens || !out->d_parent || !out->d_depth || !out->d_score || !out->d_mask)
    return fail(c, PRISM_ERR_INVALID_ARG, "NULL tree output");
  const int C = w + (depth - 1) * w * w;
  if (v > C) return fail(c, PRISM_ERR_SHAPE, "tree_nodes %d exceeds the %d candidates", v, C);
  for (int k = 1; k <= depth; ++k)
    if ((st = check_set(c, k, k == 1 ? c->cfg.feat_width : c->H))) return st;
  const prism_batch b = *batch;
  const prism_tree_out o = *out;
  const KvArgs kv = kv_of(c, &b);
  const int B = b.batch, H = c->H, V = c->V;
  std::vector<uintptr_t> key = {2, (uintptr_t)B, (uintptr_t)depth, (uintptr_t)b.d_tokens,
                                (uintptr_t)b.d_features, (uintptr_t)b.d_ctx_lens,
                                (uintptr_t)b.d_k_pool, (uintptr_t)b.d_v_pool,
                                (uintptr_t)b.d_block_table, (uintptr_t)b.n_pool_blocks,
                                (uintptr_t)o.d_tokens, (uintptr_t)o.d_parent, (uintptr_t)o.d_depth,
                                (uintptr_t)o.d_score, (uintptr_t)o.d_mask, (uintptr_t)o.d_cand_tokens,
                                (uintptr_t)o.d_cand_parent, (uintptr_t)o.d_cand_score,
                                (uintptr_t)o.d_frontier, (uintptr_t)o.d_logits};
  for (int k = 0; k < depth; ++k) key.push_back((uintptr_t)c->fmap[k]);
  TreeWs t{};
  t.B = B; t.w = w; t.D = depth; t.C = C;
  t.cand_tok = c->t_ctok; t.cand_par = c->t_cpar; t.cand_score = c->t_cscore;
  t.front = c->t_front; t.front_score = c->t_fscore;
  t.tok = c->t_tok; t.feat_row = c->t_frow; t.seq = c->t_seq; t.pos = c->t_pos; t.slot = c->t_slot;
  t.err = c->err;
  auto enqueue = [&](hipStream_t s) {
    launch_tree_setup(B, b.d_tokens, b.d_ctx_lens, c->t_tok, c->t_seq, c->t_pos, c->t_slot,
                      c->t_bits[0], s);
    for (int d = 0; d < depth; ++d) {
      Pass p{};
      p.set = c->fmap[d];
      p.R = d == 0 ? B : B * w;
      p.grp = d == 0 ? 1 : c->att_grp;   // level d > 0: sequence b owns rows b w .. b w + w - 1
      p.F = d == 0 ? c->cfg.feat_width : H;
      p.topk = w;
      p.in.tokens = c->t_tok;
      p.in.feat = d == 0 ? b.d_features : (const void *)c->hid[(d - 1) & 1];
      p.in.feat_bf16 = d == 0 ? (int)c->bf16 : 0;
      p.in.feat_ld = d == 0 ? c->cfg.feat_width : H;
      p.in.feat_rows = d == 0 ? nullptr : c->t_frow;
      p.in.seq = c->t_seq;
      p.in.pos = c->t_pos;
      p.in.slot = c->t_slot;
      p.in.bits = c->t_bits[d & 1];
      p.hid_out = c->hid[d & 1];
      p.ld_hid = H;
      if (o.d_logits) {
        p.logits = o.d_logits + (size_t)d * B * w * V;
        p.ld_logits = d == 0 ? (long)w * V : (long)V;
      }
      p.ids = c->ids;
      p.logp = c->logp;
      enqueue_pass(c, p, kv, s);
      TreeWs tt = t;
      tt.bits_prev = c->t_bits[d & 1];
      tt.bits = c->t_bits[(d + 1) & 1];
      launch_tree_expand(d, tt, b.d_ctx_lens, c->ids, c->logp, s);
    }
    launch_tree_final(t, v, o.d_tokens, o.d_parent, o.d_depth, o.d_score, o.d_mask,
                      o.d_cand_tokens, o.d_cand_parent, o.d_cand_score, o.d_frontier, s);
  };
  return run_graph(c, key, (hipStream_t)stream, enqueue);
}

prism_status prism_score_tree(prism_ctx *c, const prism_batch *batch, int32_t n_nodes,
                              const int32_t *d_tokens, const int32_t *d_depth,
                              const uint64_t *d_mask, float *d_logits, void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  prism_status st = check_batch(c, batch);
  if (st) return st;
  if (n_nodes < 1 || n_nodes > MAX_SCORE_NODES)
    return fail(c, PRISM_ERR_INVALID_ARG, "n_nodes %d out of 1..%d", n_nodes, MAX_SCORE_NODES);
  if (!d_tokens || !d_depth || !d_mask || !d_logits)
    return fail(c, PRISM_ERR_INVALID_ARG, "NULL tree or logits pointer");
  if ((st = check_set(c, 1, c->cfg.feat_width))) return st;
  const prism_batch b = *batch;
  const KvArgs kv = kv_of(c, &b);
  const int B = b.batch, V = c->V, rows = B * (n_nodes + 1);
  std::vector<uintptr_t> key = {5, (uintptr_t)B, (uintptr_t)n_nodes, (uintptr_t)b.d_tokens,
                                (uintptr_t)b.d_features, (uintptr_t)b.d_ctx_lens,
                                (uintptr_t)b.d_k_pool, (uintptr_t)b.d_v_pool,
                                (uintptr_t)b.d_block_table, (uintptr_t)b.n_pool_blocks,
                                (uintptr_t)d_tokens, (uintptr_t)d_depth, (uintptr_t)d_mask,
                                (uintptr_t)d_logits, (uintptr_t)c->fmap[0]};
  const int set = c->fmap[0];
  const int rps = n_nodes + 1;   // each tree's rows: its root, then its nodes
  // bf16: passes of whole trees, up to pass_max rows (the row-group
  // products), the tree's rows grouped in the attention, and one LM head over
  // each pass's rows; otherwise passes of up to rows_max rows with their own
  // LM heads
  const bool wide = c->bf16 && c->pass_max > c->rows_max && c->lmr_x.hi &&
                    lmhead_rows_fits(c->lm, c->pass_max) && rps <= c->pass_max;
  const int per_pass = wide ? c->pass_max / rps * rps : c->rows_max;
  return run_graph(c, key, (hipStream_t)stream, [&](hipStream_t s) {
    launch_score_setup(B, n_nodes, b.d_tokens, b.d_ctx_lens, d_tokens, d_depth, d_mask, c->s_tok,
                       c->s_seq, c->s_pos, c->s_slot, c->s_bits, c->err, s);
    // rows in tree order: a node's ancestors come before it, so their KV is
    // written by this pass or an earlier one
    for (int r0 = 0; r0 < rows; r0 += per_pass) {
      const int n = rows - r0 < per_pass ? rows - r0 : per_pass;
      Pass p{};
      p.set = set;
      p.R = n;
      p.F = c->sets[set].F;
      p.topk = 1;
      p.defer_merge = true;        // the logits are the output
      p.in.tokens = c->s_tok + r0;
      p.in.feat = b.d_features;
      p.in.feat_bf16 = (int)c->bf16;
      p.in.feat_ld = c->cfg.feat_width;
      p.in.feat_rows = c->s_seq + r0;
      p.in.seq = c->s_seq + r0;
      p.in.pos = c->s_pos + r0;
      p.in.slot = c->s_slot + r0;
      p.in.bits = c->s_bits + r0;
      p.hid_out = c->hid[0];
      p.ld_hid = c->H;
      p.logits = d_logits + (size_t)r0 * V;
      p.ld_logits = V;
      p.ids = c->ids;
      if (wide) {
        p.grp = c->score_grp;
        p.rps = rps;
        p.lm_rows_x = c->lmr_x;
        p.lm_rows_x.ld = c->H;
        p.lm_rows_scale = c->lmr_scale;
      }
      enqueue_pass(c, p, kv, s);
      if (wide) {   // the pass's LM head
        LmRowsArgs a{};
        a.m = c->lm;
        a.x = act_of(c->lmr_x, c->H);
        a.R = n;
        a.scale = c->lmr_scale;
        a.logits = d_logits + (size_t)r0 * V;
        a.ld_logits = V;
        launch_lmhead_rows(a, s);
      }
    }
  });
}

prism_status prism_profile_enable(prism_ctx *c, int32_t what) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (what & ~(PRISM_PROFILE_LMHEAD | PRISM_PROFILE_PRODUCTS | PRISM_PROFILE_PASSES))
    return fail(c, PRISM_ERR_INVALID_ARG, "unknown profile bits 0x%x", (unsigned)what);
  drop_graphs(c);
  c->profile = what != 0;
  c->prof_what = what;
  if (c->profile && c->prof_ev.empty()) {
    // per pass: one pair for the pass, five products (a split one counted
    // once) and the LM head; a tree or catch-up call runs at most max_steps
    // passes
    const int pairs = c->cfg.max_steps * 8;
    for (int i = 0; i < 2 * pairs; ++i) {
      hipEvent_t e;
      HIPCHK(c, hipEventCreate(&e));
      c->prof_ev.push_back(e);
    }
  }
  c->prof_last = 0;
  return PRISM_OK;
}

prism_status prism_profile_pairs(prism_ctx *c, float *ms, int32_t cap, int32_t *count) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (!count || (cap > 0 && !ms)) return fail(c, PRISM_ERR_INVALID_ARG, "NULL output");
  *count = 0;
  if (!c->profile) return fail(c, PRISM_ERR_INVALID_ARG, "profiling is not enabled");
  for (int i = 0; i < c->prof_last && i < cap; ++i) {
    HIPCHK(c, hipEventSynchronize(c->prof_ev[2 * i + 1]));
    HIPCHK(c, hipEventElapsedTime(&ms[i], c->prof_ev[2 * i], c->prof_ev[2 * i + 1]));
  }
  *count = c->prof_last;
  return PRISM_OK;
}

prism_status prism_profile_read(prism_ctx *c, float *total_ms, int32_t *count) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  if (!total_ms || !count) return fail(c, PRISM_ERR_INVALID_ARG, "NULL output");
  *total_ms = 0.f;
  *count = 0;
  if (!c->profile) return fail(c, PRISM_ERR_INVALID_ARG, "profiling is not enabled");
  for (int i = 0; i < c->prof_last; ++i) {
    HIPCHK(c, hipEventSynchronize(c->prof_ev[2 * i + 1]));
    float ms = 0.f;
    HIPCHK(c, hipEventElapsedTime(&ms, c->prof_ev[2 * i], c->prof_ev[2 * i + 1]));
    *total_ms += ms;
  }
  *count = c->prof_last;
  return PRISM_OK;
}

prism_status prism_graph_cache(const prism_ctx *c, int32_t *n_graphs, int32_t *capacity) {
  if (!c || !n_graphs || !capacity) return PRISM_ERR_INVALID_ARG;
  *n_graphs = (int32_t)c->graphs.size();
  *capacity = (int32_t)GRAPH_CACHE_MAX;
  return PRISM_OK;
}

prism_status prism_device_status(prism_ctx *c, void *stream) {
  if (!c) return PRISM_ERR_INVALID_ARG;
  HIPCHK(c, hipStreamSynchronize((hipStream_t)stream));
  uint32_t flags = 0, zero = 0;
  HIPCHK(c, hipMemcpy(&flags, c->err, 4, hipMemcpyDeviceToHost));
  HIPCHK(c, hipMemcpy(c->err, &zero, 4, hipMemcpyHostToDevice));
  if (flags & ERRF_NONFINITE)
    return fail(c, PRISM_ERR_NONFINITE, "NaN logits or tree scores (NaN in a feature row or a weight)");
  if (flags & ERRF_ROWS)
    return fail(c, PRISM_ERR_INVALID_ARG, "malformed catch-up offsets or tree-scoring rows");
  if (flags & ERRF_CAPACITY) return fail(c, PRISM_ERR_CAPACITY, "KV slot, block or pool out of range");
  if (flags & ERRF_TOKEN) return fail(c, PRISM_ERR_INVALID_ARG, "token id out of range");
  return PRISM_OK;
}

}  // extern "C"
