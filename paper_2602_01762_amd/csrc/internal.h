// Internal declarations shared by the kernel and runtime translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.h"

namespace prism {

typedef uint16_t bf16_t;  // bf16 storage (bit pattern)

// message of the last failed call that takes no context (prism_create, the
// static verification), read by prism_last_error(NULL)
void set_global_error(const char *msg);

// device error flags: set by kernels on an out-of-range device value
// (capacity, token, rows), or on logits that are NaN (nonfinite: every
// logit of a row NaN, or a NaN tree score)
enum : uint32_t { ERRF_CAPACITY = 1u, ERRF_TOKEN = 2u, ERRF_ROWS = 4u, ERRF_NONFINITE = 8u };
// id of an empty (value, id) candidate in the top-k merges: it survives a
// merge only when no candidate compares above -inf, i.e. every logit is NaN
constexpr int NO_TOKEN = 0x7fffffff;

constexpr int MAX_TOPK = 16;
constexpr int MAX_VERIFY_NODES = 64;   // tree nodes one verification call takes
constexpr int MAX_TREE_CAND = 2048;
constexpr int MAX_NEW_ROWS = 4096;     // accepted rows of one catch-up call
constexpr int MAX_SCORE_NODES = 63;    // nodes of one scored tree (visibility bits 1..63)

// Tiled weight matrix W[N, K] (y = W x).  Tile t holds 16 output rows;
// k-block j holds KB consecutive k (KB = 32 for bf16, 16 for fp32).  The
// 1 KiB of one (t, j) pair is laid out lane-major for a 64-lane wave: lane l
// holds the 16 bytes W[row(t, l & 15)][KB*j + E*(l >> 4) + e], e < E
// (E = 8 bf16 or 4 fp32), which is the A operand of the 16x16 MFMA.
// row(t, i) = 16t + i, except for rotated (q, k) heads, whose tile j of a
// head holds dims 8j..8j+7 in rows 0..7 and d/2+8j..d/2+8j+7 in rows 8..15,
// so that the two halves of every rotation pair sit in lanes l and l ^ 32.
struct TiledMat {
  void *w = nullptr;
  int N = 0, K = 0;
  int n_tiles = 0, nkb = 0;
};

// An activation operand [R, ld] of a product.  fp32 models: `hi` is fp32
// and `lo` is null.  bf16 models: the fp32 value x is carried as the pair
// hi = bf16(x), lo = bf16(x - hi) (two planes), both fed to the MFMA, so the
// product sees x to within 2^-17 relative.
struct Act {
  const void *hi = nullptr;
  const void *lo = nullptr;
  int ld = 0;
};
struct ActOut {
  void *hi = nullptr;
  void *lo = nullptr;
  int ld = 0;
};

// Row norms: the producer of a vector x writes, per 16-feature tile t and
// row r, ss[t * R + r] = sum of x^2 over the tile; a consumer that multiplies
// by RMSNorm(x) * g takes x*g as its operand and scales row r of its result
// by 1/sqrt(sum_t ss[t*R + r] / n + eps).
struct RowNorm {
  const float *ss = nullptr;     // partial sums of squares [n_parts][R], reduced by
                                 // the consumer itself, or
  const float *scale = nullptr;  // row scales already reduced (launch_rowscale)
  int n_parts = 0;               // partial sums per row
  int n = 0;
  float eps = 0.f;
};

struct KvArgs {
  void *k_pool, *v_pool;
  const int32_t *block_table;
  const int32_t *ctx_lens;
  int mbps;        // block-table columns
  int bs;          // slots per block
  int n_blocks;    // pool blocks
  int n_seq;       // sequences described (valid values of a row's seq)
};

struct RowsIn {
  const int32_t *tokens;
  const void *feat; int feat_bf16; int feat_ld; const int32_t *feat_rows;
  const int32_t *seq, *pos, *slot;
  const uint64_t *bits;
};

// EPI_STORE (row-group kernel only): y = scale * acc, nothing else (the LM
// head of a tree-scoring pass)
enum Epi { EPI_NORM = 0, EPI_SWIGLU = 1, EPI_QKV = 2, EPI_STORE = 3 };

// Token of each row taken straight from the previous LM head's top-1
// partials ([R][n_wg] values and ids; larger value wins, ties -> lower id),
// so that no separate merge kernel runs between two chain steps.  The chosen
// token is also recorded at rec[r * ld_rec] (one writer).
struct TokFromLm {
  const float *pval;   // NULL: tokens come from RowsIn::tokens
  const int *pid;
  int n_wg;
  int32_t *rec; int ld_rec;
};

// Fusion-FC operand rows gathered by the product kernel itself:
// x_r = [E(token_r) ; feature row], the GEMV path's staging step.
struct Gather {
  const void *embed;   // NULL: the operand comes as planes (GemmLaunch::x)
  int V, H;
  RowsIn in;           // tokens and feature rows
  TokFromLm lm;
};

struct GemmLaunch {
  TiledMat m;
  Act x;
  int R;
  int kw;          // waves of the workgroup splitting K (1..16)
  int nt;          // tiles per workgroup (1 or 2)
  int gemv;        // 1: VALU GEMV main loop (bf16, R <= 4, staged fp32 activations)
  int split;       // > 0: batched path, K split over `split` workgroup slices
  int rowgrp;      // 1: more than MAX_ROWS rows: the row-group kernel (k_gemm_rows), split slices
  float *part;     // batched path: slice partial sums [split][R][N]
  int epi;
  RowNorm norm;    // scale rows of the result (SWIGLU, QKV); n_parts = 0: none
  // EPI_NORM: y = acc (+ res) -> y [R, ldy] fp32; (y * gain) -> g planes; ss
  const float *res; int ldres;
  float *y; int ldy;
  const void *gain;
  ActOut g;
  float *ss;       // [gemm_ss_parts][R]
  // EPI_SWIGLU: interleaved gate/up rows -> z planes [R, N/2]
  ActOut z;
  // EPI_QKV: q (fp32 [R, nq*d]) and the cache slots of k, v
  float *q;
  int nq, nkv, d;
  RowsIn rows;
  KvArgs kv;
  const double *inv_freq;
  uint32_t *err;
  Gather gx;       // GEMV fusion FC: rows gathered from E and the features
  // GEMV fusion FC with the embedding table: the product covers k-blocks
  // [kb_lo, nkb) (the feature columns), and EPI_NORM adds tab[token][n], the
  // embedding half W_fc[:, :H] E[token] precomputed for every token
  const float *tab;
  int kb_lo;
  const int32_t *tab_tok;   // batched path: each row's token (-1: none), written by the FC prep
  // chain steps >= 2 without an FC prep pass: the previous step's down
  // product also writes its output y as operand planes (yx.hi != NULL), and
  // wave 0 of K-split workgroup i < R resolves row i's token (from gx.lm, or
  // gx.in.tokens; -1 if out of range) into tok_out for the finish pass
  ActOut yx;
  int32_t *tok_out;
};

struct LmLaunch {
  TiledMat m;
  Act x;
  int R, V, topk;
  RowNorm norm;
  float *logits; long ld_logits;   // optional fp32 [R, ld_logits]
  float *pmax, *psum, *pval;       // partials [R][n_wg] / [R][n_wg][topk]
  int *pid;
  int n_wg;
  int nt;                          // vocab tiles per wave (1, 2, 4 or 8)
  int gemv;                        // 1: VALU GEMV main loop (bf16, one row)
  float inv_temp;                  // pmax / psum describe logits * inv_temp (1: greedy)
  int no_part;                     // 1: store the logits only (k_lm_topk writes the partials)
};

// ---- launchers (gemm.hip) -------------------------------------------------
// false (nothing launched): the plan's workgroup exceeds the bound of the
// kernel instantiation it selects
bool launch_gemm(bool bf16, const GemmLaunch &g, hipStream_t s);
void launch_lmhead(bool bf16, const LmLaunch &g, hipStream_t s);
// LM head over up to LMR_MAX_ROWS rows in one launch, logits only (bf16,
// the row-group product kernel): logits[r][v] = scale[r] * (W x_r)[v]
constexpr int LMR_MAX_ROWS = 256;
struct LmRowsArgs {
  TiledMat m;
  Act x;                  // [R, H] hi/lo planes
  int R;
  const float *scale;     // [R] row scales, or NULL
  float *logits; long ld_logits;
};
bool lmhead_rows_fits(const TiledMat &m, int R);
void launch_lmhead_rows(const LmRowsArgs &g, hipStream_t s);
int lm_workgroups(int n_tiles, int nt);
// partial sums of squares per row that an EPI_NORM launch writes
int gemm_ss_parts(const GemmLaunch &g);
// whether the launch (its finish pass, if split) reduces the row scales of
// its operand from n_parts partials per row itself
bool gemm_own_scales(const GemmLaunch &g, int n_parts);
bool lm_own_scales(int R, int n_parts);
void launch_rowscale(int R, const float *ss, int n_parts, int n, float eps, float *scale,
                     hipStream_t s);
// rotated rows: the first rot_rows destination rows hold rotated heads of size d
void launch_repack(bool bf16, const void *src, int n_src_rows, int K, int row_stride,
                   int row_offset, int rot_rows, int d, TiledMat &dst, hipStream_t s);

// ---- launchers (misc.hip) -------------------------------------------------
void launch_fc_prep(bool bf16, int R, const RowsIn &in, const TokFromLm &lm, const void *embed,
                    int V, int H, int F, ActOut X, uint32_t *err, int32_t *tok_out, bool feat_only, hipStream_t s);
// grp > 1: rows r .. r + grp - 1 (r a multiple of grp) belong to one sequence
// and carry tree bits; the launch groups them when the kernel allows it.
// rps > 0 (with grp > 1): the rows come in runs of rps rows of one tree each,
// grouped in grp rows from each run's first row.
// The partials pm, pl, po hold R * attention_chunks(max_slots, nsub) rows
// x chunks for the steps per workgroup that attention_nsub gives this pass
// (attention_partial_rows bounds them over every pass).
void launch_attention(bool bf16, int R, int nq, int nkv, int d, const float *q, const RowsIn &in,
                      const KvArgs &kv, int max_slots, int grp, int rps, float *pm, float *pl,
                      float *po, ActOut o, uint32_t *err, hipStream_t s);
// Draw each row's token from softmax(logits * inv_temp) by inverse CDF in
// id order with the row's uniform u[r * ld_u]: the LM head's per-group
// (max, sum) of the scaled logits locate the group where the running sum
// passes u * total, and the row's stored fp32 logits locate the id inside it.
struct LmSampleArgs {
  int R, n_wg, V, group;           // group: vocab ids per LM-head workgroup
  float inv_temp;
  const float *pmax, *psum;        // [R][n_wg], scaled logits
  const float *logits; long ld_logits;
  const float *u; int ld_u;
  int *ids;                        // [R] drawn token
  float *logp; int ld_logp;        // [R * ld_logp] its log-probability, or NULL
  int *tok_a;                      // optional [R] copy
  int *tok_b; int ld_b;            // optional [R * ld_b] copy
  uint32_t *err;                   // ERRF_NONFINITE when no id has positive weight
};
// whether the sampler takes n_wg LM-head partials per row and groups of
// `group` ids
bool lm_sample_fits(int n_wg, int group);
void launch_lm_sample(const LmSampleArgs &a, hipStream_t s);
// ---- launchers (verify.hip) -----------------------------------------------
// device address of the static verification scratch on the current device
// (resolved once per device)
hipError_t verify_scratch(void **out);
// workspace for the per-slice statistics of `rows` logits rows
size_t verify_stats_bytes(int rows);
void launch_verify_chain(int B, int K, int V, float inv_t, const float *tl, const float *dl,
                         const int32_t *drafts, const float *u, int32_t *n_acc, int32_t *next,
                         void *stats, uint32_t *err, hipStream_t s);
void launch_verify_tree(int B, int nodes, int V, const float *tl, const int32_t *tokens,
                        const int32_t *parent, int32_t *n_acc, int32_t *path, int32_t *next,
                        void *stats, hipStream_t s);
// T[v][n] = sum_{k < H} W[n][k] E[v][k] for every token v: the embedding
// half of a fusion FC in the tiled layout (k-blocks [0, H / 32) of each tile)
// times the embedding rows, fp32 [V, N]; N a multiple of 64
void launch_embed_table(const TiledMat &w, const void *embed, int V, int H, float *T, hipStream_t s);
// top-k partials from stored logits [R, ld] (rows whose LM head skips its
// epilogue): n_wg = lm_topk_chunks(V) chunks per row, topk <= TK_MAXK, in the
// layout of the LM-head partials
constexpr int TK_MAXK = 16;
struct LmTopkArgs {
  const float *logits; long ld;
  int R, V, topk, n_wg;
  float inv_temp;
  float *pmax, *psum, *pval;
  int *pid;
};
int lm_topk_chunks(int V);
void launch_lm_topk(const LmTopkArgs &a, hipStream_t s);
// merge LM-head partials: top-k ids, optional log-probs, and the chain's token copies
void launch_lm_combine(int R, int n_wg, int topk, int V, const float *pmax, const float *psum,
                       const float *pval, const int *pid, int *ids, float *logp, int *tok_a,
                       int *tok_b, int ld_b, uint32_t *err, hipStream_t s);
void launch_chain_setup(int B, int K, const int32_t *tokens, const int32_t *ctx_lens, int32_t *seq,
                        int32_t *pos, int32_t *tok0, hipStream_t s);
// catch-up chain: per accepted row its sequence and position; per sequence
// its last row and the chain's positions [K][B]
void launch_catchup_setup(int B, int T, int K, const int32_t *offsets, const int32_t *ctx_lens,
                          int32_t *rseq, int32_t *rpos, int32_t *last, int32_t *seq, int32_t *pos,
                          uint32_t *err, hipStream_t s);
// Two dense fp32 matrices [*, n[m]]: destination row b takes source row
// idx[b] - r0 when r0 <= idx[b] < r0 + n_src (the source holds rows r0 ..
// r0 + n_src - 1 of a longer list), is left as it is when idx[b] falls
// outside, and is zeroed when idx[b] = -1 (on the call with r0 = 0).
struct RowsGather {
  const int32_t *idx;            // [rows]
  int r0, n_src;
  const float *src[2];
  float *dst[2];
  int n[2];
};
void launch_rows_gather(int rows, const RowsGather &a, hipStream_t s);
// tree bookkeeping
struct TreeWs {
  int B, w, D, C;                 // batch, width, depth, candidates per sequence
  int32_t *cand_tok, *cand_par;   // [B, C]
  float *cand_score;              // [B, C]
  int32_t *front;                 // [B, D-1, w] candidate index of frontier nodes
  float *front_score;             // [B, D-1, w] their scores
  int32_t *tok, *feat_row, *seq, *pos, *slot; // next-pass rows [B*w]
  uint64_t *bits;                 // next-pass visibility [B*w]
  uint64_t *bits_prev;            // visibility of the pass just run [B*w]
  uint32_t *err;                  // device error flags
};
// after pass d (0 = root): record children, choose the next frontier (if d < D-1),
// and write the rows of pass d+1
void launch_tree_expand(int d, const TreeWs &t, const int32_t *ctx_lens, const int *ids,
                        const float *logp, hipStream_t s);
// rows of a tree-scoring pass: root and nodes of each of B trees of n nodes
void launch_score_setup(int B, int n, const int32_t *root_tok, const int32_t *ctx_lens,
                        const int32_t *tokens, const int32_t *depth, const uint64_t *mask,
                        int32_t *tok, int32_t *seq, int32_t *pos, int32_t *slot, uint64_t *bits,
                        uint32_t *err, hipStream_t s);
void launch_tree_setup(int B, const int32_t *tokens, const int32_t *ctx_lens, int32_t *tok,
                       int32_t *seq, int32_t *pos, int32_t *slot, uint64_t *bits, hipStream_t s);
void launch_tree_final(const TreeWs &t, int v, int32_t *tokens, int32_t *parent, int32_t *depth,
                       float *score, uint64_t *mask, int32_t *c_tok, int32_t *c_par,
                       float *c_score, int32_t *front_out, hipStream_t s);

}  // namespace prism
