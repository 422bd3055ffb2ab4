// Internal declarations shared by the kernel and runtime translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace prism {

typedef uint16_t bf16_t;  // bf16 storage (bit pattern)

// device error flags (bit set by kernels on an out-of-range device value)
enum : uint32_t { ERRF_CAPACITY = 1u, ERRF_TOKEN = 2u };

// Tiled weight matrix W[N, K] (y = W x).  Tile t holds rows 16t..16t+15;
// k-block j holds KB consecutive k (KB = 32 for bf16, 16 for fp32).  The
// 1 KiB of one (t, j) pair is laid out lane-major for a 64-lane wave: lane l
// holds the 16 bytes W[16t + (l & 15)][KB*j + E*(l >> 4) + e], e < E
// (E = 8 bf16 or 4 fp32), which is the A operand of the 16x16 MFMA.
struct TiledMat {
  void *w = nullptr;
  int N = 0, K = 0;
  int n_tiles = 0, nkb = 0;
};

enum Epi { EPI_PARTIAL = 0, EPI_SWIGLU = 1 };

constexpr int MAX_TOPK = 16;    // largest top-k of the LM-head merge
constexpr int MAX_TREE_CAND = 2048;
constexpr int MAX_ROWS = 64;

struct GemmLaunch {
  TiledMat m;
  const void *X;   // [R, ldx] activations in the storage dtype
  int ldx;
  int R;
  int kw;          // waves of a workgroup splitting K for one tile (1, 2, 4)
  int splits;      // workgroups splitting K for one tile (grid.y)
  float *part;     // EPI_PARTIAL: [splits][R][N]
  void *Z;         // EPI_SWIGLU: [R, ldz] storage dtype, N/2 outputs
  int ldz;
};

struct LmLaunch {
  TiledMat m;
  const void *X;
  int ldx, R, V, topk;
  float *logits; long ld_logits;   // optional fp32 [R, ld_logits]
  float *pmax, *psum, *pval;       // partials [R][n_wg] / [R][n_wg][topk]
  int *pid;
  int n_wg;
};

// ---- launchers (gemm.hip) -------------------------------------------------
void launch_gemm(bool bf16, int epi, const GemmLaunch &g, hipStream_t s);
void launch_lmhead(bool bf16, const LmLaunch &g, hipStream_t s);
int lm_workgroups(int n_tiles);
void launch_repack(bool bf16, const void *src, int n_src_rows, int K, int row_stride,
                   int row_offset, TiledMat &dst, hipStream_t s);

// ---- launchers (misc.hip) -------------------------------------------------
struct RowsIn {
  const int32_t *tokens;
  const void *feat; int feat_bf16; int feat_ld; const int32_t *feat_rows;
  const int32_t *seq, *pos, *slot;
  const uint64_t *bits;
};

void launch_fc_prep(bool bf16, int R, const RowsIn &in, const void *embed, int V, int H, int F,
                    void *X, uint32_t *err, hipStream_t s);
// sum split partials (+ residual) -> fp32 row (optional) and RMSNorm(row)*g -> storage dtype
void launch_rowfin(bool bf16, int R, int N, const float *part, int splits, const float *res,
                   int ldres, float *out, int ldout, const void *gain, void *normed, float eps,
                   hipStream_t s);
struct KvArgs {
  void *k_pool, *v_pool;
  const int32_t *block_table;
  const int32_t *ctx_lens;
  int mbps;        // block-table columns
  int bs;          // slots per block
  int n_blocks;    // pool blocks
  int n_seq;       // sequences described (valid values of a row's seq)
};
// sum QKV partials, RoPE q and k, write q (storage dtype) and k, v into the cache
void launch_qkv_fin(bool bf16, int R, int nq, int nkv, int d, const float *part, int splits,
                    const RowsIn &in, const KvArgs &kv, const double *inv_freq, void *q_out,
                    uint32_t *err, hipStream_t s);
void launch_attention(bool bf16, int R, int nq, int nkv, int d, const void *q, const RowsIn &in,
                      const KvArgs &kv, int max_slots, int chunk, float *pm, float *pl, float *po,
                      void *o_out, uint32_t *err, hipStream_t s);
// merge LM-head partials: top-k ids, optional log-probs, and the chain's token copies
void launch_lm_combine(int R, int n_wg, int topk, int V, const float *pmax, const float *psum,
                       const float *pval, const int *pid, int *ids, float *logp, int *tok_a,
                       int *tok_b, int ld_b, hipStream_t s);
void launch_chain_setup(int B, int K, const int32_t *tokens, const int32_t *ctx_lens, int32_t *seq,
                        int32_t *pos, int32_t *tok0, hipStream_t s);
// tree bookkeeping
struct TreeWs {
  int B, w, D, C;                 // batch, width, depth, candidates per sequence
  int32_t *cand_tok, *cand_par;   // [B, C]
  float *cand_score;              // [B, C]
  int32_t *front;                 // [B, D-1, w] candidate index of frontier nodes
  int32_t *tok, *feat_row, *seq, *pos, *slot; // next-pass rows [B*w]
  uint64_t *bits;                 // next-pass visibility [B*w]
  uint64_t *bits_prev;            // visibility of the pass just run [B*w]
};
// after pass d (0 = root): record children, choose the next frontier (if d < D-1),
// and write the rows of pass d+1
void launch_tree_expand(int d, const TreeWs &t, const int32_t *ctx_lens, const int *ids,
                        const float *logp, hipStream_t s);
void launch_tree_setup(int B, const int32_t *tokens, const int32_t *ctx_lens, int32_t *tok,
                       int32_t *seq, int32_t *pos, int32_t *slot, uint64_t *bits, hipStream_t s);
void launch_tree_final(const TreeWs &t, int v, int32_t *tokens, int32_t *parent, int32_t *depth,
                       float *score, uint64_t *mask, int32_t *c_tok, int32_t *c_par,
                       float *c_score, int32_t *front_out, hipStream_t s);

}  // namespace prism
