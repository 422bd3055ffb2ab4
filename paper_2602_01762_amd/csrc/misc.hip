// Row-wise kernels of the drafting step: fusion-FC input gather, split-K
// finalisation with residual + RMSNorm, LM-head partial merge (top-k and
// log-sum-exp), chain setup, and the draft-tree bookkeeping.
#include "device.h"

namespace prism {

// ---------------------------------------------------------------------------
// X[r] = [E(token_r) ; feature row]  in the storage dtype.  A feature given in
// fp32 (the draft's own hidden state) is rounded to the storage dtype, as the
// FC consumes it as a matrix-product operand.
struct FcPrepArgs {
  RowsIn in;
  const void *embed;
  int V, H, F;
  void *X;
  uint32_t *err;
};

template <typename T>
__global__ __launch_bounds__(256) void k_fc_prep(FcPrepArgs a) {
  const int r = blockIdx.x, tid = threadIdx.x;
  const int ld = a.H + a.F;
  T *x = (T *)a.X + (size_t)r * ld;
  int tok = a.in.tokens[r];
  if (tok < 0 || tok >= a.V) {
    if (tid == 0) atomicOr(a.err, ERRF_TOKEN);
    tok = -1;
  }
  const T *e = (const T *)a.embed + (size_t)(tok < 0 ? 0 : tok) * a.H;
  for (int i = tid; i < a.H; i += blockDim.x) x[i] = tok < 0 ? T(0) : e[i];
  const int fr = a.in.feat_rows ? a.in.feat_rows[r] : r;
  if (a.in.feat_bf16) {
    const bf16_t *f = (const bf16_t *)a.in.feat + (size_t)fr * a.in.feat_ld;
    for (int i = tid; i < a.F; i += blockDim.x) Ty<T>::st(x, a.H + i, bf2f(f[i]));
  } else {
    const float *f = (const float *)a.in.feat + (size_t)fr * a.in.feat_ld;
    for (int i = tid; i < a.F; i += blockDim.x) Ty<T>::st(x, a.H + i, f[i]);
  }
}

void launch_fc_prep(bool bf16, int R, const RowsIn &in, const void *embed, int V, int H, int F,
                    void *X, uint32_t *err, hipStream_t s) {
  FcPrepArgs a{in, embed, V, H, F, X, err};
  if (bf16) hipLaunchKernelGGL(k_fc_prep<bf16_t>, dim3(R), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_fc_prep<float>, dim3(R), dim3(256), 0, s, a);
}

// ---------------------------------------------------------------------------
// v = sum_s part[s][r] (+ res[r]);  out[r] = v (fp32, optional);
// normed[r] = v / sqrt(mean(v^2) + eps) * g  (storage dtype, optional)
struct RowFinArgs {
  const float *part;
  int splits, R, N;
  const float *res; int ldres;
  float *out; int ldout;
  const void *gain;
  void *normed;
  float eps;
};

template <typename T>
__global__ __launch_bounds__(256) void k_rowfin(RowFinArgs a) {
  extern __shared__ float row[];
  __shared__ float red[8];
  const int r = blockIdx.x, tid = threadIdx.x;
  float ss = 0.f;
  for (int n = tid; n < a.N; n += blockDim.x) {
    float v = 0.f;
    for (int sp = 0; sp < a.splits; ++sp) v += a.part[((size_t)sp * a.R + r) * a.N + n];
    if (a.res) v += a.res[(size_t)r * a.ldres + n];
    row[n] = v;
    if (a.out) a.out[(size_t)r * a.ldout + n] = v;
    ss += v * v;
  }
  if (!a.normed) return;
  const float tot = block_sum(ss, red);
  const float scale = 1.0f / sqrtf(tot / (float)a.N + a.eps);
  const T *g = (const T *)a.gain;
  for (int n = tid; n < a.N; n += blockDim.x)
    Ty<T>::st((T *)a.normed, (size_t)r * a.N + n, row[n] * scale * Ty<T>::ld(g, n));
}

void launch_rowfin(bool bf16, int R, int N, const float *part, int splits, const float *res,
                   int ldres, float *out, int ldout, const void *gain, void *normed, float eps,
                   hipStream_t s) {
  RowFinArgs a{part, splits, R, N, res, ldres, out, ldout, gain, normed, eps};
  const size_t lds = (size_t)N * sizeof(float);
  if (bf16) hipLaunchKernelGGL(k_rowfin<bf16_t>, dim3(R), dim3(256), lds, s, a);
  else hipLaunchKernelGGL(k_rowfin<float>, dim3(R), dim3(256), lds, s, a);
}

// ---------------------------------------------------------------------------
// Merge the LM-head partials of row r:
//   lse = M + log(sum_i s_i exp(m_i - M)),  top-k by (logit desc, id asc),
//   log-prob = logit - lse.
constexpr int MAXK = MAX_TOPK;
struct LmCombArgs {
  int R, n_wg, topk, V;
  const float *pmax, *psum, *pval;
  const int *pid;
  int *ids;
  float *logp;
  int *tok_a;          // optional [R]: ids[r][0]
  int *tok_b; int ld_b; // optional [R * ld_b]: ids[r][0]
};

__global__ __launch_bounds__(256) void k_lm_combine(LmCombArgs a) {
  __shared__ float shv[8];
  __shared__ int shi[8];
  const int r = blockIdx.x, tid = threadIdx.x;
  const float *pm = a.pmax + (size_t)r * a.n_wg;
  const float *ps = a.psum + (size_t)r * a.n_wg;
  float m = -INFINITY;
  for (int i = tid; i < a.n_wg; i += blockDim.x) m = fmaxf(m, pm[i]);
  const float M = block_max(m, shv);
  float s = 0.f;
  for (int i = tid; i < a.n_wg; i += blockDim.x) s += ps[i] * expf(pm[i] - M);
  const float S = block_sum(s, shv);
  const float lse = M + logf(S);

  const int k = a.topk;
  const int nc = a.n_wg * k;
  const float *pv = a.pval + (size_t)r * nc;
  const int *pi = a.pid + (size_t)r * nc;
  // thread-local sorted top-k of a strided subset
  float lv[MAXK];
  int li[MAXK];
  for (int j = 0; j < MAXK; ++j) { lv[j] = -INFINITY; li[j] = 0x7fffffff; }
  for (int i = tid; i < nc; i += blockDim.x) {
    float v = pv[i];
    int id = pi[i];
    if (!better(v, id, lv[k - 1], li[k - 1])) continue;
    int j = k - 1;
    while (j > 0 && better(v, id, lv[j - 1], li[j - 1])) {
      lv[j] = lv[j - 1];
      li[j] = li[j - 1];
      --j;
    }
    lv[j] = v;
    li[j] = id;
  }
  int head = 0;
  for (int j = 0; j < k; ++j) {
    float v = head < k ? lv[head] : -INFINITY;
    int id = head < k ? li[head] : 0x7fffffff;
    block_argmax(v, id, shv, shi);
    if (head < k && li[head] == id) ++head;
    if (tid == 0) {
      a.ids[(size_t)r * k + j] = id;
      if (a.logp) a.logp[(size_t)r * k + j] = v - lse;
      if (j == 0) {
        if (a.tok_a) a.tok_a[r] = id;
        if (a.tok_b) a.tok_b[(size_t)r * a.ld_b] = id;
      }
    }
  }
}

void launch_lm_combine(int R, int n_wg, int topk, int V, const float *pmax, const float *psum,
                       const float *pval, const int *pid, int *ids, float *logp, int *tok_a,
                       int *tok_b, int ld_b, hipStream_t s) {
  LmCombArgs a{R, n_wg, topk, V, pmax, psum, pval, pid, ids, logp, tok_a, tok_b, ld_b};
  hipLaunchKernelGGL(k_lm_combine, dim3(R), dim3(256), 0, s, a);
}

// ---------------------------------------------------------------------------
// Chain rows: step k (0-based) of sequence b sits at position and slot
// L_b + k; the first step's token is the last accepted one.
__global__ void k_chain_setup(int B, int K, const int32_t *tokens, const int32_t *ctx_lens,
                              int32_t *seq, int32_t *pos, int32_t *tok0) {
  for (int i = threadIdx.x; i < B * K; i += blockDim.x) {
    const int k = i / B, b = i % B;
    pos[i] = ctx_lens[b] + k;
    if (k == 0) {
      seq[b] = b;
      tok0[b] = tokens[b];
    }
  }
}

void launch_chain_setup(int B, int K, const int32_t *tokens, const int32_t *ctx_lens, int32_t *seq,
                        int32_t *pos, int32_t *tok0, hipStream_t s) {
  hipLaunchKernelGGL(k_chain_setup, dim3(1), dim3(256), 0, s, B, K, tokens, ctx_lens, seq, pos,
                     tok0);
}

// ---------------------------------------------------------------------------
// Draft tree.  Candidate c of a sequence is created in order: the root's w
// children first (depth 1), then for each later pass the w children of each
// of the w frontier nodes (frontier rank major, child rank minor).  A score
// is the parent's score plus the child's log-prob (fp32).  Order key of both
// the frontier and the output: (score desc, candidate index asc).
constexpr int TREE_MAXNEW = 256;
constexpr int TREE_MAXC = MAX_TREE_CAND;

struct TreeExpArgs {
  TreeWs t;
  int d;
  const int32_t *ctx_lens;
  const int *ids;
  const float *logp;
};

__device__ __forceinline__ bool rank_before(float sj, int j, float si, int i) {
  return sj > si || (sj == si && j < i);
}

__global__ __launch_bounds__(256) void k_tree_expand(TreeExpArgs a) {
  __shared__ float sc[TREE_MAXNEW];
  __shared__ int tk[TREE_MAXNEW];
  const TreeWs &t = a.t;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int w = t.w, d = a.d;
  const int n_new = d == 0 ? w : w * w;
  const int base = d == 0 ? 0 : w + (d - 1) * w * w;
  for (int i = tid; i < n_new; i += blockDim.x) {
    int row, c, parent;
    float ps;
    if (d == 0) {
      row = b; c = i; parent = -1; ps = 0.f;
    } else {
      const int pr = i / w;
      row = b * w + pr;
      c = i % w;
      parent = t.front[((size_t)b * (t.D - 1) + (d - 1)) * w + pr];
      ps = t.cand_score[(size_t)b * t.C + parent];
    }
    const int tok = a.ids[(size_t)row * w + c];
    const float score = ps + a.logp[(size_t)row * w + c];
    const size_t ci = (size_t)b * t.C + base + i;
    t.cand_tok[ci] = tok;
    t.cand_par[ci] = parent;
    t.cand_score[ci] = score;
    sc[i] = score;
    tk[i] = tok;
  }
  if (d >= t.D - 1) return;
  __syncthreads();
  const int L = a.ctx_lens[b];
  for (int i = tid; i < n_new; i += blockDim.x) {
    int rank = 0;
    for (int j = 0; j < n_new; ++j) rank += rank_before(sc[j], j, sc[i], i);
    if (rank >= w) continue;
    t.front[((size_t)b * (t.D - 1) + d) * w + rank] = base + i;
    const int nr = b * w + rank;
    const int prow = d == 0 ? b : b * w + i / w;
    t.tok[nr] = tk[i];
    t.feat_row[nr] = prow;
    t.seq[nr] = b;
    t.pos[nr] = L + d + 1;
    t.slot[nr] = L + 1 + d * w + rank;
    const uint64_t pb = d == 0 ? 1ull : t.bits_prev[prow];
    t.bits[nr] = pb | (1ull << (1 + d * w + rank));
  }
}

void launch_tree_expand(int d, const TreeWs &t, const int32_t *ctx_lens, const int *ids,
                        const float *logp, hipStream_t s) {
  TreeExpArgs a{t, d, ctx_lens, ids, logp};
  hipLaunchKernelGGL(k_tree_expand, dim3(t.B), dim3(256), 0, s, a);
}

// Root-pass rows: sequence b at position and slot L_b, visibility bit 0.
__global__ void k_tree_setup(int B, const int32_t *tokens, const int32_t *ctx_lens, int32_t *tok,
                             int32_t *seq, int32_t *pos, int32_t *slot, uint64_t *bits) {
  for (int b = threadIdx.x; b < B; b += blockDim.x) {
    tok[b] = tokens[b];
    seq[b] = b;
    pos[b] = ctx_lens[b];
    slot[b] = ctx_lens[b];
    bits[b] = 1ull;
  }
}

void launch_tree_setup(int B, const int32_t *tokens, const int32_t *ctx_lens, int32_t *tok,
                       int32_t *seq, int32_t *pos, int32_t *slot, uint64_t *bits, hipStream_t s) {
  hipLaunchKernelGGL(k_tree_setup, dim3(1), dim3(256), 0, s, B, tokens, ctx_lens, tok, seq, pos,
                     slot, bits);
}

struct TreeFinArgs {
  TreeWs t;
  int v;
  int32_t *tokens, *parent, *depth;
  float *score;
  uint64_t *mask;
  int32_t *c_tok, *c_par;
  float *c_score;
  int32_t *front_out;
};

__global__ __launch_bounds__(256) void k_tree_final(TreeFinArgs a) {
  __shared__ float sc[TREE_MAXC];
  __shared__ short outpos[TREE_MAXC];
  __shared__ int sel[64];
  __shared__ int par[64];
  const TreeWs &t = a.t;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int C = t.C, w = t.w;
  for (int i = tid; i < C; i += blockDim.x) {
    sc[i] = t.cand_score[(size_t)b * C + i];
    outpos[i] = -1;
  }
  __syncthreads();
  for (int i = tid; i < C; i += blockDim.x) {
    int rank = 0;
    for (int j = 0; j < C; ++j) rank += rank_before(sc[j], j, sc[i], i);
    if (rank < a.v) {
      sel[rank] = i;
      outpos[i] = (short)rank;
    }
  }
  __syncthreads();
  if (tid < a.v) {
    const int n = sel[tid];
    const int p = t.cand_par[(size_t)b * C + n];
    const int po = p >= 0 ? outpos[p] : -1;
    par[tid] = po;
    const size_t o = (size_t)b * a.v + tid;
    a.tokens[o] = t.cand_tok[(size_t)b * C + n];
    a.parent[o] = po;
    a.depth[o] = n < w ? 1 : 2 + (n - w) / (w * w);
    a.score[o] = sc[n];
  }
  __syncthreads();
  if (tid < a.v) {
    uint64_t m = 1ull << tid;
    int p = par[tid];
    while (p >= 0) {
      m |= 1ull << p;
      p = par[p];
    }
    a.mask[(size_t)b * a.v + tid] = m;
  }
  if (a.c_tok)
    for (int i = tid; i < C; i += blockDim.x) a.c_tok[(size_t)b * C + i] = t.cand_tok[(size_t)b * C + i];
  if (a.c_par)
    for (int i = tid; i < C; i += blockDim.x) a.c_par[(size_t)b * C + i] = t.cand_par[(size_t)b * C + i];
  if (a.c_score)
    for (int i = tid; i < C; i += blockDim.x) a.c_score[(size_t)b * C + i] = sc[i];
  if (a.front_out) {
    const int nf = (t.D - 1) * w;
    for (int i = tid; i < nf; i += blockDim.x)
      a.front_out[(size_t)b * nf + i] = t.front[(size_t)b * nf + i];
  }
}

void launch_tree_final(const TreeWs &t, int v, int32_t *tokens, int32_t *parent, int32_t *depth,
                       float *score, uint64_t *mask, int32_t *c_tok, int32_t *c_par,
                       float *c_score, int32_t *front_out, hipStream_t s) {
  TreeFinArgs a{t, v, tokens, parent, depth, score, mask, c_tok, c_par, c_score, front_out};
  hipLaunchKernelGGL(k_tree_final, dim3(t.B), dim3(256), 0, s, a);
}

}  // namespace prism
