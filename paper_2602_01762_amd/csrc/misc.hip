// Row-wise kernels of the drafting step: fusion-FC input gather, split-K
// finalisation with residual + RMSNorm, LM-head partial merge (top-k and
// log-sum-exp), chain setup, and the draft-tree bookkeeping.
#include "device.h"
#include "tree_order.h"

namespace prism {

// ---------------------------------------------------------------------------
// X[r] = [E(token_r) ; feature row] as the FC's operand planes.  Embeddings
// and target features are exact in the storage type (lo = 0); a fp32 feature
// (the draft's own hidden state) is split into its hi/lo pair.
// The row's token is RowsIn::tokens[r], or the argmax of the previous LM
// head's top-1 partials (then recorded by one workgroup).
struct FcPrepArgs {
  RowsIn in;
  TokFromLm lm;
  const void *embed;
  int V, H, F;
  ActOut X;
  uint32_t *err;
  int32_t *tok_out;   // optional [R]: the row's token, -1 if out of range
  int feat_only;      // the embedding half comes from a table: write the feature columns only
};

template <typename T>
__global__ __launch_bounds__(256) void k_fc_prep(FcPrepArgs a) {
  __shared__ float shv[4];
  __shared__ int shi[4];
  const int r = blockIdx.y;
  int tok;
  if (a.lm.pval) {
    tok = token_from_lm(a.lm, r, shv, shi);
    if (a.lm.rec && blockIdx.x == 0 && threadIdx.x == 0) a.lm.rec[(size_t)r * a.lm.ld_rec] = tok;
  } else {
    tok = a.in.tokens[r];
  }
  const int e0 = (blockIdx.x * 256 + threadIdx.x) * 8;   // 8 consecutive columns
  if (tok < 0 || tok >= a.V) {
    // from the LM head, only a row of NaN logits leaves no token
    if (e0 == 0) atomicOr(a.err, a.lm.pval && tok == NO_TOKEN ? ERRF_NONFINITE : ERRF_TOKEN);
    tok = -1;
  }
  if (a.tok_out && e0 == 0) a.tok_out[r] = tok;
  if (e0 >= a.H + a.F || (a.feat_only && e0 < a.H)) return;
  const size_t o = (size_t)r * a.X.ld + e0;
  float v[8];
  bool exact;   // value already representable in the storage type
  if (e0 < a.H) {
    exact = true;
    const T *e = (const T *)a.embed + (size_t)(tok < 0 ? 0 : tok) * a.H + e0;
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = tok < 0 ? 0.f : Ty<T>::ld(e, i);
  } else {
    const int fr = a.in.feat_rows ? a.in.feat_rows[r] : r;
    const int c = e0 - a.H;
    if (a.in.feat_bf16) {
      exact = sizeof(T) == 2;
      const bf16_t *f = (const bf16_t *)a.in.feat + (size_t)fr * a.in.feat_ld + c;
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = bf2f(f[i]);
    } else {
      exact = sizeof(T) == 4;
      const float *f = (const float *)a.in.feat + (size_t)fr * a.in.feat_ld + c;
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = f[i];
    }
  }
  if constexpr (sizeof(T) == 2) {
    bf16_t *hi = (bf16_t *)a.X.hi + o, *lo = (bf16_t *)a.X.lo + o;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t h = f2bf(v[i]);
      hi[i] = (bf16_t)h;
      lo[i] = exact ? (bf16_t)0 : (bf16_t)f2bf(v[i] - bf2f(h));
    }
  } else {
    float *hi = (float *)a.X.hi + o;
#pragma unroll
    for (int i = 0; i < 8; ++i) hi[i] = v[i];
  }
}

void launch_fc_prep(bool bf16, int R, const RowsIn &in, const TokFromLm &lm, const void *embed,
                    int V, int H, int F, ActOut X, uint32_t *err, int32_t *tok_out, bool feat_only,
                    hipStream_t s) {
  FcPrepArgs a{in, lm, embed, V, H, F, X, err, tok_out, feat_only ? 1 : 0};
  dim3 grid((H + F + 2047) / 2048, R);
  if (bf16) hipLaunchKernelGGL(k_fc_prep<bf16_t>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_fc_prep<float>, grid, dim3(256), 0, s, a);
}

// ---------------------------------------------------------------------------
// Row scales for consumers that cannot reduce the producer's partials
// themselves: scale[r] = 1/sqrt(sum_t ss[t*R + r]/n + eps)
__global__ __launch_bounds__(256) void k_rowscale(int R, const float *ss, int n_parts, int n,
                                                  float eps, float *scale) {
  __shared__ float sh[8];
  const int r = blockIdx.x;
  float acc = 0.f;
  for (int t = threadIdx.x; t < n_parts; t += blockDim.x) acc += ss[(size_t)t * R + r];
  const float tot = block_sum(acc, sh);
  if (threadIdx.x == 0) scale[r] = 1.0f / sqrtf(tot / (float)n + eps);
}

void launch_rowscale(int R, const float *ss, int n_parts, int n, float eps, float *scale,
                     hipStream_t s) {
  hipLaunchKernelGGL(k_rowscale, dim3(R), dim3(256), 0, s, R, ss, n_parts, n, eps, scale);
}

// ---------------------------------------------------------------------------
// Merge the LM-head partials of row r:
//   lse = M + log(sum_i s_i exp(m_i - M)),  top-k by (logit desc, id asc),
//   log-prob = logit - lse.
struct LmCombArgs {
  int R, n_wg, topk, V;
  const float *pmax, *psum, *pval;
  const int *pid;
  int *ids;
  float *logp;
  int *tok_a;          // optional [R]: ids[r][0]
  int *tok_b; int ld_b; // optional [R * ld_b]: ids[r][0]
  uint32_t *err;        // ERRF_NONFINITE when a row has no token (every logit NaN)
};

// KB: a power of two >= topk.  Each LM-head workgroup's k candidates come
// sorted (best first), so thread t takes the lists of workgroups t, t + 256,
// ... and merges them into one sorted register list of compile-time length
// (fixed indices: no dynamic register indexing); the block then takes k
// rounds of arg-max over the list heads.  The loads of a batch of CL lists
// (their max and sum partials and their candidates) go out together before
// any is used, from clamped indices, so a merge over up to 256 * CL
// workgroups costs one memory latency.
template <int KB>
__global__ __launch_bounds__(256) void k_lm_combine(LmCombArgs a) {
  constexpr int CL = 16 / KB > 1 ? 16 / KB : 1;   // lists per thread and batch
  __shared__ float shv[8];
  const int r = blockIdx.x, tid = threadIdx.x;
  const int k = a.topk;
  const float *pm = a.pmax + (size_t)r * a.n_wg;
  const float *ps = a.psum + (size_t)r * a.n_wg;
  const float *pv = a.pval + (size_t)r * a.n_wg * k;
  const int *pi = a.pid + (size_t)r * a.n_wg * k;
  float m = -INFINITY, s = 0.f;   // log-sum-exp: online merge in list order
  float lv[KB];                   // this thread's sorted candidates
  int li[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) { lv[j] = -INFINITY; li[j] = 0x7fffffff; }
  for (int l0 = 0; l0 * 256 < a.n_wg; l0 += CL) {
    float vm[CL], vs[CL], cv[CL][KB];
    int ci[CL][KB];
#pragma unroll
    for (int l = 0; l < CL; ++l) {
      const int w = tid + 256 * (l0 + l);
      const int wc = w < a.n_wg ? w : 0;
      vm[l] = pm[wc];
      vs[l] = ps[wc];
#pragma unroll
      for (int j = 0; j < KB; ++j) {
        const int jc = j < k ? j : 0;
        cv[l][j] = pv[(size_t)wc * k + jc];
        ci[l][j] = pi[(size_t)wc * k + jc];
      }
    }
#pragma unroll
    for (int l = 0; l < CL; ++l) {
      if (tid + 256 * (l0 + l) >= a.n_wg) continue;
      if (vm[l] != -INFINITY) {
        if (vm[l] > m) {
          s = s * expf(m - vm[l]) + vs[l];
          m = vm[l];
        } else {
          s += vs[l] * expf(vm[l] - m);
        }
      }
      // merge this list into the running one, keeping the best KB (each
      // step takes the better head and shifts that list)
      float bv[KB], ov[KB];
      int bi[KB], oi[KB];
#pragma unroll
      for (int j = 0; j < KB; ++j) {
        const bool ok = j < k;
        bv[j] = ok ? cv[l][j] : -INFINITY;
        bi[j] = ok ? ci[l][j] : 0x7fffffff;
      }
#pragma unroll
      for (int j = 0; j < KB; ++j) {
        const bool take_b = better(bv[0], bi[0], lv[0], li[0]);
        ov[j] = take_b ? bv[0] : lv[0];
        oi[j] = take_b ? bi[0] : li[0];
#pragma unroll
        for (int q = 0; q < KB - 1; ++q) {
          bv[q] = take_b ? bv[q + 1] : bv[q];
          bi[q] = take_b ? bi[q + 1] : bi[q];
          lv[q] = take_b ? lv[q] : lv[q + 1];
          li[q] = take_b ? li[q] : li[q + 1];
        }
        bv[KB - 1] = take_b ? -INFINITY : bv[KB - 1];
        bi[KB - 1] = take_b ? 0x7fffffff : bi[KB - 1];
        lv[KB - 1] = take_b ? lv[KB - 1] : -INFINITY;
        li[KB - 1] = take_b ? li[KB - 1] : 0x7fffffff;
      }
#pragma unroll
      for (int j = 0; j < KB; ++j) { lv[j] = ov[j]; li[j] = oi[j]; }
    }
  }
  const float M = block_max(m, shv);
  const float S = block_sum(m == -INFINITY ? 0.f : s * expf(m - M), shv);
  const float lse = M + logf(S);
  // each wave takes the best k of its lanes' lists (k rounds of a wave
  // arg-max over the list heads, on 64-bit candidate keys, no barriers),
  // then thread 0 merges the four waves' sorted lists
  __shared__ uint64_t s_wk[4][KB];
  const int wave = tid >> 6, lane = tid & 63;
  uint64_t lk[KB];
#pragma unroll
  for (int j = 0; j < KB; ++j) lk[j] = cand_key(lv[j], li[j]);
  const uint64_t none = cand_key(-INFINITY, 0x7fffffff);
#pragma unroll
  for (int j = 0; j < KB; ++j) {
    if (j >= k) break;
    uint64_t b[1] = {lk[0]};
    wave_max_key_n<1>(b);
    if (lane == 0) s_wk[wave][j] = b[0];
    const bool win = lk[0] == b[0];   // keys are distinct: one owner (or all spent)
#pragma unroll
    for (int q = 0; q + 1 < KB; ++q) lk[q] = win ? lk[q + 1] : lk[q];
    lk[KB - 1] = win ? none : lk[KB - 1];
  }
  __syncthreads();
  if (tid != 0) return;
  int hd[4] = {0, 0, 0, 0};
  for (int j = 0; j < k; ++j) {
    int bw = 0;
    uint64_t best = hd[0] < k ? s_wk[0][hd[0]] : 0ull;
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const uint64_t c = hd[w] < k ? s_wk[w][hd[w]] : 0ull;
      if (c > best) { best = c; bw = w; }
    }
    ++hd[bw];
    const int id = key_id(best);
    if (j == 0 && id == NO_TOKEN) atomicOr(a.err, ERRF_NONFINITE);
    a.ids[(size_t)r * k + j] = id;
    if (a.logp) a.logp[(size_t)r * k + j] = key_value(best) - lse;
    if (j == 0) {
      if (a.tok_a) a.tok_a[r] = id;
      if (a.tok_b) a.tok_b[(size_t)r * a.ld_b] = id;
    }
  }
}

// ---------------------------------------------------------------------------
// Stochastic drafting: inverse-CDF draw of row r (one workgroup).  Groups
// are contiguous vocab ranges in id order; thread t owns a contiguous run of
// at most SAMP_PER groups, so an exclusive prefix of the per-thread sums in
// thread order orders the whole vocabulary.  The prefix is a fixed-order
// scan (a wave scan, then the four wave totals in order), so the draw does
// not depend on scheduling.  The first group whose running sum passes u * S
// holds the token; wave 0 then scans that group's ids with a fixed-order wave
// prefix sum.  A draw that rounding pushes past the last group takes the
// highest id of nonzero probability.  Every load goes out unconditionally
// (clamped index, masked value), so that each phase costs one memory
// latency.
constexpr int SAMP_PER = 8;         // groups per thread: n_wg <= 2048
constexpr int SAMP_GROUP_MAX = 512; // ids per group scanned by wave 0
__device__ __forceinline__ float wave_incl_scan(float x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float t = __shfl_up(x, o, 64);
    if (lane >= o) x += t;
  }
  return x;
}

__global__ __launch_bounds__(256) void k_lm_sample(LmSampleArgs a) {
  __shared__ float shv[8];
  __shared__ float s_wtot[4];
  __shared__ int s_hit[4], s_last[4];
  __shared__ int s_g;
  __shared__ float s_base;
  const int r = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float *pm = a.pmax + (size_t)r * a.n_wg;
  const float *ps = a.psum + (size_t)r * a.n_wg;
  const int per = (a.n_wg + 255) / 256;   // <= SAMP_PER (checked by the launcher)
  const int g0 = tid * per;
  float vm[SAMP_PER], vs[SAMP_PER];
#pragma unroll
  for (int i = 0; i < SAMP_PER; ++i) {
    const int g = g0 + i < a.n_wg ? g0 + i : 0;
    vm[i] = pm[g];
    vs[i] = ps[g];
  }
  const float u = fminf(fmaxf(a.u[(size_t)r * a.ld_u], 0.f), 1.f);
  auto mine = [&](int i) { return i < per && g0 + i < a.n_wg; };
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < SAMP_PER; ++i)
    if (mine(i)) m = fmaxf(m, vm[i]);
  const float M = block_max(m, shv);
  float w[SAMP_PER], loc = 0.f;
#pragma unroll
  for (int i = 0; i < SAMP_PER; ++i) {
    w[i] = mine(i) && vm[i] != -INFINITY ? vs[i] * expf(vm[i] - M) : 0.f;
    loc += w[i];
  }
  // exclusive prefix of the thread sums, in thread order
  const float incl = wave_incl_scan(loc, lane);
  if (lane == 63) s_wtot[wave] = incl;
  __syncthreads();
  float wbase = 0.f, S = 0.f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (q < wave) wbase += s_wtot[q];
    S += s_wtot[q];
  }
  const float goal = u * S;
  // this thread's first group that passes the goal
  int cg = 0x7fffffff;
  float cb = 0.f;
  {
    float run = wbase + incl - loc;
#pragma unroll
    for (int i = 0; i < SAMP_PER; ++i) {
      if (cg == 0x7fffffff && w[i] > 0.f && run + w[i] > goal) {
        cg = g0 + i;
        cb = run;
      }
      run += w[i];
    }
  }
  // the lowest thread with a hit wins (groups are in thread order)
  const unsigned long long hb = __ballot(cg != 0x7fffffff);
  if (lane == 0) s_hit[wave] = hb ? 64 * wave + __ffsll((long long)hb) - 1 : 0x7fffffff;
  // fallback: the last group of nonzero weight
  int lastg = -1;
  float lastw = 0.f;
#pragma unroll
  for (int i = 0; i < SAMP_PER; ++i)
    if (w[i] > 0.f) {
      lastg = g0 + i;
      lastw = w[i];
    }
  __syncthreads();
  int win = 0x7fffffff;
#pragma unroll
  for (int q = 0; q < 4; ++q) win = min(win, s_hit[q]);
  if (win != 0x7fffffff) {
    if (tid == win) {
      s_g = cg;
      s_base = cb;
    }
  } else {
    int hl = lastg;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) hl = max(hl, __shfl_xor(hl, o, 64));
    if (lane == 0) s_last[wave] = hl;
    __syncthreads();
    int gl = -1;
#pragma unroll
    for (int q = 0; q < 4; ++q) gl = max(gl, s_last[q]);
    if (gl >= 0 && lastg == gl) {   // its owner: base = S - its weight (all later weights are zero)
      s_g = gl;
      s_base = S - lastw;
    }
    if (gl < 0 && tid == 0) {
      s_g = -1;
      s_base = 0.f;
    }
  }
  __syncthreads();
  if (tid >= 64) return;
  const int g = s_g;
  int tok = -1;
  if (g >= 0) {
    const float *lg = a.logits + (size_t)r * a.ld_logits;
    const int id0 = g * a.group;
    constexpr int NC = SAMP_GROUP_MAX / 64;
    float e[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int id = id0 + 64 * c + lane;
      e[c] = lg[id < a.V && 64 * c < a.group ? id : id0];
    }
    float run = s_base;
    int last_nz = -1;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      if (64 * c >= a.group || tok >= 0) break;
      const int id = id0 + 64 * c + lane;
      const float ev = id < a.V ? expf(e[c] * a.inv_temp - M) : 0.f;
      const float x = wave_incl_scan(ev, lane);   // inclusive prefix over the wave, fixed order
      const unsigned long long hit = __ballot(ev > 0.f && run + x > goal);
      const unsigned long long nz = __ballot(ev > 0.f);
      if (nz) last_nz = id0 + 64 * c + 63 - __clzll((long long)nz);
      if (hit) tok = id0 + 64 * c + __ffsll((long long)hit) - 1;
      run += __shfl(x, 63, 64);
    }
    if (tok < 0) tok = last_nz;
  }
  if (lane == 0) {
    if (tok < 0) atomicOr(a.err, ERRF_NONFINITE);   // no id of positive weight
    a.ids[r] = tok;
    if (a.logp) {
      const float lt = tok >= 0 ? a.logits[(size_t)r * a.ld_logits + tok] * a.inv_temp : -INFINITY;
      a.logp[(size_t)r * a.ld_logp] = lt - M - logf(S);
    }
    if (a.tok_a) a.tok_a[r] = tok;
    if (a.tok_b) a.tok_b[(size_t)r * a.ld_b] = tok;
  }
}

bool lm_sample_fits(int n_wg, int group) {
  return n_wg <= 256 * SAMP_PER && group <= SAMP_GROUP_MAX && group % 64 == 0;
}

void launch_lm_sample(const LmSampleArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(k_lm_sample, dim3(a.R), dim3(256), 0, s, a);
}

// Top-k partials from stored fp32 logits, for rows whose LM head skips its
// own epilogue: workgroup (chunk c, row r) reduces the ids [c * TK_CHUNK,
// (c + 1) * TK_CHUNK) of row r to the partials the LM-head epilogue writes
// (max, sum of exp(logit - max), and the top-k sorted best first), so the
// merge kernel takes them unchanged.  Thread t holds ids t, t + 256, ...
// (coalesced loads).
//
// The top-k is exact but filters first, because the arithmetic of k full
// arg-max rounds over every candidate bounds this kernel: each wave finds a
// threshold T_w, the k-th largest of its 64 lane maxima (k rounds over one
// float per lane; lanes that tie are removed together, so at least k lane
// maxima are >= T_w, and so are the wave's k best).  The workgroup keeps
// only the candidates >= max_w T_w (typically about k of them) in LDS, and
// each candidate's place is the number of better ones.  A chunk with fewer
// than k or more than TK_CAP such candidates (ties, NaN) takes the plain
// path instead: per-thread sorted keys, k rounds of wave arg-max, and wave 0
// merging the four wave lists the same way.
constexpr int TK_PER = 16;
constexpr int TK_CHUNK = 256 * TK_PER;
constexpr int TK_CAP = 256;
__global__ __launch_bounds__(256) void k_lm_topk(LmTopkArgs a) {
  __shared__ float sh[8];
  __shared__ float s_thr[4];
  __shared__ int s_n;
  __shared__ uint64_t s_cand[TK_CAP];
  __shared__ uint64_t wl[4][TK_MAXK];
  const int c = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int base = c * TK_CHUNK;
  const float *row = a.logits + (size_t)r * a.ld;
  const int k = a.topk;
  float v[TK_PER];
#pragma unroll
  for (int j = 0; j < TK_PER; ++j) {
    const int id = base + tid + 256 * j;
    v[j] = id < a.V ? row[id] : -INFINITY;
  }
  if (tid == 0) s_n = 0;
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < TK_PER; ++j) mx = fmaxf(mx, v[j]);
  const float M = block_max(mx, sh);
  float e = 0.f;
#pragma unroll
  for (int j = 0; j < TK_PER; ++j)
    e += base + tid + 256 * j < a.V ? expf(v[j] * a.inv_temp - M * a.inv_temp) : 0.f;
  const float S = block_sum(e, sh);
  const size_t pi = (size_t)r * a.n_wg + c;
  if (tid == 0) {
    a.pmax[pi] = M * a.inv_temp;
    a.psum[pi] = S;
  }
  // the wave's threshold: k-th largest lane maximum (ties removed together)
  float cur = mx, thr = -INFINITY;
  int removed = 0;
  for (int j = 0; j < k && removed < k; ++j) {
    thr = wave_max(cur);
    const bool hit = cur == thr;
    removed += __popcll(__ballot(hit));
    cur = hit ? -INFINITY : cur;
  }
  if (lane == 0) s_thr[wave] = thr;
  __syncthreads();
  const float T = fmaxf(fmaxf(s_thr[0], s_thr[1]), fmaxf(s_thr[2], s_thr[3]));
#pragma unroll
  for (int j = 0; j < TK_PER; ++j) {
    const int id = base + tid + 256 * j;
    if (id < a.V && v[j] >= T) {
      const int slot = atomicAdd(&s_n, 1);
      if (slot < TK_CAP) s_cand[slot] = cand_key(v[j], id);
    }
  }
  __syncthreads();
  const int n = s_n;
  if (n >= k && n <= TK_CAP) {   // uniform
    if (tid < n) {
      const uint64_t mine = s_cand[tid];
      int rank = 0;
#pragma unroll 8
      for (int i = 0; i < n; ++i) rank += s_cand[i] > mine ? 1 : 0;
      if (rank < k) {
        a.pval[pi * k + rank] = key_value(mine);
        a.pid[pi * k + rank] = key_id(mine);
      }
    }
    return;
  }
  // plain path
  uint64_t key[TK_PER];
#pragma unroll
  for (int j = 0; j < TK_PER; ++j) {
    const int id = base + tid + 256 * j;
    key[j] = cand_key(v[j], id < a.V ? id : 0x7fffffff);
  }
  // odd-even transposition sort, best first
#pragma unroll
  for (int pass = 0; pass < TK_PER; ++pass)
#pragma unroll
    for (int j = pass & 1; j + 1 < TK_PER; j += 2) {
      const uint64_t lo = key[j], hi = key[j + 1];
      key[j] = hi > lo ? hi : lo;
      key[j + 1] = hi > lo ? lo : hi;
    }
  const uint64_t none = cand_key(-INFINITY, 0x7fffffff);
  for (int j = 0; j < k; ++j) {
    uint64_t bk[1] = {key[0]};
    wave_max_key_n<1>(bk);
    if (lane == 0) wl[wave][j] = bk[0];
    // the winning lane drops its head (ids are distinct; "none" keys are
    // only ever dropped for one another)
    const bool win = key[0] == bk[0];
#pragma unroll
    for (int q = 0; q + 1 < TK_PER; ++q) key[q] = win ? key[q + 1] : key[q];
    key[TK_PER - 1] = win ? none : key[TK_PER - 1];
  }
  __syncthreads();
  if (wave != 0) return;
  // lane l holds candidate l % k of wave l / k (4 k <= 64)
  uint64_t ck = lane < 4 * k ? wl[lane / k][lane % k] : none;
  for (int j = 0; j < k; ++j) {
    uint64_t bk[1] = {ck};
    wave_max_key_n<1>(bk);
    if (lane == 0) {
      a.pval[pi * k + j] = key_value(bk[0]);
      a.pid[pi * k + j] = key_id(bk[0]);
    }
    ck = ck == bk[0] ? none : ck;
  }
}

int lm_topk_chunks(int V) { return (V + TK_CHUNK - 1) / TK_CHUNK; }

void launch_lm_topk(const LmTopkArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(k_lm_topk, dim3(a.n_wg, a.R), dim3(256), 0, s, a);
}

// The same merge for at most 64 partial lists per row (the tree levels'
// top-k pass), one wave per row, 4 rows per workgroup: lane l holds list l
// and its (max, sum of exp); two wave reductions give the log-sum-exp and k
// rounds of a wave arg-max over the list heads the top-k, with no barriers.
// (A workgroup per row left 7 of 8 threads idle and paid the block
// reductions' barriers.)
template <int KB>
__global__ __launch_bounds__(256) void k_lm_combine_w(LmCombArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + wave;
  if (r >= a.R) return;                       // whole waves; no barriers below
  const int k = a.topk;
  const bool has = lane < a.n_wg;             // n_wg <= 64 (launcher)
  const int wc = has ? lane : 0;
  const float *pv = a.pval + ((size_t)r * a.n_wg + wc) * k;
  const int *pi = a.pid + ((size_t)r * a.n_wg + wc) * k;
  const uint64_t none = cand_key(-INFINITY, 0x7fffffff);
  uint64_t lk[KB];                            // the lane's list, best first
#pragma unroll
  for (int j = 0; j < KB; ++j) {
    const int jc = j < k ? j : 0;
    const float v = pv[jc];
    const int id = pi[jc];
    lk[j] = has && j < k ? cand_key(v, id) : none;
  }
  const float m = has ? a.pmax[(size_t)r * a.n_wg + wc] : -INFINITY;
  const float sl = has ? a.psum[(size_t)r * a.n_wg + wc] : 0.f;
  const float M = wave_max(m);
  const float S = wave_sum(m == -INFINITY ? 0.f : sl * expf(m - M));
  const float lse = M + logf(S);
  for (int j = 0; j < k; ++j) {
    uint64_t b[1] = {lk[0]};
    wave_max_key_n<1>(b);
    const bool win = lk[0] == b[0];           // keys are distinct: one owner (or all spent)
#pragma unroll
    for (int q = 0; q + 1 < KB; ++q) lk[q] = win ? lk[q + 1] : lk[q];
    lk[KB - 1] = win ? none : lk[KB - 1];
    if (lane == 0) {
      const int id = key_id(b[0]);
      if (j == 0 && id == NO_TOKEN) atomicOr(a.err, ERRF_NONFINITE);
      a.ids[(size_t)r * k + j] = id;
      if (a.logp) a.logp[(size_t)r * k + j] = key_value(b[0]) - lse;
      if (j == 0) {
        if (a.tok_a) a.tok_a[r] = id;
        if (a.tok_b) a.tok_b[(size_t)r * a.ld_b] = id;
      }
    }
  }
}

void launch_lm_combine(int R, int n_wg, int topk, int V, const float *pmax, const float *psum,
                       const float *pval, const int *pid, int *ids, float *logp, int *tok_a,
                       int *tok_b, int ld_b, uint32_t *err, hipStream_t s) {
  LmCombArgs a{R, n_wg, topk, V, pmax, psum, pval, pid, ids, logp, tok_a, tok_b, ld_b, err};
  if (n_wg <= 64 && topk > 1) {   // few lists per row (the tree's top-k pass): a wave per row
    const dim3 g((R + 3) / 4);
    if (topk <= 2) hipLaunchKernelGGL(k_lm_combine_w<2>, g, dim3(256), 0, s, a);
    else if (topk <= 4) hipLaunchKernelGGL(k_lm_combine_w<4>, g, dim3(256), 0, s, a);
    else if (topk <= 8) hipLaunchKernelGGL(k_lm_combine_w<8>, g, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_lm_combine_w<16>, g, dim3(256), 0, s, a);
    return;
  }
  if (topk <= 1) hipLaunchKernelGGL(k_lm_combine<1>, dim3(R), dim3(256), 0, s, a);
  else if (topk <= 2) hipLaunchKernelGGL(k_lm_combine<2>, dim3(R), dim3(256), 0, s, a);
  else if (topk <= 4) hipLaunchKernelGGL(k_lm_combine<4>, dim3(R), dim3(256), 0, s, a);
  else if (topk <= 8) hipLaunchKernelGGL(k_lm_combine<8>, dim3(R), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_lm_combine<16>, dim3(R), dim3(256), 0, s, a);
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
// Catch-up chain rows.  Accepted row r (of T) belongs to the sequence b with
// offsets[b] <= r < offsets[b+1] and sits at position and slot
// L_b + r - offsets[b]; step k (0-based) of the chain then runs at
// L_b + n_b - 1 + k, step 0 being the prefill's last row.  A malformed table
// (offsets[0] != 0, offsets[B] != T, or an empty sequence) raises ERRF_ROWS;
// rows that fall in no sequence get seq -1, which every later kernel skips.
__global__ void k_catchup_setup(int B, int T, int K, const int32_t *offsets,
                                const int32_t *ctx_lens, int32_t *rseq, int32_t *rpos,
                                int32_t *last, int32_t *seq, int32_t *pos, uint32_t *err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < T) {
    int lo = 0, hi = B;   // largest b with offsets[b] <= i (bounded search)
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (offsets[mid] <= i) lo = mid; else hi = mid;
    }
    const bool ok = offsets[lo] <= i && i < offsets[lo + 1];
    rseq[i] = ok ? lo : -1;
    rpos[i] = ok ? ctx_lens[lo] + (i - offsets[lo]) : 0;
  }
  if (i < B) {
    const int o0 = offsets[i], o1 = offsets[i + 1];
    const bool bad = o1 <= o0 || (i == 0 && o0 != 0) || (i == B - 1 && o1 != T);
    if (bad) atomicOr(err, ERRF_ROWS);
    last[i] = bad || o1 - 1 >= T ? -1 : o1 - 1;
    seq[i] = bad ? -1 : i;
    for (int k = 0; k < K; ++k) pos[(size_t)k * B + i] = ctx_lens[i] + (o1 - o0 - 1) + k;
  }
}

void launch_catchup_setup(int B, int T, int K, const int32_t *offsets, const int32_t *ctx_lens,
                          int32_t *rseq, int32_t *rpos, int32_t *last, int32_t *seq, int32_t *pos,
                          uint32_t *err, hipStream_t s) {
  const int n = T > B ? T : B;
  hipLaunchKernelGGL(k_catchup_setup, dim3((n + 255) / 256), dim3(256), 0, s, B, T, K, offsets,
                     ctx_lens, rseq, rpos, last, seq, pos, err);
}

// For each of two dense fp32 matrices m (blockIdx.z), destination row b <
// rows: the source row idx[b] - r0 if it is one of the n_src source rows,
// zeros if idx[b] = -1 (first chunk only), else nothing.
__global__ void k_rows_gather(RowsGather a) {
  const int b = blockIdx.y, m = blockIdx.z;
  const int i = a.idx[b];
  const int r = i - a.r0;
  const bool take = i >= 0 && r >= 0 && r < a.n_src;
  const bool zero = i < 0 && a.r0 == 0;
  if (!take && !zero) return;
  const int n = a.n[m];
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < n; c += gridDim.x * blockDim.x)
    a.dst[m][(size_t)b * n + c] = take ? a.src[m][(size_t)r * n + c] : 0.f;
}

void launch_rows_gather(int rows, const RowsGather &a, hipStream_t s) {
  const int n = a.n[0] > a.n[1] ? a.n[0] : a.n[1];
  hipLaunchKernelGGL(k_rows_gather, dim3((n + 255) / 256, rows, 2), dim3(256), 0, s, a);
}

// ---------------------------------------------------------------------------
// Draft tree.  Candidate c of a sequence is created in order: the root's w
// children first (depth 1), then for each later pass the w children of each
// of the w frontier nodes (frontier rank major, child rank minor).  A score
// is the parent's score plus the child's log-prob (fp32).  Order key of both
// the frontier and the output: (score desc, candidate index asc), with NaN
// scores after every number (tree_before; tree_rank_key as one integer), a
// total order, so that every rank below the cut has exactly one candidate.
constexpr int TREE_MAXNEW = 256;
constexpr int TREE_MAXC = MAX_TREE_CAND;

// Rank of candidate key k among n keys in LDS: the number of greater keys.
// Unrolled so that the LDS reads of a batch are in flight together (one
// read at a time waits its full latency per candidate: 30 us for 328).
__device__ __forceinline__ int tree_rank(const uint64_t *keys, int n, uint64_t k) {
  int r = 0;
#pragma unroll 16
  for (int j = 0; j < n; ++j) r += keys[j] > k ? 1 : 0;
  return r;
}

struct TreeExpArgs {
  TreeWs t;
  int d;
  const int32_t *ctx_lens;
  const int *ids;
  const float *logp;
};

__global__ __launch_bounds__(256) void k_tree_expand(TreeExpArgs a) {
  __shared__ uint64_t rk[TREE_MAXNEW];
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
      // the parent's index and score, both recorded with the frontier (no
      // load that waits on another)
      const int pr = i / w;
      row = b * w + pr;
      c = i % w;
      const size_t fi = ((size_t)b * (t.D - 1) + (d - 1)) * w + pr;
      parent = t.front[fi];
      ps = t.front_score[fi];
    }
    const int tok = a.ids[(size_t)row * w + c];
    const float score = ps + a.logp[(size_t)row * w + c];
    const size_t ci = (size_t)b * t.C + base + i;
    t.cand_tok[ci] = tok;
    t.cand_par[ci] = parent;
    t.cand_score[ci] = score;
    rk[i] = tree_rank_key(score, i);
    sc[i] = score;
    tk[i] = tok;
  }
  if (d >= t.D - 1) return;
  __syncthreads();
  const int L = a.ctx_lens[b];
  for (int i = tid; i < n_new; i += blockDim.x) {
    const int rank = tree_rank(rk, n_new, rk[i]);
    if (rank >= w) continue;
    t.front[((size_t)b * (t.D - 1) + d) * w + rank] = base + i;
    t.front_score[((size_t)b * (t.D - 1) + d) * w + rank] = sc[i];
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

// Rows of a tree-scoring pass (the target model's side of tree
// verification): sequence b owns rows b * (n + 1) .. b * (n + 1) + n.  Row 0
// is the root (the last accepted token) at position and slot L_b; row 1 + j
// is node j at position L_b + depth_j and slot L_b + 1 + j, seeing the root
// (bit 0) and its ancestor mask shifted by one.  A depth outside 1..n or a
// mask that lacks the node's own bit or names a later node is clamped to a
// well-formed row and raises ERRF_ROWS.
__global__ void k_score_setup(int B, int n, const int32_t *root_tok, const int32_t *ctx_lens,
                              const int32_t *tokens, const int32_t *depth, const uint64_t *mask,
                              int32_t *tok, int32_t *seq, int32_t *pos, int32_t *slot,
                              uint64_t *bits, uint32_t *err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * (n + 1)) return;
  const int b = i / (n + 1), r = i % (n + 1);
  const int L = ctx_lens[b];
  seq[i] = b;
  if (r == 0) {
    tok[i] = root_tok[b];
    pos[i] = L;
    slot[i] = L;
    bits[i] = 1ull;
    return;
  }
  const int j = r - 1;                     // j <= 62
  const size_t o = (size_t)b * n + j;
  int dp = depth[o];
  uint64_t m = mask[o];
  const uint64_t keep = (2ull << j) - 1;   // bits 0..j
  if (dp < 1 || dp > n || (m & ~keep) || !((m >> j) & 1ull)) atomicOr(err, ERRF_ROWS);
  dp = dp < 1 ? 1 : (dp > n ? n : dp);
  m = (m & keep) | (1ull << j);
  tok[i] = tokens[o];
  pos[i] = L + dp;
  slot[i] = L + 1 + j;
  bits[i] = 1ull | (m << 1);
}

void launch_score_setup(int B, int n, const int32_t *root_tok, const int32_t *ctx_lens,
                        const int32_t *tokens, const int32_t *depth, const uint64_t *mask,
                        int32_t *tok, int32_t *seq, int32_t *pos, int32_t *slot, uint64_t *bits,
                        uint32_t *err, hipStream_t s) {
  const int rows = B * (n + 1);
  hipLaunchKernelGGL(k_score_setup, dim3((rows + 255) / 256), dim3(256), 0, s, B, n, root_tok,
                     ctx_lens, tokens, depth, mask, tok, seq, pos, slot, bits, err);
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

// Final top-v of the C candidates of sequence b.  Every candidate's score,
// token and parent goes out in one batch of loads (unconditional, clamped
// index) into LDS; the ranks, outputs and copies then read LDS only.
__global__ __launch_bounds__(256) void k_tree_final(TreeFinArgs a) {
  constexpr int PER = (TREE_MAXC + 255) / 256;
  __shared__ float sc[TREE_MAXC];
  __shared__ uint64_t rk[TREE_MAXC];
  __shared__ int tk[TREE_MAXC], pa[TREE_MAXC];
  __shared__ short outpos[TREE_MAXC];
  __shared__ int sel[64];
  __shared__ int par[64];
  const TreeWs &t = a.t;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int C = t.C, w = t.w;
  // the frontier copy is requested with the candidates, not after the
  // ranking: (D - 1) w <= 63 entries (the context admits at most 64 draft
  // slots), one per thread
  const int nf = a.front_out ? (t.D - 1) * w : 0;
  const int fr = tid < nf ? t.front[(size_t)b * nf + tid] : 0;
  bool nan_seen = false;
  {
    float vs[PER];
    int vt[PER], vp[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int i = tid + 256 * q;
      const size_t ci = (size_t)b * C + (i < C ? i : 0);
      vs[q] = t.cand_score[ci];
      vt[q] = t.cand_tok[ci];
      vp[q] = t.cand_par[ci];
    }
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int i = tid + 256 * q;
      if (i < C) {
        sc[i] = vs[q];
        rk[i] = tree_rank_key(vs[q], i);
        tk[i] = vt[q];
        pa[i] = vp[q];
        outpos[i] = -1;
        nan_seen |= vs[q] != vs[q];
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < C; i += blockDim.x) {
    const int rank = tree_rank(rk, C, rk[i]);
    if (rank < a.v) {
      sel[rank] = i;
      outpos[i] = (short)rank;
    }
  }
  // a NaN score (from a NaN feature row or weight) is reported; the tree
  // is still well formed (NaN candidates rank last, parents first)
  if (nan_seen) atomicOr(t.err, ERRF_NONFINITE);
  __syncthreads();
  if (tid < a.v) {
    const int n = sel[tid];
    const int p = pa[n];
    const int po = p >= 0 && p < C ? outpos[p] : -1;
    par[tid] = po;
    const size_t o = (size_t)b * a.v + tid;
    a.tokens[o] = tk[n];
    a.parent[o] = po;
    a.depth[o] = n < w ? 1 : 2 + (n - w) / (w * w);
    a.score[o] = sc[n];
  }
  __syncthreads();
  if (tid < a.v) a.mask[(size_t)b * a.v + tid] = tree_ancestor_bits(par, tid);
  for (int i = tid; i < C; i += blockDim.x) {
    if (a.c_tok) a.c_tok[(size_t)b * C + i] = tk[i];
    if (a.c_par) a.c_par[(size_t)b * C + i] = pa[i];
    if (a.c_score) a.c_score[(size_t)b * C + i] = sc[i];
  }
  if (tid < nf) a.front_out[(size_t)b * nf + tid] = fr;
}

void launch_tree_final(const TreeWs &t, int v, int32_t *tokens, int32_t *parent, int32_t *depth,
                       float *score, uint64_t *mask, int32_t *c_tok, int32_t *c_par,
                       float *c_score, int32_t *front_out, hipStream_t s) {
  TreeFinArgs a{t, v, tokens, parent, depth, score, mask, c_tok, c_par, c_score, front_out};
  hipLaunchKernelGGL(k_tree_final, dim3(t.B), dim3(256), 0, s, a);
}

}  // namespace prism
