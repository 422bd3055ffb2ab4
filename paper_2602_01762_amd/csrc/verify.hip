// Verification step that follows drafting (paper Sec. 2): the target model
// scores the drafted tokens in one pass, and the drafts are kept while they
// pass the test -- greedy: the target's own arg-max equals the draft;
// sampled: the rejection rule r < min(1, p_target(x) / p_draft(x)), with the
// replacement drawn from max(0, p_target - p_draft) at the first rejection,
// or one extra token from p_target when all pass.  Trees (greedy): the
// longest root path whose every node is the target's choice at its parent.
//
// Logits rows are V-wide fp32 (0.5 MB at V = 128256), so the work is a
// stream over them: k_rows_stats splits each row over VSPLIT workgroups,
// each reducing its slice to (max z, sum exp(z - max), arg-max of the raw
// logits), z = logit / T (greedy verification: the arg-max only); one
// workgroup per sequence then merges the slices in order and takes the
// decisions.  Draws use the drafter's inverse CDF
// in token-id order.
#include <cstdarg>
#include <cstdio>
#include <mutex>

#include "device.h"
#include "prism_draft.h"

namespace prism {

constexpr int VSPLIT = 8;
constexpr int VER_UNROLL = 4;

struct RowStat {      // one slice of one row
  float mx, sum, best;
  int arg;
};

// slice of a row: ids [lo, hi) with lo a multiple of 4 (16-byte loads)
__device__ __forceinline__ void slice_of(int V, int part, int &lo, int &hi) {
  const int per = (((V + VSPLIT - 1) / VSPLIT) + 3) & ~3;
  lo = min(V, part * per);
  hi = min(V, lo + per);
}

// SOFT = false (greedy verification, which reads only the arg-max): no
// exponentials, and the statistics stored as (-inf, 0).
template <bool SOFT>
__global__ __launch_bounds__(256) void k_rows_stats(const float *__restrict__ x, int V,
                                                    float inv_t, RowStat *out) {
  __shared__ float shv[8];
  __shared__ int shi[8];
  const int row = blockIdx.y, part = blockIdx.x, tid = threadIdx.x;
  int lo, hi;
  slice_of(V, part, lo, hi);
  const float *r = x + (size_t)row * V;   // V % 4 == 0: rows are 16-byte aligned
  float mz = -INFINITY, s = 0.f, bv = -INFINITY;
  int bi = 0x7fffffff;
  auto take = [&](float v, int i) {
    if (better(v, i, bv, bi)) { bv = v; bi = i; }
    if (!SOFT) return;
    const float z = v * inv_t;            // online max / sum of exp(z - max)
    if (z > mz) {
      s = s * expf(mz - z) + 1.f;
      mz = z;
    } else {
      s += expf(z - mz);
    }
  };
  for (int i0 = lo + 4 * tid; i0 < hi; i0 += 4 * 256 * VER_UNROLL) {
    f32x4 v[VER_UNROLL];
#pragma unroll
    for (int u = 0; u < VER_UNROLL; ++u) {   // all loads first
      const int i = i0 + u * 4 * 256;
      v[u] = i + 3 < hi ? *(const f32x4 *)(r + i) : f32x4{0.f, 0.f, 0.f, 0.f};
      if (i < hi && i + 3 >= hi)
        for (int q = 0; q < 4; ++q) v[u][q] = i + q < hi ? r[i + q] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < VER_UNROLL; ++u) {
      const int i = i0 + u * 4 * 256;
      for (int q = 0; q < 4; ++q)
        if (i + q < hi) take(v[u][q], i + q);
    }
  }
  float M = -INFINITY, S = 0.f;
  if constexpr (SOFT) {
    M = block_max(mz, shv);
    S = block_sum(mz == -INFINITY ? 0.f : s * expf(mz - M), shv);
  }
  block_argmax(bv, bi, shv, shi);
  if (tid == 0) out[(size_t)row * VSPLIT + part] = RowStat{M, S, bv, bi};
}

// merge the slices of one row: max z, sum exp(z - max), arg-max
struct RowSum {
  float M, S;
  int arg;
};
__device__ __forceinline__ RowSum merge_row(const RowStat *st) {
  float M = -INFINITY, bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int p = 0; p < VSPLIT; ++p) {
    M = fmaxf(M, st[p].mx);
    if (better(st[p].best, st[p].arg, bv, bi)) { bv = st[p].best; bi = st[p].arg; }
  }
  float S = 0.f;
  for (int p = 0; p < VSPLIT; ++p)
    if (st[p].mx != -INFINITY) S += st[p].sum * expf(st[p].mx - M);
  return RowSum{M, S, bi};
}

// Block-wide inverse-CDF draw over ids 0..V-1 with weights w(i) >= 0 (id
// order).  Ids go in blocks of 256 (lane l of a wave holds ids 4l..4l+3 of a
// block, one 16-byte load per row); wave w owns a contiguous run of blocks.
// Pass 1 sums each wave's run; an in-order prefix over the waves finds the
// run holding u * total.  Pass 2 splits that run over the waves again (a
// share of a few blocks each, all loaded at once), and a second in-order
// prefix finds the share; pass 3 walks the share block by block with a lane
// prefix sum (lane order = id order) to the id.  (One wave walking the whole
// run waited on one block's load after another.)  Rounding that leaves no
// crossing takes the highest id of positive weight of the run.  L(base)
// loads the raw values of ids base..base+3 (unconditionally) and
// W(raw, base, v[4]) gives their 4 weights (ids >= V weigh 0); the passes
// load a batch of DRAW_BATCH blocks before weighing them, so that the loads
// are in flight together.  s_wave holds DRAW_SHARED floats, s_pick 3 ints.
constexpr int DRAW_THREADS = 1024;
constexpr int DRAW_WAVES = DRAW_THREADS / 64;
constexpr int DRAW_SHARED = 2 * DRAW_WAVES + 4;
constexpr int DRAW_BATCH = 8;
struct DrawRaw {
  f32x4 x, y;          // the target row's values (and the draft row's, for the residual)
};

// sum of the weights of blocks [b0, b1) in this lane's columns, loaded a
// batch at a time
template <typename L, typename W>
__device__ __forceinline__ float lane_sum(int b0, int b1, int lane, L ld, W wg) {
  float acc = 0.f;
  for (int blk = b0; blk < b1; blk += DRAW_BATCH) {
    DrawRaw raw[DRAW_BATCH];
#pragma unroll
    for (int j = 0; j < DRAW_BATCH; ++j) raw[j] = ld(min(blk + j, b1 - 1) * 256 + 4 * lane);
#pragma unroll
    for (int j = 0; j < DRAW_BATCH; ++j) {
      if (blk + j >= b1) break;
      float v[4];
      wg(raw[j], (blk + j) * 256 + 4 * lane, v);
      acc += (v[0] + v[1]) + (v[2] + v[3]);
    }
  }
  return acc;
}

// the first of n in-order sums that carries the running total (from base)
// past goal: its index and the total before it; none (rounding): the last
// positive one, with the goal moved to +inf
__device__ __forceinline__ void pick_in_order(const float *sums, int n, float base, float goal,
                                              int &pick, float &at, float &g) {
  float run = base;
  pick = -1;
  at = base;
  g = goal;
  for (int i = 0; i < n; ++i) {
    if (sums[i] > 0.f && run + sums[i] > goal) { pick = i; at = run; return; }
    run += sums[i];
  }
  for (int i = n - 1; i >= 0; --i)
    if (sums[i] > 0.f) { pick = i; break; }
  g = INFINITY;
}

template <typename L, typename W>
__device__ int draw_ids(int V, float u, L ld, W wg, float *s_wave, int *s_pick) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nblk = (V + 255) / 256;
  {   // pass 1: each wave's run
    const int r0 = (int)((long)wave * nblk / DRAW_WAVES), r1 = (int)((long)(wave + 1) * nblk / DRAW_WAVES);
    const float acc = wave_sum(r1 > r0 ? lane_sum(r0, r1, lane, ld, wg) : 0.f);
    if (lane == 0) s_wave[wave] = acc;
  }
  __syncthreads();
  if (tid == 0) {
    float total = 0.f;
    for (int i = 0; i < DRAW_WAVES; ++i) total += s_wave[i];
    int pick;
    float at, g;
    pick_in_order(s_wave, DRAW_WAVES, 0.f, fminf(fmaxf(u, 0.f), 1.f) * total, pick, at, g);
    s_pick[0] = pick;
    s_wave[2 * DRAW_WAVES] = at;
    s_wave[2 * DRAW_WAVES + 1] = g;
    s_pick[1] = -1;
  }
  __syncthreads();
  const int run_w = s_pick[0];
  if (run_w >= 0) {   // uniform
    // pass 2: the run's blocks split over the waves
    const int p0 = (int)((long)run_w * nblk / DRAW_WAVES), p1 = (int)((long)(run_w + 1) * nblk / DRAW_WAVES);
    const int b0 = p0 + (int)((long)wave * (p1 - p0) / DRAW_WAVES);
    const int b1 = p0 + (int)((long)(wave + 1) * (p1 - p0) / DRAW_WAVES);
    const float acc = wave_sum(b1 > b0 ? lane_sum(b0, b1, lane, ld, wg) : 0.f);
    if (lane == 0) s_wave[DRAW_WAVES + wave] = acc;
    __syncthreads();
    if (tid == 0) {
      int pick;
      float at, g;
      pick_in_order(s_wave + DRAW_WAVES, DRAW_WAVES, s_wave[2 * DRAW_WAVES], s_wave[2 * DRAW_WAVES + 1],
                    pick, at, g);
      s_pick[2] = pick;
      s_wave[2 * DRAW_WAVES + 2] = at;
      s_wave[2 * DRAW_WAVES + 3] = g;
    }
    __syncthreads();
    // pass 3: the share that holds the goal, walked by its wave
    if (wave == s_pick[2]) {
      float run = s_wave[2 * DRAW_WAVES + 2];
      const float goal = s_wave[2 * DRAW_WAVES + 3];
      int found = -1, last = -1;
      for (int blk = b0; blk < b1 && found < 0; ++blk) {
        float v[4];
        wg(ld(blk * 256 + 4 * lane), blk * 256 + 4 * lane, v);
        const float ls = (v[0] + v[1]) + (v[2] + v[3]);
        float x = ls;   // inclusive prefix over the lanes, fixed order
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const float t = __shfl_up(x, o, 64);
          if (lane >= o) x += t;
        }
        const unsigned long long hit = __ballot(ls > 0.f && run + x > goal);
        const unsigned long long nz = __ballot(ls > 0.f);
        if (nz) {
          const int l = 63 - __clzll((long long)nz);
          const float vl[4] = {__shfl(v[0], l, 64), __shfl(v[1], l, 64), __shfl(v[2], l, 64),
                               __shfl(v[3], l, 64)};
          for (int q = 3; q >= 0; --q)
            if (vl[q] > 0.f) { last = blk * 256 + 4 * l + q; break; }
        }
        if (hit) {
          const int l = __ffsll((long long)hit) - 1;
          float r = run + __shfl(x, l, 64) - __shfl(ls, l, 64);   // prefix before lane l
          const float vl[4] = {__shfl(v[0], l, 64), __shfl(v[1], l, 64), __shfl(v[2], l, 64),
                               __shfl(v[3], l, 64)};
          int id = -1, lastl = -1;
          for (int q = 0; q < 4; ++q) {
            if (vl[q] > 0.f) lastl = blk * 256 + 4 * l + q;
            if (vl[q] > 0.f && r + vl[q] > goal) { id = blk * 256 + 4 * l + q; break; }
            r += vl[q];
          }
          found = id >= 0 ? id : lastl;
        }
        run += __shfl(x, 63, 64);
      }
      if (lane == 0) s_pick[1] = found >= 0 ? found : last;
    }
  }
  __syncthreads();
  return s_pick[1];
}

struct VerifyChainArgs {
  int K, V;
  float inv_t;                   // 0: greedy
  const float *tl, *dl;          // [B, K+1, V], [B, K, V]
  const RowStat *ts, *ds;        // [B*(K+1)][VSPLIT], [B*K][VSPLIT]
  const int32_t *drafts;         // [B, K]
  const float *u;                // [B, K+1]
  int32_t *n_acc, *next;         // [B]
  uint32_t *err;
};

constexpr int VER_MAXK = 64;     // drafts per sequence (max_steps <= 63)

__global__ __launch_bounds__(DRAW_THREADS) void k_verify_chain(VerifyChainArgs a) {
  __shared__ float s_wave[DRAW_SHARED];
  __shared__ int s_pick[3];
  __shared__ RowSum s_t[VER_MAXK + 1], s_d[VER_MAXK];
  __shared__ int s_x[VER_MAXK];
  __shared__ float s_lt[VER_MAXK], s_ld[VER_MAXK];
  __shared__ int s_n, s_mode;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int K = a.K, V = a.V;
  const bool sampled = a.inv_t > 0.f;
  // row statistics and the drafts' own logits, in parallel
  if (tid <= K) s_t[tid] = merge_row(a.ts + ((size_t)b * (K + 1) + tid) * VSPLIT);
  if (sampled && tid < K) s_d[tid] = merge_row(a.ds + ((size_t)b * K + tid) * VSPLIT);
  if (tid < K) {
    const int x = a.drafts[(size_t)b * K + tid];
    const bool ok = x >= 0 && x < V;
    s_x[tid] = ok ? x : -1;
    if (!ok) atomicOr(a.err, ERRF_TOKEN);
    if (sampled) {
      s_lt[tid] = ok ? a.tl[((size_t)b * (K + 1) + tid) * V + x] : 0.f;
      s_ld[tid] = ok ? a.dl[((size_t)b * K + tid) * V + x] : 0.f;
    }
  }
  __syncthreads();
  if (tid == 0) {
    int n = 0, mode = 0;         // mode 0: draw from p_target row n; 1: the residual at n
    for (; n < K; ++n) {
      const int x = s_x[n];
      if (x < 0) break;          // an invalid draft is never kept
      if (!sampled) {
        if (s_t[n].arg != x) break;
      } else {
        const float pt = expf(s_lt[n] * a.inv_t - s_t[n].M) / s_t[n].S;
        const float pd = expf(s_ld[n] * a.inv_t - s_d[n].M) / s_d[n].S;
        const float r = a.u[(size_t)b * (K + 1) + n];
        if (!(r < fminf(1.f, pt / pd))) { mode = 1; break; }
      }
    }
    s_n = n;
    s_mode = mode;
  }
  __syncthreads();
  const int n = s_n;
  int next;
  if (!sampled) {
    next = s_t[n].arg;
  } else {
    const float it = a.inv_t, u = a.u[(size_t)b * (K + 1) + K];
    const RowSum t = s_t[n];
    const float *trow = a.tl + ((size_t)b * (K + 1) + n) * V;
    // V is a multiple of 16, so ids i0..i0+3 are all inside or all past the
    // row; the loads are unconditional (clamped to id 0, masked), so that a
    // batch of blocks keeps its loads in flight together
    auto lt = [&](int i0) {   // the target row's values (clamped past the row)
      DrawRaw r;
      r.x = *(const f32x4 *)(trow + (i0 < V ? i0 : 0));
      r.y = r.x;
      return r;
    };
    auto wt = [&](const DrawRaw &r, int i0, float (&v)[4]) {   // p_target up to its normaliser
      const bool in = i0 < V;
      v[0] = in ? expf(r.x.x * it - t.M) : 0.f; v[1] = in ? expf(r.x.y * it - t.M) : 0.f;
      v[2] = in ? expf(r.x.z * it - t.M) : 0.f; v[3] = in ? expf(r.x.w * it - t.M) : 0.f;
    };
    if (s_mode == 1) {   // max(0, p_target - p_draft) at the rejected position
      const RowSum d = s_d[n];
      const float *drow = a.dl + ((size_t)b * K + n) * V;
      const float ist = 1.f / t.S, isd = 1.f / d.S;
      auto lr = [&](int i0) {   // both rows' values (clamped past the row)
        DrawRaw r;
        r.x = *(const f32x4 *)(trow + (i0 < V ? i0 : 0));
        r.y = *(const f32x4 *)(drow + (i0 < V ? i0 : 0));
        return r;
      };
      auto wr = [&](const DrawRaw &r, int i0, float (&v)[4]) {
        const bool in = i0 < V;
        const float p[4] = {r.x.x, r.x.y, r.x.z, r.x.w}, q4[4] = {r.y.x, r.y.y, r.y.z, r.y.w};
        for (int q = 0; q < 4; ++q)
          v[q] = in ? fmaxf(0.f, expf(p[q] * it - t.M) * ist - expf(q4[q] * it - d.M) * isd) : 0.f;
      };
      next = draw_ids(V, u, lr, wr, s_wave, s_pick);
      if (next < 0) next = draw_ids(V, u, lt, wt, s_wave, s_pick);   // identical distributions
    } else {
      next = draw_ids(V, u, lt, wt, s_wave, s_pick);
    }
  }
  if (tid == 0) {
    a.n_acc[b] = n;
    a.next[b] = next;
  }
}

struct VerifyTreeArgs {
  int nodes, V;
  const RowStat *ts;             // [B*(nodes+1)][VSPLIT]
  const int32_t *tokens, *parent;   // [B, nodes]
  int32_t *n_acc, *path, *next;  // [B], [B, nodes], [B]
};

// one wave per tree; lane j holds node j (v <= 64), so each step of the walk
// is one ballot over the nodes: the first child of the current position
// whose token is the target's choice there
__global__ __launch_bounds__(64) void k_verify_tree(VerifyTreeArgs a) {
  __shared__ int s_arg[MAX_VERIFY_NODES + 1];
  const int b = blockIdx.x, lane = threadIdx.x, v = a.nodes;
  for (int j = lane; j <= v; j += 64) s_arg[j] = merge_row(a.ts + ((size_t)b * (v + 1) + j) * VSPLIT).arg;
  const int tok = lane < v ? a.tokens[(size_t)b * v + lane] : -1;
  const int par = lane < v ? a.parent[(size_t)b * v + lane] : -2;
  __syncthreads();
  int at = -1, n = 0;
  int32_t *path = a.path + (size_t)b * v;
  while (n < v) {   // a path has at most v nodes (also bounds a malformed parent table)
    const int want = s_arg[at + 1];
    const unsigned long long m = __ballot(lane < v && par == at && tok == want);
    if (!m) break;
    at = __ffsll((long long)m) - 1;
    if (lane == 0) path[n] = at;
    ++n;
  }
  for (int j = n + lane; j < v; j += 64) path[j] = -1;
  if (lane == 0) {
    a.n_acc[b] = n;
    a.next[b] = s_arg[at + 1];
  }
}

size_t verify_stats_bytes(int rows) { return (size_t)rows * VSPLIT * sizeof(RowStat); }

// ---------------------------------------------------------------------------
// Chain verification that allocates nothing, for callers that cannot call
// hipMalloc (graph capture, serving loops): the per-slice row statistics and
// the kernels' error word live in this file-scope device array, one copy per
// GPU, held until the process ends.  Its device address comes from
// hipGetSymbolAddress, once per device (in prism_create, or at the first
// call on a device); host code never passes the array's own name.
constexpr int VSTATIC_ROWS = 8192;   // logits rows statistics are kept for
constexpr size_t VSTATIC_BYTES = 256 + (size_t)VSTATIC_ROWS * VSPLIT * sizeof(RowStat);
static __device__ __align__(256) unsigned char scratch[VSTATIC_BYTES];

namespace {
constexpr int SCRATCH_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[SCRATCH_DEVICES] = {};

prism_status static_fail(prism_status st, const char *fmt, ...) {
  char buf[256];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  set_global_error(buf);
  return st;
}
}  // namespace

hipError_t verify_scratch(void **out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= SCRATCH_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace prism

extern "C" prism_status prism_verify_chain_static(int32_t vocab, int32_t batch, int32_t K,
                                                  float temperature, const float *d_target_logits,
                                                  const float *d_draft_logits,
                                                  const int32_t *d_draft_tokens,
                                                  const float *d_uniforms, int32_t *d_n_accepted,
                                                  int32_t *d_next_token, void *stream) {
  using namespace prism;
  if (vocab < 16 || vocab % 16)
    return static_fail(PRISM_ERR_SHAPE, "vocab %d must be a positive multiple of 16", vocab);
  if (batch < 1 || K < 1 || K >= VER_MAXK)
    return static_fail(PRISM_ERR_INVALID_ARG, "batch %d / K %d out of range (K < %d)", batch,
                       K, VER_MAXK);
  if (!(temperature >= 0.f) || (temperature > 0.f && !std::isfinite(1.f / temperature)))
    return static_fail(PRISM_ERR_INVALID_ARG, "temperature %g", (double)temperature);
  const bool sampled = temperature > 0.f;
  if (!d_target_logits || !d_draft_tokens || !d_n_accepted || !d_next_token ||
      (sampled && (!d_draft_logits || !d_uniforms)))
    return static_fail(PRISM_ERR_INVALID_ARG, "NULL pointer");
  const long rows = (long)batch * (K + 1) + (sampled ? (long)batch * K : 0);
  if (rows > VSTATIC_ROWS)
    return static_fail(PRISM_ERR_SHAPE,
                       "%ld logits rows exceed the %d the static scratch holds "
                       "(batch * (K + 1), plus batch * K when sampled)",
                       rows, VSTATIC_ROWS);
  void *base = nullptr;
  hipError_t e = verify_scratch(&base);
  if (e != hipSuccess)
    return static_fail(PRISM_ERR_HIP, "hipGetSymbolAddress: %s", hipGetErrorString(e));
  uint32_t *err = (uint32_t *)base;                    // written by the kernels, never read
  void *stats = (unsigned char *)base + 256;
  launch_verify_chain(batch, K, vocab, sampled ? 1.f / temperature : 0.f, d_target_logits,
                      d_draft_logits, d_draft_tokens, d_uniforms, d_n_accepted, d_next_token,
                      stats, err, (hipStream_t)stream);
  e = hipGetLastError();
  if (e != hipSuccess) return static_fail(PRISM_ERR_HIP, "launch: %s", hipGetErrorString(e));
  return PRISM_OK;
}

namespace prism {

void launch_verify_chain(int B, int K, int V, float inv_t, const float *tl, const float *dl,
                         const int32_t *drafts, const float *u, int32_t *n_acc, int32_t *next,
                         void *stats, uint32_t *err, hipStream_t s) {
  RowStat *ts = (RowStat *)stats;
  RowStat *ds = ts + (size_t)B * (K + 1) * VSPLIT;
  const float it = inv_t > 0.f ? inv_t : 1.f;
  if (inv_t > 0.f) {   // sampled: the target and draft rows' softmax statistics
    hipLaunchKernelGGL(k_rows_stats<true>, dim3(VSPLIT, B * (K + 1)), dim3(256), 0, s, tl, V, it, ts);
    hipLaunchKernelGGL(k_rows_stats<true>, dim3(VSPLIT, B * K), dim3(256), 0, s, dl, V, it, ds);
  } else {             // greedy: the target rows' arg-max only
    hipLaunchKernelGGL(k_rows_stats<false>, dim3(VSPLIT, B * (K + 1)), dim3(256), 0, s, tl, V, it, ts);
  }
  VerifyChainArgs a{K, V, inv_t, tl, dl, ts, ds, drafts, u, n_acc, next, err};
  hipLaunchKernelGGL(k_verify_chain, dim3(B), dim3(DRAW_THREADS), 0, s, a);
}

void launch_verify_tree(int B, int nodes, int V, const float *tl, const int32_t *tokens,
                        const int32_t *parent, int32_t *n_acc, int32_t *path, int32_t *next,
                        void *stats, hipStream_t s) {
  RowStat *ts = (RowStat *)stats;
  hipLaunchKernelGGL(k_rows_stats<false>, dim3(VSPLIT, B * (nodes + 1)), dim3(256), 0, s, tl, V, 1.f, ts);
  VerifyTreeArgs a{nodes, V, ts, tokens, parent, n_acc, path, next};
  hipLaunchKernelGGL(k_verify_tree, dim3(B), dim3(64), 0, s, a);
}

}  // namespace prism
