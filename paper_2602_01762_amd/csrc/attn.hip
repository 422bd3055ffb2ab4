// Decode attention of the drafting step over the paged draft KV cache, with
// causal or tree visibility.
//
// Visibility of row r (sequence b, prior context L_b):
//   tree bits given:  slots [0, L_b)  plus  L_b + j for every set bit j
//   no tree bits:     slots [0, slot[r]]  (causal)
// Split-KV: a workgroup takes one (row, KV head, chunk of 64*nsub slots) and
// all g = n_q/n_kv query heads that share the KV head, walking the chunk in
// 64-slot steps with an online softmax.  K and V rows are read as whole
// contiguous rows (4 threads per K row, d/8 threads per V row).  The partial
// states (max, sum, unnormalised output) are merged by a second kernel in
// chunk order, so the result does not depend on scheduling.  The merged
// output is written as the W_o operand (hi/lo pair for bf16).
#include "device.h"

namespace prism {

constexpr int ATT_S = ATT_STEP;  // slots per step
constexpr int ATT_MAXG = 8;      // query heads per KV head
constexpr int ATT_MAXGD = 1024;  // g * d
constexpr int ATT_MAXVS = 8;     // slots per thread in P.V: 64 / (256 / (d / 8)) for d <= 256
constexpr int ATT_MAXCH = ATT_MAX_CHUNKS;  // chunks per row merged by the combine kernel

struct AttnArgs {
  const float *q;             // [R, nq*d] fp32, RoPE applied
  const int32_t *seq, *slot;
  const uint64_t *bits;
  KvArgs kv;
  int R, nq, nkv, d, nch, nsub;
  int grp;                    // rows per workgroup of the grouped MFMA kernel (one sequence's tree rows)
  int rps;                    // > 0: rows come in runs of rps rows of one tree each, grouped from
                              // each run's first row (its last group may be shorter)
  float scale;
  float *pm, *pl, *po;        // [R, nq, nch] / [R, nq, nch, d]
  ActOut o;                   // [R, nq*d]
  uint32_t *err;
};

__device__ __forceinline__ bool row_range(const AttnArgs &a, int r, int &b, int &L, int &prefix,
                                          int &total, uint64_t &bits) {
  // the row's own entries are loaded together; only the tree's context
  // length depends on the sequence index
  b = a.seq[r];
  const int slot = a.bits ? 0 : a.slot[r];
  const uint64_t bw = a.bits ? a.bits[r] : 0ull;
  L = prefix = total = 0;
  bits = 0ull;
  if (b < 0 || b >= a.kv.n_seq) return false;
  if (a.bits) {
    L = a.kv.ctx_lens[b];
    bits = bw;
    prefix = L;
    total = L + (bits ? 64 - __clzll((long long)bits) : 0);
  } else {   // causal: the slot alone bounds the range (no context-length load)
    prefix = slot + 1;
    total = prefix;
  }
  return true;
}

template <typename T>
__device__ __forceinline__ void load8(const T *p, float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    const u32x4 raw = *(const u32x4 *)p;
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  } else {
    const f32x4 x0 = *(const f32x4 *)p, x1 = *(const f32x4 *)(p + 4);
    v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w;
    v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_attn_partial(AttnArgs a) {
  const int c = blockIdx.z, j = blockIdx.x, r = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  int b, L, prefix, total;
  uint64_t bits;
  if (!row_range(a, r, b, L, prefix, total, bits)) {
    if (c == 0 && j == 0 && tid == 0) atomicOr(a.err, ERRF_CAPACITY);
    return;
  }
  const int tbeg = c * ATT_S * a.nsub;
  if (tbeg >= total) return;
  const int d = a.d, g = a.nq / a.nkv;

  __shared__ float qs[ATT_MAXGD];
  __shared__ float sc[ATT_MAXG][ATT_S];
  __shared__ long offs[ATT_S];
  __shared__ float m_run[ATT_MAXG], l_run[ATT_MAXG], alpha[ATT_MAXG];
  __shared__ float red[4][ATT_MAXGD];

  const float *q = a.q + (size_t)r * a.nq * d + (size_t)j * g * d;
  for (int e = tid; e < g * d; e += 256) qs[e] = q[e];
  if (tid < ATT_MAXG) {
    m_run[tid] = -INFINITY;
    l_run[tid] = 0.f;
  }
  // P.V thread layout: 8 dims per thread, dg = dim group, tg = slot group
  const int ndg = d >> 3, G = 256 / ndg;
  const int dg = tid % ndg, tg = tid / ndg;
  float acc[ATT_MAXG][8];
#pragma unroll
  for (int h = 0; h < ATT_MAXG; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[h][i] = 0.f;

  for (int sub = 0; sub < a.nsub; ++sub) {
    const int t0 = tbeg + sub * ATT_S;
    if (t0 >= total) break;                // uniform across the workgroup
    const int n_here = min(ATT_S, total - t0);
    if (tid < ATT_S) {
      const int t = t0 + tid;
      long off = -1;
      if (tid < n_here && (t < prefix || (a.bits && t >= L && ((bits >> (t - L)) & 1ull)))) {
        const int bi = t / a.kv.bs;
        const int blk = bi < a.kv.mbps ? a.kv.block_table[(size_t)b * a.kv.mbps + bi] : -1;
        // pool layout [block, kv head, slot in block, d]
        if (blk < 0 || blk >= a.kv.n_blocks) atomicOr(a.err, ERRF_CAPACITY);
        else off = ((long)blk * a.nkv + j) * a.kv.bs * d + (long)(t % a.kv.bs) * d;
      }
      offs[tid] = off;
    }
    __syncthreads();
    // V rows of this thread's slots, fetched together with the K rows
    u32x4 vraw[ATT_MAXVS][sizeof(T) == 2 ? 1 : 2];
    if (tg < G) {
#pragma unroll
      for (int i = 0; i < ATT_MAXVS; ++i) {
        const int ts = tg + i * G;
        const long off = ts < n_here ? offs[ts] : -1;
        if (off >= 0) {
          const u32x4 *vp = (const u32x4 *)((const T *)a.kv.v_pool + off + dg * 8);
          vraw[i][0] = vp[0];
          if (sizeof(T) == 4) vraw[i][sizeof(T) == 2 ? 0 : 1] = vp[1];
        }
      }
    }
    // scores: 4 threads per slot, d/4 dims each
    {
      const int ts = tid >> 2, part = tid & 3;
      const long off = offs[ts];
      float s[ATT_MAXG];
#pragma unroll
      for (int h = 0; h < ATT_MAXG; ++h) s[h] = 0.f;
      if (off >= 0) {
        const int dq = d >> 2;
        const T *kp = (const T *)a.kv.k_pool + off + part * dq;
        for (int e = 0; e < dq; e += 8) {
          float kv[8];
          load8<T>(kp + e, kv);
#pragma unroll
          for (int h = 0; h < ATT_MAXG; ++h)
            if (h < g) {
              const float *qh = qs + h * d + part * dq + e;
#pragma unroll
              for (int i = 0; i < 8; ++i) s[h] += qh[i] * kv[i];
            }
        }
      }
#pragma unroll
      for (int h = 0; h < ATT_MAXG; ++h) {
        s[h] += __shfl_xor(s[h], 1, 64);
        s[h] += __shfl_xor(s[h], 2, 64);
      }
      if (part == 0) {
#pragma unroll
        for (int h = 0; h < ATT_MAXG; ++h)
          if (h < g) sc[h][ts] = off >= 0 ? s[h] * a.scale : -INFINITY;
      }
    }
    __syncthreads();
    // online softmax update: wave w takes heads w, w + 4
    for (int h = wave; h < g; h += 4) {
      const float v = sc[h][lane];
      const float mo = m_run[h];
      const float mn = fmaxf(mo, wave_max(v));
      const float p = v == -INFINITY ? 0.f : expf(v - mn);
      const float al = mo == -INFINITY ? 0.f : expf(mo - mn);
      const float ls = wave_sum(p);
      sc[h][lane] = p;
      if (lane == 0) {
        alpha[h] = al;
        l_run[h] = l_run[h] * al + ls;
        m_run[h] = mn;
      }
    }
    __syncthreads();
    // P V
#pragma unroll
    for (int h = 0; h < ATT_MAXG; ++h)
      if (h < g) {
        const float al = alpha[h];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[h][i] *= al;
      }
    if (tg < G) {
#pragma unroll
      for (int vi = 0; vi < ATT_MAXVS; ++vi) {
        const int ts = tg + vi * G;
        if (ts >= n_here || offs[ts] < 0) continue;
        float vv[8];
        if constexpr (sizeof(T) == 2) {
          const uint32_t w4[4] = {vraw[vi][0].x, vraw[vi][0].y, vraw[vi][0].z, vraw[vi][0].w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            vv[2 * i] = __uint_as_float(w4[i] << 16);
            vv[2 * i + 1] = __uint_as_float(w4[i] & 0xffff0000u);
          }
        } else {
          const u32x4 x0 = vraw[vi][0], x1 = vraw[vi][sizeof(T) == 2 ? 0 : 1];
          vv[0] = __uint_as_float(x0.x); vv[1] = __uint_as_float(x0.y);
          vv[2] = __uint_as_float(x0.z); vv[3] = __uint_as_float(x0.w);
          vv[4] = __uint_as_float(x1.x); vv[5] = __uint_as_float(x1.y);
          vv[6] = __uint_as_float(x1.z); vv[7] = __uint_as_float(x1.w);
        }
#pragma unroll
        for (int h = 0; h < ATT_MAXG; ++h)
          if (h < g) {
            const float p = sc[h][ts];
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[h][i] += p * vv[i];
          }
      }
    }
    __syncthreads();
  }
  // reduce the slot groups: lanes of one wave sharing dg (butterfly over the
  // slot-group bits of the lane index), then the waves in order
  for (int o = ndg; o < 64; o <<= 1)
#pragma unroll
    for (int h = 0; h < ATT_MAXG; ++h)
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[h][i] += __shfl_xor(acc[h][i], o, 64);
  if (lane < ndg && tg < G) {
#pragma unroll
    for (int h = 0; h < ATT_MAXG; ++h)
      if (h < g)
#pragma unroll
        for (int i = 0; i < 8; ++i) red[wave][h * d + dg * 8 + i] = acc[h][i];
  }
  __syncthreads();
  const int nw = (G * ndg + 63) / 64;
  for (int e = tid; e < g * d; e += 256) {
    float sum = 0.f;
    for (int w = 0; w < nw; ++w) sum += red[w][e];
    const int h = e / d, dim = e % d;
    a.po[(((size_t)r * a.nq + j * g + h) * a.nch + c) * d + dim] = sum;
  }
  if (tid < g) {
    const size_t pi = ((size_t)r * a.nq + j * g + tid) * a.nch + c;
    a.pm[pi] = m_run[tid];
    a.pl[pi] = l_run[tid];
  }
}


// MFMA variant for bf16 caches.  Each wave takes 16 slots of every 64-slot
// step: the scores of those slots against all g query heads are one 16x16
// MFMA tile (K rows as the A operand, q as the B operand carried as a
// hi/lo bf16 pair), the online softmax runs per head with lane shuffles, and
// P.V is a 16x16x16 MFMA per 16 dims with P (hi/lo pair) straight from the
// score layout and V transposed through the wave's own LDS tile.  The
// chunk's block-table entries are staged in LDS once, and each wave loads
// the K/V rows of its next step before it computes the current one, so the
// waves stream independently.  Each wave keeps its own softmax state; the 4
// waves merge in LDS at the end and write the same per-chunk partials as the
// VALU kernel.
//
// Grouped form (GRP, tree rows): a workgroup takes grp rows of one sequence,
// and score column col is (row col / g of the group, head col % g), so the
// 16 columns hold grp * g query rows instead of g.  The rows share the prior
// context [0, L) and differ only in which of the 64 tree slots after it they
// see, so each context slot's K/V is read once for the group instead of once
// per row.  A slot is loaded if any row of the group sees it and masked per
// column; the partials are written per row as in the ungrouped form.
typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return f2bf(lo) | (f2bf(hi) << 16);
}

constexpr int ATT_MAXSUB = ATT_MAX_SUB;    // 64-slot steps per workgroup

// DK: head_dim / 32; NTL: K/V rows read with streaming (nontemporal) loads;
// GRP: grouped form (a.grp rows of one sequence per workgroup, tree bits)
template <int DK, bool NTL, bool GRP>
__global__ __launch_bounds__(256) void k_attn_mfma(AttnArgs a) {
  constexpr int ATT_MAXDK = DK, ATT_MAXDT = 2 * DK;
  const int c = blockIdx.z, j = blockIdx.x;
  int gs = GRP ? a.grp : 1;
  int r = blockIdx.y * gs;                   // the workgroup's (first) row
  if (GRP && a.rps > 0) {                    // runs of rps rows: ceil(rps / grp) groups each
    const int gpr = (a.rps + a.grp - 1) / a.grp, gi = blockIdx.y % gpr;
    r = blockIdx.y / gpr * a.rps + gi * a.grp;
    gs = min(a.grp, a.rps - gi * a.grp);
  }
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, q4 = lane >> 4;
  int b, L, prefix, total;
  uint64_t bits;
  if (!row_range(a, r, b, L, prefix, total, bits) || (GRP && !a.bits)) {
    if (c == 0 && j == 0 && tid == 0) atomicOr(a.err, ERRF_CAPACITY);
    return;
  }
  const int g = a.nq / a.nkv;
  // column col: query head col (ungrouped), or row r + col / g, head col % g;
  // its own tree bits (grouped)
  bool cvalid = col < g;
  uint64_t cbits = 0ull;
  if constexpr (GRP) {
    // every row of the group must belong to the row-r sequence (the launcher
    // groups the rows of one tree); another row's columns stay masked
    uint64_t ub = 0ull;
    for (int i = 0; i < gs; ++i) {
      if (a.seq[r + i] == b) ub |= a.bits[r + i];
      else if (c == 0 && j == 0 && tid == 0) atomicOr(a.err, ERRF_ROWS);
    }
    const int rc = r + col / g;
    cvalid = col < gs * g && a.seq[rc < r + gs ? rc : r] == b;
    cbits = cvalid ? a.bits[rc] : 0ull;
    bits = ub;                                 // slots loaded: seen by any row
    total = L + (ub ? 64 - __clzll((long long)ub) : 0);
  }
  const int span = ATT_S * a.nsub;
  const int tbeg = c * span;
  if (tbeg >= total) return;                 // uniform across the workgroup
  // the launcher instantiates DK = d / 32, so every head-dim loop below is full
  constexpr int d = 32 * DK;
  constexpr int NCOLD = GRP ? 16 * d : ATT_MAXGD;   // merge buffer: columns x dims
  const int bs = a.kv.bs;

  __shared__ bf16_t vt[4][32 * DK][16];     // per wave: V tile as [dim][slot]
  __shared__ float mg_m[4][16], mg_l[4][16];
  __shared__ float mg_o[4][NCOLD];
  __shared__ int s_blk[ATT_S * ATT_MAXSUB];  // physical blocks of the chunk's slots

  // block-table entries of the chunk (at most one per slot)
  const int tend = min(total, tbeg + span);
  const int bfirst = tbeg / bs;
  const int nblk = (tend - 1) / bs - bfirst + 1;
  for (int i = tid; i < nblk; i += 256) {
    const int bi = bfirst + i;
    s_blk[i] = bi < a.kv.mbps ? a.kv.block_table[(size_t)b * a.kv.mbps + bi] : -1;
  }

  // q of head `col` as the B operand (k = dims 32 kk + 8 q4 .. +7), hi/lo
  u32x4 qh[ATT_MAXDK], ql[ATT_MAXDK];
#pragma unroll
  for (int kk = 0; kk < ATT_MAXDK; ++kk) {
    qh[kk] = ql[kk] = u32x4{0, 0, 0, 0};
    if (cvalid) {
      const int rq = GRP ? r + col / g : r, hq = GRP ? col % g : col;
      const float *qp = a.q + (size_t)rq * a.nq * d + (size_t)(j * g + hq) * d + 32 * kk + 8 * q4;
      const f32x4 x0 = *(const f32x4 *)qp, x1 = *(const f32x4 *)(qp + 4);
      const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
      float hi[8], lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        hi[e] = bf2f(f2bf(x[e]));
        lo[e] = x[e] - hi[e];
      }
      qh[kk] = u32x4{pack2(hi[0], hi[1]), pack2(hi[2], hi[3]), pack2(hi[4], hi[5]), pack2(hi[6], hi[7])};
      ql[kk] = u32x4{pack2(lo[0], lo[1]), pack2(lo[2], lo[3]), pack2(lo[4], lo[5]), pack2(lo[6], lo[7])};
    }
  }
  __syncthreads();                            // s_blk

  // cache offset of slot t for this KV head, or -1 (not visible / no block)
  auto slot_off = [&](int t) -> long {
    if (t >= tend || !(t < prefix || (a.bits && t >= L && ((bits >> (t - L)) & 1ull)))) return -1;
    const int blk = s_blk[t / bs - bfirst];
    // pool layout [block, kv head, slot in block, d]
    if (blk < 0 || blk >= a.kv.n_blocks) {
      atomicOr(a.err, ERRF_CAPACITY);
      return -1;
    }
    return ((long)blk * a.nkv + j) * bs * d + (long)(t % bs) * d;
  };
  // K/V rows of one slot.  The loads are unconditional (an invisible slot
  // reads slot 0 of block 0 instead, and its values are masked at use), so
  // that the compiler can count them exactly and the next step's loads stay
  // in flight while the current step computes.
  auto load_kv = [&](long off, u32x4 (&ka)[ATT_MAXDK], u32x4 (&va)[ATT_MAXDK]) {
    const long o = off >= 0 ? off : 0;
#pragma unroll
    for (int kk = 0; kk < ATT_MAXDK; ++kk) {
      const u32x4 *kp = (const u32x4 *)((const bf16_t *)a.kv.k_pool + o + 32 * kk + 8 * q4);
      const u32x4 *vp = (const u32x4 *)((const bf16_t *)a.kv.v_pool + o + 32 * kk + 8 * q4);
      ka[kk] = NTL ? __builtin_nontemporal_load(kp) : *kp;
      va[kk] = NTL ? __builtin_nontemporal_load(vp) : *vp;
    }
  };

  float m_run = -INFINITY, l_run = 0.f;      // softmax state of column `col`
  f32x4 o[ATT_MAXDT];                         // O[head 4 q4 + i][dim 16 dt + col]
#pragma unroll
  for (int dt = 0; dt < ATT_MAXDT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One 64-slot step of the wave's 16 slots tb + [0, 16) (tb = t0 + 16 wave):
  // lane (col, q4) holds the K/V rows of slot tb + col (offset off, -1 =
  // invisible).
  auto step = [&](int tb, long off, const u32x4 (&ka)[ATT_MAXDK], const u32x4 (&va)[ATT_MAXDK]) {
    // scores S[slot 4 q4 + i][head col]
    f32x4 sc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < ATT_MAXDK; ++kk) {
      sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka[kk]),
                                                    __builtin_bit_cast(bf16x8, qh[kk]), sc, 0, 0, 0);
      sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ka[kk]),
                                                    __builtin_bit_cast(bf16x8, ql[kk]), sc, 0, 0, 0);
    }
    const bool vis = off >= 0;
    // visibility of every slot of the tile (bit s: lane s, i.e. slot s, q4 = 0)
    const uint64_t vmask = __ballot(vis);
    float sv[4] = {sc.x, sc.y, sc.z, sc.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bool v = (vmask >> (4 * q4 + i)) & 1ull;
      if constexpr (GRP) {   // the column's row: the prior context and its own tree slots
        const int sh = tb + 4 * q4 + i - L;
        v = v && cvalid && (sh < 0 || (sh < 64 && ((cbits >> (sh & 63)) & 1ull)));
      }
      sv[i] = v ? sv[i] * a.scale : -INFINITY;
    }
    // online softmax of column col over these 16 slots (lanes col, col^16, ...)
    float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    mx = fmaxf(mx, xor16_f(mx));
    mx = fmaxf(mx, xor32_f(mx));
    const float mn = fmaxf(m_run, mx);
    // alpha = 1 while nothing has accumulated (O and l are still zero)
    const float al = m_run == -INFINITY ? 1.f : expf(m_run - mn);
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = sv[i] == -INFINITY ? 0.f : expf(sv[i] - mn);
    float ps = (p[0] + p[1]) + (p[2] + p[3]);
    ps += xor16_f(ps);
    ps += xor32_f(ps);
    l_run = l_run * al + ps;
    m_run = mn;
    // V tile -> LDS as [dim][slot] (zero rows for invisible slots)
#pragma unroll
    for (int kk = 0; kk < ATT_MAXDK; ++kk) {
      const uint32_t w4[4] = {vis ? va[kk].x : 0u, vis ? va[kk].y : 0u, vis ? va[kk].z : 0u,
                              vis ? va[kk].w : 0u};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vt[wave][32 * kk + 8 * q4 + 2 * e][col] = (bf16_t)(w4[e] & 0xffffu);
        vt[wave][32 * kk + 8 * q4 + 2 * e + 1][col] = (bf16_t)(w4[e] >> 16);
      }
    }
    wave_lds_sync();
    // rescale O rows (columns 4 q4 + i) by their alpha, which is exactly 1
    // for every column once its running max stops moving (most steps of a
    // long context): the wave then skips the broadcasts and multiplies
    if (__ballot(al != 1.f)) {
      float ah[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) ah[i] = __shfl(al, 4 * q4 + i, 64);
#pragma unroll
      for (int dt = 0; dt < ATT_MAXDT; ++dt) {
        o[dt].x *= ah[0]; o[dt].y *= ah[1]; o[dt].z *= ah[2]; o[dt].w *= ah[3];
      }
    }
    // O += P V
    float ph[4], pl[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ph[i] = bf2f(f2bf(p[i]));
      pl[i] = p[i] - ph[i];
    }
    const s16x4 pah = __builtin_bit_cast(s16x4, uint2{pack2(ph[0], ph[1]), pack2(ph[2], ph[3])});
    const s16x4 pal = __builtin_bit_cast(s16x4, uint2{pack2(pl[0], pl[1]), pack2(pl[2], pl[3])});
#pragma unroll
    for (int dt = 0; dt < ATT_MAXDT; ++dt) {
      const s16x4 vb = *(const s16x4 *)&vt[wave][16 * dt + col][4 * q4];
      o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pah, vb, o[dt], 0, 0, 0);
      o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pal, vb, o[dt], 0, 0, 0);
    }
    wave_lds_sync();                          // reads done before the next step's writes
  };
  // Steps in pairs over two register sets: each step's successor is already
  // in flight while it computes, with no copies between the sets.
  const int slot0 = tbeg + 16 * wave + col;  // this lane's slot in the first step
  long off0 = slot_off(slot0), off1 = -1;
  u32x4 k0[ATT_MAXDK], v0[ATT_MAXDK], k1[ATT_MAXDK], v1[ATT_MAXDK];
  load_kv(off0, k0, v0);
  for (int sub = 0; sub < a.nsub; sub += 2) {
    const int t0 = tbeg + sub * ATT_S;
    if (t0 >= tend) break;                    // uniform
    off1 = sub + 1 < a.nsub ? slot_off(slot0 + (sub + 1) * ATT_S) : -1;
    load_kv(off1, k1, v1);
    step(t0 + 16 * wave, off0, k0, v0);
    if (sub + 1 >= a.nsub || t0 + ATT_S >= tend) break;   // uniform
    off0 = sub + 2 < a.nsub ? slot_off(slot0 + (sub + 2) * ATT_S) : -1;
    load_kv(off0, k0, v0);
    step(t0 + ATT_S + 16 * wave, off1, k1, v1);
  }
  // merge the 4 waves' states and write this chunk's partials
  const int ncol = GRP ? gs * g : g;
  if (q4 == 0) {
    mg_m[wave][col] = m_run;
    mg_l[wave][col] = l_run;
  }
#pragma unroll
  for (int dt = 0; dt < ATT_MAXDT; ++dt) {
    const float ov[4] = {o[dt].x, o[dt].y, o[dt].z, o[dt].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * q4 + i;
      if (h < ncol) mg_o[wave][h * d + 16 * dt + col] = ov[i];
    }
  }
  __syncthreads();
  for (int e = tid; e < ncol * d; e += 256) {
    const int h = e / d, dim = e % d;        // h: column
    const int rr = GRP ? r + h / g : r, hh = GRP ? h % g : h;
    if (GRP && a.seq[rr] != b) continue;     // another sequence's row (flagged above)
    float M = -INFINITY;
    for (int w = 0; w < 4; ++w) M = fmaxf(M, mg_m[w][h]);
    float lsum = 0.f, osum = 0.f;
    for (int w = 0; w < 4; ++w) {
      const float wt = mg_m[w][h] == -INFINITY ? 0.f : expf(mg_m[w][h] - M);
      lsum += mg_l[w][h] * wt;
      osum += mg_o[w][e] * wt;
    }
    const size_t pi = ((size_t)rr * a.nq + j * g + hh) * a.nch + c;
    a.po[pi * d + dim] = osum;
    if (dim == 0) {
      a.pm[pi] = M;
      a.pl[pi] = lsum;
    }
  }
}

constexpr int CMB_PRE = 24;   // partial-output loads per thread issued before the softmax stats
template <typename T>
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs a) {
  __shared__ float wch[ATT_MAXCH], lch[ATT_MAXCH];
  __shared__ float red[256];
  __shared__ float sh[8];
  const int h = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  int b, L, prefix, total;
  uint64_t bits;
  row_range(a, r, b, L, prefix, total, bits);
  const int span = ATT_S * a.nsub;
  if (total > a.nch * span && h == 0 && tid == 0) atomicOr(a.err, ERRF_CAPACITY);
  const int nch = min((total + span - 1) / span, a.nch);
  const size_t base = ((size_t)r * a.nq + h) * a.nch;
  // output dims: thread = (dim, chunk group); its chunks are grp, grp + G, ...
  const int d = a.d, G = 256 / d;
  const int dim = tid % d, grp = tid / d;
  const bool has_grp = grp < G;
  // the first CMB_PRE partial outputs of this thread go out with the stats
  float pre[CMB_PRE];
#pragma unroll
  for (int j = 0; j < CMB_PRE; ++j) {
    const int c = grp + j * G;
    pre[j] = has_grp && c < nch ? a.po[(base + c) * d + dim] : 0.f;
  }
  // chunk weights exp(m_c - M) and the total sum, in fixed order
  float m = -INFINITY;
  for (int c = tid; c < nch; c += 256) {
    const float l = a.pl[base + c], mc = a.pm[base + c];
    lch[c] = l;
    wch[c] = mc;
    if (l > 0.f) m = fmaxf(m, mc);
  }
  const float M = block_max(m, sh);        // its barriers make lch / wch visible
  float lp = 0.f;
  for (int c = tid; c < nch; c += 256) {
    const float l = lch[c];
    const float w = l > 0.f ? expf(wch[c] - M) : 0.f;
    wch[c] = w;
    lp += l * w;
  }
  const float lsum = block_sum(lp, sh);   // ends with a barrier: wch is visible
  float o = 0.f;
  if (has_grp) {
#pragma unroll
    for (int j = 0; j < CMB_PRE; ++j) {
      const int c = grp + j * G;
      if (c < nch) o += pre[j] * wch[c];
    }
    for (int c = grp + CMB_PRE * G; c < nch; c += G) o += a.po[(base + c) * d + dim] * wch[c];
  }
  red[tid] = o;
  __syncthreads();
  if (grp != 0) return;
  float sum = 0.f;
  for (int gg = 0; gg < G; ++gg) sum += red[gg * d + dim];
  const float v = lsum > 0.f ? sum / lsum : 0.f;
  const size_t i = (size_t)r * a.o.ld + (size_t)h * d + dim;
  if constexpr (sizeof(T) == 2) {
    const uint32_t hb = f2bf(v);
    ((bf16_t *)a.o.hi)[i] = (bf16_t)hb;
    ((bf16_t *)a.o.lo)[i] = (bf16_t)f2bf(v - bf2f(hb));
  } else {
    ((float *)a.o.hi)[i] = v;
  }
}

// The same merge for passes of at most CMBW_MAX_CHUNKS chunks per row and
// head dims up to 256, by one wave per (row, query head), 4 per workgroup:
// lane c holds chunk c's statistics, two wave reductions (fixed order)
// replace the workgroup's barriers, and lane l adds, in chunk order, the
// partial outputs of dims l, l + 64, ...  (A workgroup per (row, head) with
// block reductions spent most of its time in its barriers when a row has 2-5
// chunks: 7808 workgroups for a 244-row scoring pass.)
constexpr int CMBW_MAX_CHUNKS = 8;
template <typename T>
__global__ __launch_bounds__(256) void k_attn_combine_w(AttnArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int h = blockIdx.x * 4 + wave, r = blockIdx.y;
  if (h >= a.nq) return;                      // whole waves; no barriers below
  int b, L, prefix, total;
  uint64_t bits;
  row_range(a, r, b, L, prefix, total, bits);
  const int span = ATT_S * a.nsub;
  if (total > a.nch * span && h == 0 && lane == 0) atomicOr(a.err, ERRF_CAPACITY);
  const int nch = min((total + span - 1) / span, a.nch);   // <= CMBW_MAX_CHUNKS (launcher)
  const size_t base = ((size_t)r * a.nq + h) * a.nch;
  const int d = a.d;
  // the partial outputs first, then the statistics they are weighted by
  float po[CMBW_MAX_CHUNKS][4];
#pragma unroll
  for (int c = 0; c < CMBW_MAX_CHUNKS; ++c)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int dim = lane + 64 * j;
      po[c][j] = c < nch && dim < d ? a.po[(base + c) * d + dim] : 0.f;
    }
  const float l = lane < nch ? a.pl[base + lane] : 0.f;
  const float mc = lane < nch ? a.pm[base + lane] : -INFINITY;
  const float M = wave_max(l > 0.f ? mc : -INFINITY);
  const float w = l > 0.f ? expf(mc - M) : 0.f;
  const float lsum = wave_sum(l * w);
  float o[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < CMBW_MAX_CHUNKS; ++c) {
    const float wc = readlane_f32(w, c);      // 0 past nch
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] += po[c][j] * wc;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int dim = lane + 64 * j;
    if (dim >= d) break;
    const float v = lsum > 0.f ? o[j] / lsum : 0.f;
    const size_t i = (size_t)r * a.o.ld + (size_t)h * d + dim;
    if constexpr (sizeof(T) == 2) {
      const uint32_t hb = f2bf(v);
      ((bf16_t *)a.o.hi)[i] = (bf16_t)hb;
      ((bf16_t *)a.o.lo)[i] = (bf16_t)f2bf(v - bf2f(hb));
    } else {
      ((float *)a.o.hi)[i] = v;
    }
  }
}

void launch_attention(bool bf16, int R, int nq, int nkv, int d, const float *q, const RowsIn &in,
                      const KvArgs &kv, int max_slots, int grp, int rps, float *pm, float *pl,
                      float *po, ActOut o, uint32_t *err, hipStream_t s) {
  AttnArgs a;
  a.q = q;
  a.seq = in.seq;
  a.slot = in.slot;
  a.bits = in.bits;
  a.kv = kv;
  a.R = R;
  a.nq = nq;
  a.nkv = nkv;
  a.d = d;
  a.scale = 1.0f / sqrtf((float)d);
  a.pm = pm;
  a.pl = pl;
  a.po = po;
  a.o = o;
  a.err = err;
  // grouped rows: tree rows (bits), bf16, head_dim 64 or 128, the group's
  // query rows within the 16 score columns, whole groups (or whole runs)
  const int g = nq / nkv;
  const bool grouped = grp > 1 && bf16 && in.bits && (d == 64 || d == 128) && grp * g <= 16 &&
                       (rps > 0 ? R % rps == 0 : R % grp == 0);
  a.grp = grouped ? grp : 1;
  a.rps = grouped ? rps : 0;
  const int units = !grouped ? R : rps > 0 ? R / rps * ((rps + grp - 1) / grp) : R / grp;
  // steps per workgroup for this pass's rows (or row groups)
  a.nsub = attention_nsub(units, nkv, max_slots);
  a.nch = attention_chunks(max_slots, a.nsub);
  // chunk index slowest: every row's first chunks are dispatched before any
  // row's later ones, so the last workgroups to start are the short tails
  dim3 g1(nkv, units, a.nch), g2(nq, R);
  // few chunks per row: the merge by one wave per (row, head)
  const bool small = a.nch <= CMBW_MAX_CHUNKS && d <= 256;
  const dim3 g2w((nq + 3) / 4, R);
  // K/V that one pass requests at capacity (R rows of max_slots slots):
  // beyond 1.5 times the 256 MiB infinity cache the rows are streamed with
  // nontemporal loads (70B batch 32, 539 MB: 5.917 -> 5.847 ms); below it
  // ordinary loads let the cache keep the prior context from one step to the
  // next (batch 16 paged, 269 MB at capacity and 151 MB on average:
  // nontemporal loads were 3.7% slower; the tree, 140 MB: 0.6% slower)
  const double kv_bytes = (double)units * max_slots * nkv * d * 2 * (bf16 ? 2 : 4);
  const bool ntl = kv_bytes > 1.5 * 256 * 1024 * 1024;
  if (bf16) {
    if (a.grp > 1) {
      if (d == 64) hipLaunchKernelGGL((k_attn_mfma<2, false, true>), g1, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_attn_mfma<4, false, true>), g1, dim3(256), 0, s, a);
    } else if (d == 64) {
      if (ntl) hipLaunchKernelGGL((k_attn_mfma<2, true, false>), g1, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_attn_mfma<2, false, false>), g1, dim3(256), 0, s, a);
    } else if (d == 128) {
      if (ntl) hipLaunchKernelGGL((k_attn_mfma<4, true, false>), g1, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_attn_mfma<4, false, false>), g1, dim3(256), 0, s, a);
    } else if (d == 256) {
      if (ntl) hipLaunchKernelGGL((k_attn_mfma<8, true, false>), g1, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_attn_mfma<8, false, false>), g1, dim3(256), 0, s, a);
    } else {
      hipLaunchKernelGGL(k_attn_partial<bf16_t>, g1, dim3(256), 0, s, a);
    }
    if (small) hipLaunchKernelGGL(k_attn_combine_w<bf16_t>, g2w, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_attn_combine<bf16_t>, g2, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(k_attn_partial<float>, g1, dim3(256), 0, s, a);
    if (small) hipLaunchKernelGGL(k_attn_combine_w<float>, g2w, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_attn_combine<float>, g2, dim3(256), 0, s, a);
  }
}

}  // namespace prism
