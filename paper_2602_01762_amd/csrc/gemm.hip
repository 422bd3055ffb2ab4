// Skinny products of the drafting step: Y[R, N] = X[R, K] . W[N, K]^T with
// R <= 64 rows (batch rows or tree nodes) and N, K in the thousands, and the
// LM head with its fused top-k partials.
//
// These products are HBM-bound (a weight byte feeds 2R flops), so the design
// is about streaming W: W is pre-tiled so that every wave-wide load is one
// contiguous KiB (see TiledMat), and each wave issues a batch of k-block
// loads (16 KiB in the GEMV, about 96 VGPRs of A and B in the MFMA loop)
// before it consumes them.
//  * 1-2 rows: VALU GEMV.  The workgroup stages its rows in LDS as fp32 and
//    each lane multiplies its weights by LDS-broadcast activations; up to 16
//    waves of one workgroup split K and meet in LDS in wave order.  The
//    one-row LM head streams four consecutive vocab tiles per wave instead.
//  * More rows: MFMA with 16 rows of W as the M side and 16 rows of X as the
//    N side; bf16 activations come as hi/lo pairs (two MFMAs per W fragment),
//    so the products see fp32-exact activations at no extra HBM traffic.
//    Wide products split K across the waves of a workgroup (LDS reduction);
//    narrow ones split it across workgroups, and a finish pass adds the
//    slices in order.  Every reduction has a fixed order (deterministic).
//
// Epilogues write whatever the next kernel needs: the fp32 residual row,
// (y * gain) as the next operand, partial sums of squares for the next
// RMSNorm (reduced by the consumer itself), the SwiGLU product, or q and the
// rotated k, v cache slots.
#include "device.h"

namespace prism {

template <typename T, int RT, int NT, bool PAIR>
__device__ __forceinline__ void mainloop(const u32x4 *__restrict__ w0, int nkb, const Act &x,
                                         int R, int kb0, int kb1, f32x4 (&acc)[NT][RT]) {
  constexpr int E = Ty<T>::E, KB = Ty<T>::KB;
  // k-blocks in flight: about 96 VGPRs of A and B fragments per lane
  constexpr int U0 = 24 / (NT + (PAIR ? 2 : 1) * RT);
  constexpr int U = U0 > 8 ? 8 : (U0 < 1 ? 1 : U0);
  const int lane = threadIdx.x & 63;
  const int col = lane & 15, kq = lane >> 4;
  const T *xh[RT];
  const T *xl[RT];
  bool ok[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = col + 16 * rt;
    ok[rt] = r < R;
    const size_t off = (size_t)(ok[rt] ? r : 0) * x.ld + kq * E;
    xh[rt] = (const T *)x.hi + off;
    xl[rt] = PAIR ? (const T *)x.lo + off : nullptr;
  }
  const u32x4 *wp[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) wp[n] = w0 + ((size_t)n * nkb + kb0) * 64 + lane;
  const u32x4 z4 = {0, 0, 0, 0};
  // batches of U k-blocks; the last batch is partial (n < U) but its loads
  // are still issued together, so no k-block waits for another
  for (int kb = kb0; kb < kb1; kb += U) {
    const int nb = kb1 - kb;
    u32x4 a[U][NT];
    u32x4 bh[U][RT], bl[U][RT];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int n = 0; n < NT; ++n) a[u][n] = u < nb ? __builtin_nontemporal_load(wp[n] + u * 64) : z4;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const size_t o = (size_t)(kb + u) * KB;
        const bool ld = ok[rt] && u < nb;
        bh[u][rt] = ld ? *(const u32x4 *)(xh[rt] + o) : z4;
        if (PAIR) bl[u][rt] = ld ? *(const u32x4 *)(xl[rt] + o) : z4;
      }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u < nb) {
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            acc[n][rt] = Ty<T>::mma(a[u][n], bh[u][rt], acc[n][rt]);
            if (PAIR) acc[n][rt] = Ty<T>::mma(a[u][n], bl[u][rt], acc[n][rt]);
          }
      }
    }
#pragma unroll
    for (int n = 0; n < NT; ++n) wp[n] += U * 64;
  }
}

// The same with two register sets: the k-blocks of batch j + 1 are in flight
// while batch j is consumed.  Loads past kb1 are clamped to the last k-block
// (re-read, discarded), so every batch issues the same loads.
template <typename T, int RT, int NT, bool PAIR>
__device__ __forceinline__ void mainloop_db(const u32x4 *__restrict__ w0, int nkb, const Act &x,
                                            int R, int kb0, int kb1, f32x4 (&acc)[NT][RT]) {
  constexpr int E = Ty<T>::E, KB = Ty<T>::KB;
  constexpr int U0 = 24 / (NT + (PAIR ? 2 : 1) * RT);
  constexpr int U = U0 > 8 ? 8 : (U0 < 1 ? 1 : U0);
  const int lane = threadIdx.x & 63;
  const int col = lane & 15, kq = lane >> 4;
  const T *xh[RT];
  const T *xl[RT];
  bool ok[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = col + 16 * rt;
    ok[rt] = r < R;
    const size_t off = (size_t)(ok[rt] ? r : 0) * x.ld + kq * E;
    xh[rt] = (const T *)x.hi + off;
    xl[rt] = PAIR ? (const T *)x.lo + off : nullptr;
  }
  const u32x4 *wp[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) wp[n] = w0 + (size_t)n * nkb * 64 + lane;
  const u32x4 z4 = {0, 0, 0, 0};
  u32x4 a[2][U][NT], bh[2][U][RT], bl[2][U][RT];
  auto load = [&](int s, int kb) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = min(kb + u, kb1 - 1);
#pragma unroll
      for (int n = 0; n < NT; ++n) a[s][u][n] = __builtin_nontemporal_load(wp[n] + (size_t)k * 64);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const size_t o = (size_t)k * KB;
        bh[s][u][rt] = ok[rt] ? *(const u32x4 *)(xh[rt] + o) : z4;
        if (PAIR) bl[s][u][rt] = ok[rt] ? *(const u32x4 *)(xl[rt] + o) : z4;
      }
    }
  };
  auto mma = [&](int s, int nb) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u < nb) {
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            acc[n][rt] = Ty<T>::mma(a[s][u][n], bh[s][u][rt], acc[n][rt]);
            if (PAIR) acc[n][rt] = Ty<T>::mma(a[s][u][n], bl[s][u][rt], acc[n][rt]);
          }
      }
    }
  };
  if (kb1 <= kb0) return;
  load(0, kb0);
  for (int kb = kb0; kb < kb1; kb += 2 * U) {
    load(1, kb + U);
    mma(0, kb1 - kb);
    if (kb + U >= kb1) break;
    load(0, kb + 2 * U);
    mma(1, kb1 - kb - U);
  }
}

// GEMV main loop for a few rows (R <= RR <= 4) of a bf16 matrix: each wave
// stages the activation columns of its own K range in LDS as fp32 (hi + lo),
// then each lane multiplies its 8 weights of a k-block by the matching fp32
// activations (an LDS broadcast: the 16 lanes of a k-quarter read the same
// address).  Only weight fragments occupy registers, so 16 k-blocks
// (16 KiB) stay in flight per wave, and the products are fp32-exact.  The
// first batch of weight loads is issued before the staging so the two
// overlap; as the staged columns are private to the wave, no workgroup
// barrier separates a wave's staging from its products.  Leaves the result
// in the MFMA accumulator layout so that all epilogues are shared.
constexpr int UV = 16;

__device__ __forceinline__ float lo_bf(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// 8 columns of a staged row from a packed bf16 plane (8 values) or from the
// hi + lo pair of planes
__device__ __forceinline__ void unpack8(const u32x4 q, float (&v)[8]) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    v[2 * m] = lo_bf(w[m]);
    v[2 * m + 1] = hi_bf(w[m]);
  }
}

// One wave stages the columns [c0, c1) (multiples of 32) of the operand rows
// as fp32 into xs (row stride K); rows R .. RR-1 read as zero.  Plain
// operands come as hi/lo planes; gathered fusion-FC rows are x_r =
// [E(tok_r) ; feature row] (K = H + F columns), and tok_r < 0 reads a zero
// embedding.
template <int RR, bool GX>
__device__ __forceinline__ void stage_wave(const Act &x, const Gather &gx, const int (&tok)[RR],
                                           int R, int K, float *xs, int c0, int c1) {
  const int lane = threadIdx.x & 63;
  for (int k = c0 + lane * 8; k < c1; k += 512) {
#pragma unroll
    for (int r = 0; r < RR; ++r) {
      float v[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) v[m] = 0.f;
      if (r < R) {
        if constexpr (!GX) {
          float h[8], l[8];
          unpack8(*(const u32x4 *)((const bf16_t *)x.hi + (size_t)r * x.ld + k), h);
          unpack8(*(const u32x4 *)((const bf16_t *)x.lo + (size_t)r * x.ld + k), l);
#pragma unroll
          for (int m = 0; m < 8; ++m) v[m] = h[m] + l[m];
        } else if (k < gx.H) {
          if (tok[r] >= 0)
            unpack8(*(const u32x4 *)((const bf16_t *)gx.embed + (size_t)tok[r] * gx.H + k), v);
        } else {
          const int fr = gx.in.feat_rows ? gx.in.feat_rows[r] : r;
          const size_t o = (size_t)fr * gx.in.feat_ld + (k - gx.H);
          if (gx.in.feat_bf16) {
            unpack8(*(const u32x4 *)((const bf16_t *)gx.in.feat + o), v);
          } else {
            const f32x4 f0 = *(const f32x4 *)((const float *)gx.in.feat + o);
            const f32x4 f1 = *(const f32x4 *)((const float *)gx.in.feat + o + 4);
            v[0] = f0.x; v[1] = f0.y; v[2] = f0.z; v[3] = f0.w;
            v[4] = f1.x; v[5] = f1.y; v[6] = f1.z; v[7] = f1.w;
          }
        }
      }
      *(f32x4 *)(xs + r * K + k) = f32x4{v[0], v[1], v[2], v[3]};
      *(f32x4 *)(xs + r * K + k + 4) = f32x4{v[4], v[5], v[6], v[7]};
    }
  }
}

// x rows staged in LDS as fp32 by the whole workgroup (every wave multiplies
// all K columns): R rows of the hi/lo operand (rows R .. RR-1 zero), 8
// columns per thread step
template <int RR>
__device__ __forceinline__ void stage_x(const Act &x, int R, int K, float *xs) {
  for (int i = threadIdx.x * 8; i < RR * K; i += blockDim.x * 8) {
    const int r = i / K, k = i % K;
    float v[8];
    if (r < R) {
      float h[8], l[8];
      unpack8(*(const u32x4 *)((const bf16_t *)x.hi + (size_t)r * x.ld + k), h);
      unpack8(*(const u32x4 *)((const bf16_t *)x.lo + (size_t)r * x.ld + k), l);
#pragma unroll
      for (int m = 0; m < 8; ++m) v[m] = h[m] + l[m];
    } else {
#pragma unroll
      for (int m = 0; m < 8; ++m) v[m] = 0.f;
    }
    *(f32x4 *)(xs + i) = f32x4{v[0], v[1], v[2], v[3]};
    *(f32x4 *)(xs + i + 4) = f32x4{v[4], v[5], v[6], v[7]};
  }
}

// one batch of a GEMV wave: up to UV loaded k-blocks (nb of them live)
// starting at k-block kb, times the staged rows
template <int RR>
__device__ __forceinline__ void valu_batch(const u32x4 (&a)[UV], int nb, int kb, int kq,
                                           const float *xs, int K, float (&acc)[RR]) {
#pragma unroll
  for (int u = 0; u < UV; ++u) {
    if (u < nb) {
      const int k0 = (kb + u) * 32 + kq * 8;
      const uint32_t w[4] = {a[u].x, a[u].y, a[u].z, a[u].w};
#pragma unroll
      for (int r = 0; r < RR; ++r) {
        const f32x4 x0 = *(const f32x4 *)(xs + r * K + k0);
        const f32x4 x1 = *(const f32x4 *)(xs + r * K + k0 + 4);
        float t = acc[r];
        t += lo_bf(w[0]) * x0.x; t += hi_bf(w[0]) * x0.y;
        t += lo_bf(w[1]) * x0.z; t += hi_bf(w[1]) * x0.w;
        t += lo_bf(w[2]) * x1.x; t += hi_bf(w[2]) * x1.y;
        t += lo_bf(w[3]) * x1.z; t += hi_bf(w[3]) * x1.w;
        acc[r] = t;
      }
    }
  }
}

// the same over a full batch of N k-blocks
template <int RR, int N>
__device__ __forceinline__ void valu_batch_n(const u32x4 (&a)[N], int kb, int kq,
                                             const float *xs, int K, float (&acc)[RR]) {
#pragma unroll
  for (int u = 0; u < N; ++u) {
    const int k0 = (kb + u) * 32 + kq * 8;
    const uint32_t w[4] = {a[u].x, a[u].y, a[u].z, a[u].w};
#pragma unroll
    for (int r = 0; r < RR; ++r) {
      const f32x4 x0 = *(const f32x4 *)(xs + r * K + k0);
      const f32x4 x1 = *(const f32x4 *)(xs + r * K + k0 + 4);
      float t = acc[r];
      t += lo_bf(w[0]) * x0.x; t += hi_bf(w[0]) * x0.y;
      t += lo_bf(w[1]) * x0.z; t += hi_bf(w[1]) * x0.w;
      t += lo_bf(w[2]) * x1.x; t += hi_bf(w[2]) * x1.y;
      t += lo_bf(w[3]) * x1.z; t += hi_bf(w[3]) * x1.w;
      acc[r] = t;
    }
  }
}

// A GEMV wave's per-lane sums -> the MFMA accumulator layout of its tile
template <int RR>
__device__ __forceinline__ f32x4 valu_result(float (&acc)[RR]) {
  const int lane = threadIdx.x & 63;
  // sum the 4 k-quarters of each tile row (lanes l, l^16, l^32, l^48)
#pragma unroll
  for (int r = 0; r < RR; ++r) {
    acc[r] += xor16_f(acc[r]);
    acc[r] += xor32_f(acc[r]);
  }
  // lane l now holds tile row (l & 15); the MFMA layout wants, in lane L,
  // tile rows 4 (L >> 4) + i of batch row (L & 15)
  const int col = lane & 15, rq = lane >> 4;
  float v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float t = 0.f;
#pragma unroll
    for (int r = 0; r < RR; ++r) {
      const float sv = __shfl(acc[r], 4 * rq + i, 64);
      if (col == r) t = sv;
    }
    v[i] = t;
  }
  return f32x4{v[0], v[1], v[2], v[3]};
}

template <int RR, bool GX>
__device__ __forceinline__ void mainloop_valu(const u32x4 *__restrict__ w0, const Act &x, int R,
                                              int K, float *xs, int kb0, int kb1, f32x4 &out,
                                              const Gather &gx, uint32_t *err,
                                              const float *tab = nullptr, int N = 0, int t0 = 0,
                                              f32x4 *tv = nullptr) {
  const int lane = threadIdx.x & 63, kq = lane >> 4;
  const u32x4 z4 = {0, 0, 0, 0};
  const u32x4 *wp = w0 + (size_t)kb0 * 64 + lane;
  // gathered FC rows: a wave whose K range covers embedding columns resolves
  // the rows' tokens itself; the previous LM head's partials are requested
  // ahead of the weights, so that the argmax does not wait for them.  With
  // the embedding table (tab), wave 0 resolves them for the epilogue and
  // requests its tile's table values right after its first weight batch.
  const bool tab_wave = GX && tab != nullptr && (threadIdx.x >> 6) == 0;
  const bool need_tok = GX && ((kb1 > kb0 && kb0 * 32 < gx.H) || tab_wave);
  const bool from_lm = need_tok && gx.lm.pval;
  constexpr int PRE = RR == 1 ? 8 : 2;   // entries per lane issued early (registers)
  TokLoads<PRE> tl[RR];
  if (from_lm) {
#pragma unroll
    for (int r = 0; r < RR; ++r)
      if (r < R) tl[r] = issue_tok<PRE>(gx.lm, r);
  }
  u32x4 a[UV];
  {
    const int nb = kb1 - kb0;
#pragma unroll
    for (int u = 0; u < UV; ++u) a[u] = u < nb ? __builtin_nontemporal_load(wp + u * 64) : z4;
  }
  int tok[RR];
#pragma unroll
  for (int r = 0; r < RR; ++r) tok[r] = -1;
  if (need_tok) {
    const bool lead = blockIdx.x == 0 && threadIdx.x == 0;   // wave 0 covers column 0
#pragma unroll
    for (int r = 0; r < RR; ++r) {
      if (r >= R) continue;
      int t = from_lm ? finish_tok(gx.lm, r, tl[r]) : gx.in.tokens[r];
      if (lead && from_lm && gx.lm.rec) gx.lm.rec[(size_t)r * gx.lm.ld_rec] = t;
      if (t < 0 || t >= gx.V) {
        // from the LM head, only a row of NaN logits leaves no token
        if (lead) atomicOr(err, from_lm && t == NO_TOKEN ? ERRF_NONFINITE : ERRF_TOKEN);
        t = -1;
      }
      tok[r] = t;
    }
  }
  if (tab_wave) {
    // lane (row, q4) of the epilogue layout: features 16 t0 + 4 q4 .. + 3
    const int r = lane & 15;
    int t = -1;
#pragma unroll
    for (int q = 0; q < RR; ++q) t = r == q ? tok[q] : t;
    *tv = r < R && t >= 0 ? *(const f32x4 *)(tab + (size_t)t * N + 16 * t0 + 4 * kq)
                          : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  stage_wave<RR, GX>(x, gx, tok, R, K, xs, kb0 * 32, kb1 * 32);
  wave_lds_sync();
  float acc[RR];
#pragma unroll
  for (int r = 0; r < RR; ++r) acc[r] = 0.f;
  for (int kb = kb0; kb < kb1; kb += UV) {
    const int nb = kb1 - kb;
    if (kb > kb0) {
#pragma unroll
      for (int u = 0; u < UV; ++u) a[u] = u < nb ? __builtin_nontemporal_load(wp + u * 64) : z4;
    }
    valu_batch<RR>(a, nb, kb, kq, xs, K, acc);
    wp += UV * 64;
  }
  out = valu_result<RR>(acc);
}

// The same over NT consecutive tiles per wave, each over the full K (nkb a
// multiple of UV, which the host checks, so the wave's weights are one
// contiguous stream of NT * nkb k-blocks).  Longer streams per wave and a
// grid that fits the chip in one round read HBM faster than one tile per
// wave.  Two register sets of UV / 2 k-blocks: batch j + 1 is in flight
// while batch j is consumed, so the stream has no gap between batches (8B
// LM head 163.0 -> 161.3 us, Llama-2 shape 50.1 -> 48.5 us against one set
// of UV k-blocks loaded and then consumed).  With several tiles per wave the
// stream's last pair is peeled, so every other load is unconditional: with a
// conditional one the compiler's wait counts drained every load at each pair
// (8B LM head 161.2 -> 160.8 us).
template <int RR, int NT>
__device__ __forceinline__ void mainloop_valu_tiles(const u32x4 *__restrict__ w0, int nkb,
                                                    const Act &x, int R, int K, float *xs,
                                                    bool live, f32x4 (&out)[NT]) {
  const int lane = threadIdx.x & 63, kq = lane >> 4;
  const u32x4 z4 = {0, 0, 0, 0};
  const u32x4 *wp = w0 + lane;
  constexpr int UP = UV / 2;
  const int bpt = nkb / UP;   // batches per tile (even)
  const int total = live ? NT * bpt : 0;
  u32x4 a[UP], b[UP];
#pragma unroll
  for (int u = 0; u < UP; ++u) a[u] = live ? __builtin_nontemporal_load(wp + u * 64) : z4;
  stage_x<RR>(x, R, K, xs);
  __syncthreads();
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    float acc[RR];
#pragma unroll
    for (int r = 0; r < RR; ++r) acc[r] = 0.f;
    // every pair but the stream's last loads the next one unconditionally,
    // so that the compiler counts the loads in flight exactly (several
    // tiles; a one-tile stream keeps the conditional load, which measured
    // faster there: Llama-2 shape 48.2 against 50.4 us)
    const int iend = NT > 1 && n == NT - 1 ? bpt - 2 : bpt;
    int i = 0;
    for (; i < iend && live; i += 2) {
      const int j = n * bpt + i;
#pragma unroll
      for (int u = 0; u < UP; ++u) b[u] = __builtin_nontemporal_load(wp + (size_t)(j + 1) * UP * 64 + u * 64);
      valu_batch_n<RR, UP>(a, i * UP, kq, xs, K, acc);
      if (NT > 1 || j + 2 < total) {
#pragma unroll
        for (int u = 0; u < UP; ++u) a[u] = __builtin_nontemporal_load(wp + (size_t)(j + 2) * UP * 64 + u * 64);
      }
      valu_batch_n<RR, UP>(b, (i + 1) * UP, kq, xs, K, acc);
    }
    if (NT > 1 && n == NT - 1 && live) {
      const int j = n * bpt + i;
#pragma unroll
      for (int u = 0; u < UP; ++u) b[u] = __builtin_nontemporal_load(wp + (size_t)(j + 1) * UP * 64 + u * 64);
      valu_batch_n<RR, UP>(a, i * UP, kq, xs, K, acc);
      valu_batch_n<RR, UP>(b, (i + 1) * UP, kq, xs, K, acc);
    }
    out[n] = valu_result<RR>(acc);
  }
}

// store an fp32 value as the storage-type operand (hi/lo pair for bf16)
template <typename T>
__device__ __forceinline__ void put_act(const ActOut &o, size_t i, float v) {
  if constexpr (sizeof(T) == 2) {
    const uint32_t h = f2bf(v);
    ((bf16_t *)o.hi)[i] = (bf16_t)h;
    ((bf16_t *)o.lo)[i] = (bf16_t)f2bf(v - bf2f(h));
  } else {
    ((float *)o.hi)[i] = v;
  }
}

// Row scales 1/sqrt(mean(x^2) + eps) of rows r0 .. r0 + nr - 1 from the
// producer's partial sums of squares (layout [part][R]).  Thread t serves row
// r0 + t / tpr and adds parts t % tpr, t % tpr + tpr, ... in that order; the
// tpr threads of a row (adjacent lanes of one wave) then meet in a fixed
// butterfly, so the result does not depend on scheduling.  The first
// SS_PER_THREAD parts of each thread are requested before the main loop
// (issue_scales); finish_scales adds them and loads any further ones (up to
// SS_MAX_ROUNDS times as many) after it.
constexpr int SS_PER_THREAD = 16;
constexpr int SS_MAX_ROUNDS = 4;
struct ScaleLoads {
  float v[SS_PER_THREAD];
};
__host__ __device__ inline int scale_tpr(int threads, int nr) {
  int t = 64;
  while (t > 1 && t * nr > threads) t >>= 1;
  return t;
}
__host__ __device__ inline bool scales_fit(int threads, int nr, int n_parts) {
  return nr <= threads && n_parts <= SS_MAX_ROUNDS * SS_PER_THREAD * scale_tpr(threads, nr);
}
__device__ __forceinline__ ScaleLoads issue_scales(const RowNorm &nm, int R, int r0, int nr) {
  ScaleLoads s;
  const int tpr = scale_tpr(blockDim.x, nr);
  const int r = threadIdx.x / tpr, sub = threadIdx.x % tpr;
#pragma unroll
  for (int j = 0; j < SS_PER_THREAD; ++j) {
    const int p = sub + j * tpr;
    s.v[j] = r < nr && p < nm.n_parts ? nm.ss[(size_t)p * R + r0 + r] : 0.f;
  }
  return s;
}
// every thread of the block calls it (barrier); rowscale[0 .. nr - 1]
__device__ __forceinline__ void finish_scales(const RowNorm &nm, int R, int r0, int nr,
                                              const ScaleLoads &s, float *rowscale) {
  const int tpr = scale_tpr(blockDim.x, nr);
  float acc = 0.f;
#pragma unroll
  for (int j = 0; j < SS_PER_THREAD; ++j) acc += s.v[j];
  {
    const int r = threadIdx.x / tpr;
    for (int p = threadIdx.x % tpr + SS_PER_THREAD * tpr; r < nr && p < nm.n_parts; p += tpr)
      acc += nm.ss[(size_t)p * R + r0 + r];
  }
  for (int o = 1; o < tpr; o <<= 1) acc += __shfl_xor(acc, o, 64);
  const int r = threadIdx.x / tpr;
  if (r < nr && threadIdx.x % tpr == 0) rowscale[r] = 1.0f / sqrtf(acc / (float)nm.n + nm.eps);
  __syncthreads();
}

// Operands of one lane's epilogue that do not depend on the product: the
// residual and gain values (EPI_NORM) or the RoPE inverse frequencies
// (EPI_QKV) of its 4 outputs.  The finish pass loads them before the slice
// sums, so that they do not add a round trip after them.
struct EpiPre {
  f32x4 res;
  float gain[4];
  float freq[4];
};

template <typename T, int EPI>
__device__ __forceinline__ EpiPre epilogue_prefetch(const GemmLaunch &g, int tile, int r) {
  const int n0 = tile * 16 + 4 * ((threadIdx.x & 63) >> 4);
  EpiPre p;
  p.res = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < 4; ++i) p.gain[i] = p.freq[i] = 0.f;
  if (r >= g.R) return p;
  if (EPI == EPI_NORM) {
    if (g.res) p.res = *(const f32x4 *)(g.res + (size_t)r * g.ldres + n0);
#pragma unroll
    for (int i = 0; i < 4; ++i) p.gain[i] = Ty<T>::ld((const T *)g.gain, n0 + i);
  } else if (EPI == EPI_QKV) {
    const int f0 = tile * 16, d = g.d;
    const int qd = g.nq * d, kd = g.nkv * d;
    if (f0 < qd + kd) {
      const int fr = f0 < qd ? f0 : f0 - qd;
      const int dim0 = 8 * ((fr % d) / 16) + 4 * ((threadIdx.x & 63) >> 4 & 1);
#pragma unroll
      for (int i = 0; i < 4; ++i) p.freq[i] = g.inv_freq[dim0 + i];
    }
  }
  return p;
}

// Epilogue of one 16x16 accumulator tile in the MFMA layout: the lane holds
// output rows n0..n0+3 (tiled order) of batch row r = (lane & 15) + 16 rt.
// Every lane of the wave must call it (it shuffles).  scale: the row's
// RMSNorm scale (1 if none); cbase / rpos: the row's cache slot and position
// (QKV only); pre: the lane's prefetched operands (else loaded here).
// EPI_NORM returns the tile's sum of squares of row r (valid in lanes
// 0..15); the caller stores it.
template <typename T, int EPI>
__device__ __forceinline__ float epilogue_tile(const GemmLaunch &g, int tile, int r, f32x4 a,
                                               float scale, long cbase, int rpos,
                                               f32x4 tadd = f32x4{0.f, 0.f, 0.f, 0.f},
                                               const EpiPre *pre = nullptr) {
  const int lane = threadIdx.x & 63, q4 = lane >> 4;
  const int n0 = tile * 16 + 4 * q4;
  const bool live = r < g.R;
  float v[4] = {a.x * scale, a.y * scale, a.z * scale, a.w * scale};
  if (EPI == EPI_NORM) {
    float ss = 0.f;
    if (live) {
      if (pre) {
        v[0] += pre->res.x; v[1] += pre->res.y; v[2] += pre->res.z; v[3] += pre->res.w;
      } else if (g.res) {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] += g.res[(size_t)r * g.ldres + n0 + i];
      }
      // embedding-table term of the fusion FC (zero otherwise)
      v[0] += tadd.x; v[1] += tadd.y; v[2] += tadd.z; v[3] += tadd.w;
      *(f32x4 *)(g.y + (size_t)r * g.ldy + n0) = f32x4{v[0], v[1], v[2], v[3]};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float gn = pre ? pre->gain[i] : Ty<T>::ld((const T *)g.gain, n0 + i);
        put_act<T>(g.g, (size_t)r * g.g.ld + n0 + i, v[i] * gn);
        if (g.yx.hi) put_act<T>(g.yx, (size_t)r * g.yx.ld + n0 + i, v[i]);
        ss += v[i] * v[i];
      }
    }
    // tile sum over the 4 lanes holding row r: fixed butterfly order
    ss += xor16_f(ss);
    ss += xor32_f(ss);
    return ss;
  } else if (EPI == EPI_SWIGLU) {
    if (live) {
      // rows interleave (gate c, up c, gate c + 1, up c + 1)
      const int c = n0 >> 1;
      put_act<T>(g.z, (size_t)r * g.z.ld + c, silu(v[0]) * v[1]);
      put_act<T>(g.z, (size_t)r * g.z.ld + c + 1, silu(v[2]) * v[3]);
    }
  } else {  // EPI_QKV
    const int d = g.d, half = d >> 1;
    const int qd = g.nq * d, kd = g.nkv * d;
    const int f0 = tile * 16;            // first feature of the tile (tiled order)
    // partner values for the rotation (lanes l and l ^ 32 hold the two halves)
    float pv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) pv[i] = xor32_f(v[i]);
    if (!live) return 0.f;
    if (f0 < qd + kd) {
      const bool isq = f0 < qd;
      const int fr = isq ? f0 : f0 - qd;
      const int head = fr / d;
      const int j = (fr % d) / 16;       // tile index within the head
      const bool first = q4 < 2;
      const int dim0 = 8 * j + 4 * (q4 & 1);   // dim within the first half
      float out[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // angle in fp64, reduced to [-pi, pi] in fp64, cos/sin in fp32
        const double ang = (double)rpos * (pre ? pre->freq[i] : g.inv_freq[dim0 + i]);
        const double red = ang - 6.283185307179586 * rint(ang * 0.15915494309189535);
        float sn, cs;
        sincosf((float)red, &sn, &cs);
        // first half: y1 = x1 c - x2 s ; second half: y2 = x2 c + x1 s
        out[i] = first ? v[i] * cs - pv[i] * sn : v[i] * cs + pv[i] * sn;
      }
      const int dimb = first ? dim0 : half + dim0;
      if (isq) {
        *(f32x4 *)(g.q + (size_t)r * qd + head * d + dimb) = f32x4{out[0], out[1], out[2], out[3]};
      } else {
        // pool layout [block, kv head, slot in block, d]
        const long base = cbase < 0 ? -1 : cbase + (long)head * g.kv.bs * d;
        if (base < 0) {
          atomicOr(g.err, ERRF_CAPACITY);
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) Ty<T>::st((T *)g.kv.k_pool, base + dimb + i, out[i]);
        }
      }
    } else {
      const int fr = f0 - qd - kd;
      const int head = fr / d;
      const int dim = fr % d + 4 * q4;
      const long base = cbase < 0 ? -1 : cbase + (long)head * g.kv.bs * d;
      if (base < 0) {
        atomicOr(g.err, ERRF_CAPACITY);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) Ty<T>::st((T *)g.kv.v_pool, base + dim + i, v[i]);
      }
    }
  }
  return 0.f;
}

// cache slot (block, head 0, offset) and position of row r, or -1
__device__ __forceinline__ long cache_base(const GemmLaunch &g, int r, int &pos) {
  pos = g.rows.pos[r];
  const int b = g.rows.seq[r], slot = g.rows.slot[r];
  const int bi = slot / g.kv.bs;
  if (b >= 0 && b < g.kv.n_seq && slot >= 0 && bi < g.kv.mbps) {
    const int blk = g.kv.block_table[(size_t)b * g.kv.mbps + bi];
    if (blk >= 0 && blk < g.kv.n_blocks)
      return (long)blk * g.nkv * g.kv.bs * g.d + (long)(slot % g.kv.bs) * g.d;
  }
  return -1;
}

// batched variants (more accumulators) run at most 8 waves per workgroup,
// which leaves them 256 VGPRs; the planner caps its wave counts the same way
template <int RT, int NT>
constexpr int gemm_max_threads() { return 64 * product_max_waves(RT, NT); }

// kernel-only epilogue tag: EPI_NORM on fusion-FC rows that the GEMV main
// loop gathers itself (no input norm), a separate instantiation so that the
// other EPI_NORM products carry none of the gather's registers
constexpr int EPI_NORM_GATHER = 3;

template <typename T, int RT, int NT, bool PAIR, int EPI_K, int VR>
__global__ __launch_bounds__((gemm_max_threads<RT, NT>())) void k_gemm(GemmLaunch g) {
  constexpr bool GX = EPI_K == EPI_NORM_GATHER;
  constexpr int EPI = GX ? EPI_NORM : EPI_K;
  // dynamic LDS: [(kw - 1) * NT * RT * 64] f32x4 partial sums, kw floats,
  // then (GEMV path, VR > 0) VR * K floats of staged activations
  extern __shared__ f32x4 red[];
  __shared__ float rowscale[MAX_ROWS];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int kw = g.kw;
  const int t0 = blockIdx.x * NT;
  const TiledMat &m = g.m;
  const bool has_norm = !GX && (g.norm.scale != nullptr || g.norm.n_parts > 0);
  const bool own_scales = !GX && g.norm.scale == nullptr && g.norm.n_parts > 0;
  ScaleLoads sl;
  if (own_scales) sl = issue_scales(g.norm, g.R, 0, g.R);

  // QKV: wave 0 looks up its rows' cache slots and positions before the
  // main loop, so these dependent loads overlap the weight stream
  long cbase[RT];
  int rpos[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    cbase[rt] = -1;
    rpos[rt] = 0;
  }
  if constexpr (EPI == EPI_QKV) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = (lane & 15) + 16 * rt;
      if (wave == 0 && r < g.R) cbase[rt] = cache_base(g, r, rpos[rt]);
    }
  }
  f32x4 acc[NT][RT];
  f32x4 tv = f32x4{0.f, 0.f, 0.f, 0.f};   // GEMV fusion FC: wave 0's embedding-table values
#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[n][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nk = m.nkb - g.kb_lo;
  const int kb0 = g.kb_lo + (int)((long)wave * nk / kw);
  const int kb1 = g.kb_lo + (int)((long)(wave + 1) * nk / kw);
  if constexpr (VR > 0) {
    float *xs = (float *)&red[(kw - 1) * NT * RT * 64] + 64 * kw;
    mainloop_valu<VR, GX>((const u32x4 *)m.w + (size_t)t0 * m.nkb * 64, g.x, g.R, m.K, xs, kb0,
                          kb1, acc[0][0], g.gx, g.err, g.tab, m.N, t0, &tv);
  } else {
    // up to 16 rows (7 or more tiles: registers) the next batch of k-blocks
    // is in flight while one is consumed: batch 16 -0.7%; at 32 rows the
    // second register set spills (tree +5%)
    if constexpr (RT == 1 && NT >= 7 && sizeof(T) == 2)
      mainloop_db<T, RT, NT, PAIR>((const u32x4 *)m.w + (size_t)t0 * m.nkb * 64, m.nkb, g.x, g.R,
                                   kb0, kb1, acc);
    else
      mainloop<T, RT, NT, PAIR>((const u32x4 *)m.w + (size_t)t0 * m.nkb * 64, m.nkb, g.x, g.R, kb0,
                                kb1, acc);
  }
  if (kw > 1) {
    if (wave > 0) {
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) red[(((wave - 1) * NT + n) * RT + rt) * 64 + lane] = acc[n][rt];
    }
  }
  if (own_scales) {
    __syncthreads();
    finish_scales(g.norm, g.R, 0, g.R, sl, rowscale);
  } else if (kw > 1) {
    __syncthreads();
  }
  if (wave != 0) return;
  for (int j = 1; j < kw; ++j)
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[n][rt] += red[(((j - 1) * NT + n) * RT + rt) * 64 + lane];

#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = (lane & 15) + 16 * rt;
      const float sc = has_norm && r < g.R ? (own_scales ? rowscale[r] : g.norm.scale[r]) : 1.f;
      f32x4 tadd = GX ? tv : f32x4{0.f, 0.f, 0.f, 0.f};
      if (EPI == EPI_NORM && !GX && g.tab && r < g.R) {   // batched rows: tokens from the prep
        const int t = g.tab_tok[r];
        if (t >= 0) tadd = *(const f32x4 *)(g.tab + (size_t)t * m.N + (t0 + n) * 16 + 4 * (lane >> 4));
      }
      const float ss = epilogue_tile<T, EPI>(g, t0 + n, r, acc[n][rt], sc, cbase[rt], rpos[rt], tadd);
      if (EPI == EPI_NORM && r < g.R && lane < 16) g.ss[(size_t)(t0 + n) * g.R + r] = ss;
    }
}

// Token of row i for a K-split fusion FC that has no prep pass: wave 0 of
// the workgroup with linear index i resolves it, its loads of the previous
// LM head's top-1 partials issued at the start of the kernel and reduced
// after them, so that the other loads of the workgroup do not wait.
constexpr int SPLIT_TOK_PRE = 4;
struct SplitTok {
  int row = -1;                  // wave-uniform; -1: this wave resolves none
  int tok = -1;
  TokLoads<SPLIT_TOK_PRE> l;
};
__device__ __forceinline__ SplitTok split_tok_issue(const GemmLaunch &g) {
  SplitTok st;
  const int i = blockIdx.y * gridDim.x + blockIdx.x;
  if (!g.tok_out || (threadIdx.x >> 6) != 0 || i >= g.R) return st;
  st.row = i;
  if (g.gx.lm.pval) st.l = issue_tok<SPLIT_TOK_PRE>(g.gx.lm, i);
  else st.tok = g.gx.in.tokens[i];
  return st;
}
__device__ __forceinline__ void split_tok_store(const GemmLaunch &g, const SplitTok &st) {
  if (st.row < 0) return;
  const bool from_lm = g.gx.lm.pval != nullptr;
  int t = from_lm ? finish_tok<SPLIT_TOK_PRE>(g.gx.lm, st.row, st.l) : st.tok;
  if ((threadIdx.x & 63) != 0) return;
  if (from_lm && g.gx.lm.rec) g.gx.lm.rec[(size_t)st.row * g.gx.lm.ld_rec] = t;
  if (t < 0 || t >= g.gx.V) {
    // from the LM head, only a row of NaN logits leaves no token
    atomicOr(g.err, from_lm && t == NO_TOKEN ? ERRF_NONFINITE : ERRF_TOKEN);
    t = -1;
  }
  g.tok_out[st.row] = t;
}

// Batched products (R > 4 rows): the 4 waves of a workgroup take 4
// consecutive groups of NT tiles over the same K slice (slice blockIdx.y of
// gridDim.y), so the B fragments a wave loads are the ones its neighbours
// load at about the same time (L1 hits), and each fragment feeds NT tiles.
// Slice partial sums go to part[s][r][n]; k_gemm_finish adds the slices in
// order and applies the epilogue.
template <typename T, int RT, int NT, bool PAIR>
__global__ __launch_bounds__(256) void k_gemm_split(GemmLaunch g) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const TiledMat &m = g.m;
  const int t0 = (blockIdx.x * 4 + wave) * NT;
  if (t0 >= m.n_tiles) return;   // n_tiles is a multiple of NT; no barriers below
  // (resolved before the main loop: kept across it, its registers lowered
  // the occupancy of some instantiations)
  split_tok_store(g, split_tok_issue(g));   // wave 0 is never idle
  const int S = gridDim.y, sl = blockIdx.y;
  const int nk = m.nkb - g.kb_lo;
  const int kb0 = g.kb_lo + (int)((long)sl * nk / S), kb1 = g.kb_lo + (int)((long)(sl + 1) * nk / S);
  f32x4 acc[NT][RT];
#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[n][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // up to 16 rows with two register sets of k-blocks (batch 16 -0.8%); at
  // 32 rows it was slower (70B +0.6%)
  if constexpr (RT == 1 && sizeof(T) == 2)
    mainloop_db<T, RT, NT, PAIR>((const u32x4 *)m.w + (size_t)t0 * m.nkb * 64, m.nkb, g.x, g.R, kb0,
                                 kb1, acc);
  else
    mainloop<T, RT, NT, PAIR>((const u32x4 *)m.w + (size_t)t0 * m.nkb * 64, m.nkb, g.x, g.R, kb0,
                              kb1, acc);
  const int q4 = lane >> 4;
#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = (lane & 15) + 16 * rt;
      if (r < g.R)
        *(f32x4 *)(g.part + ((size_t)sl * g.R + r) * m.N + (t0 + n) * 16 + 4 * q4) = acc[n][rt];
    }
}

// The same for bf16 with the slice's activation fragments staged in LDS once
// per workgroup: the 4 waves share the K slice, so instead of each wave
// loading every B fragment, the workgroup loads each once and the waves read
// them from LDS.  Layout xs[(k-block, plane, row tile)][lane], the B operand
// order, so each ds_read_b128 is one contiguous, conflict-free KiB.  The
// first batch of weight loads is issued right after the staging loads, so
// the two overlap; only weight fragments occupy registers in the loop (two
// sets, the next batch in flight while one is consumed).  The launcher takes
// this path when a wave stages at most SPLIT_LDS_FRAGS / 4 fragments.
constexpr int SPLIT_LDS_FRAGS = 64;   // staged fragments per workgroup (64 KiB)
template <int RT, int NT>
__global__ __launch_bounds__(256) void k_gemm_split_lds(GemmLaunch g) {
  extern __shared__ u32x4 xs_split[];    // [nf][64]
  constexpr int SF = SPLIT_LDS_FRAGS / 4;  // fragments per wave
  constexpr int U = 16 / NT > 0 ? 16 / NT : 1;   // k-blocks per batch
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const TiledMat &m = g.m;
  const int t0 = (blockIdx.x * 4 + wave) * NT;
  const bool live = t0 < m.n_tiles;       // n_tiles is a multiple of NT
  const int S = gridDim.y, sl = blockIdx.y;
  const int nk = m.nkb - g.kb_lo;
  const int kb0 = g.kb_lo + (int)((long)sl * nk / S), kb1 = g.kb_lo + (int)((long)(sl + 1) * nk / S);
  const int nf = (kb1 - kb0) * 2 * RT;    // <= SPLIT_LDS_FRAGS (checked by the launcher)
  const SplitTok stok = split_tok_issue(g);   // wave 0 is live in every workgroup
  // staging loads: fragment f = (k-block i, plane p, row tile rt), lane (row
  // 16 rt + (lane & 15), k 8 (lane >> 4)); unconditional (clamped) so that
  // the weight loads issued after them stay in flight
  u32x4 sv[SF];
#pragma unroll
  for (int i = 0; i < SF; ++i) {
    const int f = max(min(wave + 4 * i, nf - 1), 0);
    const int kbi = f / (2 * RT), pl = (f / RT) & 1, rt = f % RT;
    const int r = (lane & 15) + 16 * rt;
    const int kb = min(kb0 + kbi, m.nkb - 1);
    const bf16_t *src = (const bf16_t *)(pl ? g.x.lo : g.x.hi) + (size_t)(r < g.R ? r : 0) * g.x.ld +
                        (size_t)kb * 32 + 8 * (lane >> 4);
    sv[i] = *(const u32x4 *)src;
    if (r >= g.R) sv[i] = u32x4{0, 0, 0, 0};
  }
  const u32x4 *wp[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) wp[n] = (const u32x4 *)m.w + ((size_t)(live ? t0 : 0) + n) * m.nkb * 64 + lane;
  u32x4 a[2][U][NT];
  auto loadw = [&](int st, int kb) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = min(kb + u, kb1 - 1);
#pragma unroll
      for (int n = 0; n < NT; ++n) a[st][u][n] = __builtin_nontemporal_load(wp[n] + (size_t)k * 64);
    }
  };
  if (live && kb1 > kb0) loadw(0, kb0);
#pragma unroll
  for (int i = 0; i < SF; ++i) {
    const int f = wave + 4 * i;
    if (f < nf) xs_split[f * 64 + lane] = sv[i];
  }
  __syncthreads();
  split_tok_store(g, stok);               // its loads returned before the staging ones
  if (!live || kb1 <= kb0) return;        // no barriers below
  f32x4 acc[NT][RT];
#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[n][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](int st, int kb, int nb) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (u < nb) {
        const int kbi = kb + u - kb0;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const u32x4 bh = xs_split[((kbi * 2 + 0) * RT + rt) * 64 + lane];
          const u32x4 bl = xs_split[((kbi * 2 + 1) * RT + rt) * 64 + lane];
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            acc[n][rt] = Ty<bf16_t>::mma(a[st][u][n], bh, acc[n][rt]);
            acc[n][rt] = Ty<bf16_t>::mma(a[st][u][n], bl, acc[n][rt]);
          }
        }
      }
    }
  };
  for (int kb = kb0; kb < kb1; kb += 2 * U) {
    loadw(1, kb + U);
    mma(0, kb, kb1 - kb);
    if (kb + U >= kb1) break;
    loadw(0, kb + 2 * U);
    mma(1, kb + U, kb1 - kb - U);
  }
  const int q4 = lane >> 4;
#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = (lane & 15) + 16 * rt;
      if (r < g.R)
        *(f32x4 *)(g.part + ((size_t)sl * g.R + r) * m.N + (t0 + n) * 16 + 4 * q4) = acc[n][rt];
    }
}

// Tiles per workgroup of the finish pass (a divisor of n_tiles, at most 8):
// few, so that the pass spreads over many CUs, but for EPI_NORM enough that
// a row's sums-of-squares parts (n_tiles / ft) stay within FIN_PARTS, which
// the consumers reduce themselves.
constexpr int FIN_TILES = 2, FIN_TILES_NORM = 2, FIN_PARTS = 128;
static int finish_tiles(int n_tiles, int epi) {
  int f = epi == EPI_NORM ? FIN_TILES_NORM : FIN_TILES;
  if (epi == EPI_NORM)
    while (f < 8 && n_tiles / f > FIN_PARTS) f *= 2;
  while (f > 1 && n_tiles % f) f >>= 1;
  return f;
}

// One wave per (tile, 16-row group), FT = blockDim.x / 64 consecutive tiles
// per workgroup: the slices' partial sums in slice order, then the shared
// epilogue.  The row scales of a normed operand (QKV, SWIGLU) are reduced
// here from the producer's partials (or come precomputed).  EPI_NORM sums of
// squares are added over the workgroup's tiles in wave order, which leaves
// one partial per workgroup and row (n_tiles / FT per row in all).
constexpr int FIN_UNROLL = 16;
template <typename T, int EPI>
__global__ __launch_bounds__(512) void k_gemm_finish(GemmLaunch g) {
  __shared__ float rowscale[16];
  __shared__ float ssw[8][16];    // [wave][row of the group]
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int ft = blockDim.x >> 6;
  const int tile = blockIdx.x * ft + wave;
  const int r0 = 16 * blockIdx.y, nr = min(16, g.R - r0);
  const int r = (lane & 15) + r0;
  const bool own = g.norm.scale == nullptr && g.norm.n_parts > 0;
  ScaleLoads sl;
  if (own) sl = issue_scales(g.norm, g.R, r0, nr);
  const int n0 = tile * 16 + 4 * (lane >> 4);
  f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 tadd = f32x4{0.f, 0.f, 0.f, 0.f};   // fusion FC: the row's embedding-table term
  long cbase = -1;
  int rpos = 0;
  // operands that do not depend on the slices go out before them
  const EpiPre pre = epilogue_prefetch<T, EPI>(g, tile, r);
  if (r < g.R) {
    if (EPI == EPI_QKV) cbase = cache_base(g, r, rpos);
    // the row's token goes out first, its table row right after the first
    // batch of slice loads, so the two dependent loads overlap the slices
    const bool tab = EPI == EPI_NORM && g.tab;
    const int ttok = tab ? g.tab_tok[r] : -1;
    // slices in order, their loads issued FIN_UNROLL at a time
    const f32x4 *pp = (const f32x4 *)(g.part + (size_t)r * g.m.N + n0);
    const size_t stride = (size_t)g.R * g.m.N / 4;
    for (int s0 = 0; s0 < g.split; s0 += FIN_UNROLL) {
      f32x4 v[FIN_UNROLL];
#pragma unroll
      for (int j = 0; j < FIN_UNROLL; ++j)
        v[j] = s0 + j < g.split ? pp[(size_t)(s0 + j) * stride] : f32x4{0.f, 0.f, 0.f, 0.f};
      if (s0 == 0 && ttok >= 0) tadd = *(const f32x4 *)(g.tab + (size_t)ttok * g.m.N + n0);
#pragma unroll
      for (int j = 0; j < FIN_UNROLL; ++j)
        if (s0 + j < g.split) a += v[j];
    }
  }
  float sc = 1.f;
  if (own) {
    finish_scales(g.norm, g.R, r0, nr, sl, rowscale);
    if (r < g.R) sc = rowscale[r - r0];
  } else if (g.norm.scale && r < g.R) {
    sc = g.norm.scale[r];
  }
  const float ss = epilogue_tile<T, EPI>(g, tile, r, a, sc, cbase, rpos, tadd, &pre);
  if constexpr (EPI == EPI_NORM) {
    if (lane < 16) ssw[wave][lane] = ss;
    __syncthreads();
    if (threadIdx.x < nr) {
      float t = 0.f;
      for (int w = 0; w < ft; ++w) t += ssw[w][threadIdx.x];
      g.ss[(size_t)blockIdx.x * g.R + r0 + threadIdx.x] = t;
    }
  }
}

// LM head: each wave covers NT 16-row vocab tiles over the full K; a
// workgroup (4 waves) covers 64*NT vocab ids.  The epilogue applies the
// final-norm row scale and reduces the workgroup's logits of each row to
// partials: max, sum of exp(logit - max), and the top-k (logit desc, id asc);
// optional fp32 logits store.  With no_part set it only stores the logits
// (top-k > 1 on MFMA tiles: there the in-kernel top-k rounds, run by one wave
// per SIMD after the weight stream, cost more than storing the logits and
// reducing them in a separate, fully occupied pass).
template <typename T, int RT, int NT, bool PAIR, int VR>
__global__ __launch_bounds__(256) void k_lmhead(LmLaunch g) {
  extern __shared__ float xs_lm[];   // GEMV path: VR * K staged activations
  __shared__ float sl[RT * 16][64 * NT + 1];
  __shared__ float rowscale[MAX_ROWS];
  const TiledMat &m = g.m;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t0 = (blockIdx.x * 4 + wave) * NT;
  const bool has_norm = g.norm.scale != nullptr || g.norm.n_parts > 0;
  const bool own_scales = g.norm.scale == nullptr && g.norm.n_parts > 0;
  ScaleLoads sc;
  if (own_scales) sc = issue_scales(g.norm, g.R, 0, g.R);
  f32x4 acc[NT][RT];
#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) acc[n][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bool live = t0 < m.n_tiles;    // n_tiles is a multiple of NT
  if constexpr (VR > 0) {
    // every wave takes part (staging barrier); idle waves stream nothing
    f32x4 res[NT];
    mainloop_valu_tiles<VR, NT>((const u32x4 *)m.w + (size_t)(live ? t0 : 0) * m.nkb * 64, m.nkb,
                                g.x, g.R, m.K, xs_lm, live, res);
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[n][0] = res[n];
  } else if (live) {
    // up to 16 rows the double-buffered loop (16-row LM head 166.3 -> 164.8 us);
    // at 32 rows it was slower (327 -> 348 us), so those keep one batch at a time
    if constexpr (RT == 1)
      mainloop_db<T, RT, NT, PAIR>((const u32x4 *)m.w + (size_t)t0 * m.nkb * 64, m.nkb, g.x, g.R,
                                   0, m.nkb, acc);
    else
      mainloop<T, RT, NT, PAIR>((const u32x4 *)m.w + (size_t)t0 * m.nkb * 64, m.nkb, g.x, g.R, 0,
                                m.nkb, acc);
  }
  if (own_scales) {
    __syncthreads();
    finish_scales(g.norm, g.R, 0, g.R, sc, rowscale);
  }
  const int q4 = lane >> 4;
#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = (lane & 15) + 16 * rt;
      if (r >= g.R) continue;
      const float s = has_norm ? (own_scales ? rowscale[r] : g.norm.scale[r]) : 1.f;
      const float v[4] = {acc[n][rt].x * s, acc[n][rt].y * s, acc[n][rt].z * s, acc[n][rt].w * s};
      if (!g.no_part) {
#pragma unroll
        for (int i = 0; i < 4; ++i) sl[r][(wave * NT + n) * 16 + 4 * q4 + i] = v[i];
      }
      if (live && g.logits)
        *(f32x4 *)(g.logits + (size_t)r * g.ld_logits + (t0 + n) * 16 + 4 * q4) =
            f32x4{v[0], v[1], v[2], v[3]};
    }
  if (g.no_part) return;   // uniform: the partials come from k_lm_topk
  __syncthreads();
  // Each wave reduces rows wave, wave + 4, ...: up to RB of them together,
  // so that the dependent shuffle chains of their reductions overlap.
  constexpr int RB = VR > 0 ? 1 : 4;
  const int base_id = blockIdx.x * 64 * NT;
  for (int r0 = wave; r0 < g.R; r0 += 4 * RB) {
    float v[RB][NT];
    int id[RB][NT];
    float mx[RB];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const int r = r0 + 4 * b;
      mx[b] = -INFINITY;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int c = n * 64 + lane;
        id[b][n] = base_id + c;
        const bool valid = r < g.R && id[b][n] < g.V;
        v[b][n] = valid ? sl[r < g.R ? r : 0][c] : -INFINITY;
        if (!valid) id[b][n] = 0x7fffffff;
        mx[b] = fmaxf(mx[b], v[b][n]);
      }
    }
    wave_max_n<RB>(mx);
    // max and sum of exp over the scaled logits z = v * inv_temp (inv_temp > 0)
    float e[RB];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      e[b] = 0.f;
#pragma unroll
      for (int n = 0; n < NT; ++n)
        e[b] += id[b][n] != 0x7fffffff ? expf(v[b][n] * g.inv_temp - mx[b] * g.inv_temp) : 0.f;
    }
    wave_sum_n<RB>(e);
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const int r = r0 + 4 * b;
      if (lane == 0 && r < g.R) {
        const size_t pi = (size_t)r * g.n_wg + blockIdx.x;
        g.pmax[pi] = mx[b] * g.inv_temp;
        g.psum[pi] = e[b];
      }
    }
    // top-k on 64-bit candidate keys (one unsigned compare per pair)
    uint64_t key[RB][NT];
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
      for (int n = 0; n < NT; ++n) key[b][n] = cand_key(v[b][n], id[b][n]);
    if (g.topk > 1) {
      // each lane sorts its NT candidates once (odd-even transposition,
      // best first); the rounds then take the list heads
#pragma unroll
      for (int b = 0; b < RB; ++b)
#pragma unroll
        for (int pass = 0; pass < NT; ++pass)
#pragma unroll
          for (int n = pass & 1; n + 1 < NT; n += 2) {
            const uint64_t lo = key[b][n], hi = key[b][n + 1];
            key[b][n] = hi > lo ? hi : lo;
            key[b][n + 1] = hi > lo ? lo : hi;
          }
    }
    const uint64_t none = cand_key(-INFINITY, 0x7fffffff);
    for (int j = 0; j < g.topk; ++j) {
      uint64_t bk[RB];
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        bk[b] = key[b][0];
        if (g.topk == 1) {
#pragma unroll
          for (int n = 1; n < NT; ++n) bk[b] = key[b][n] > bk[b] ? key[b][n] : bk[b];
        }
      }
      wave_max_key_n<RB>(bk);
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        const int r = r0 + 4 * b;
        if (lane == 0 && r < g.R) {
          const size_t pi = (size_t)r * g.n_wg + blockIdx.x;
          g.pval[pi * g.topk + j] = key_value(bk[b]);
          g.pid[pi * g.topk + j] = key_id(bk[b]);
        }
        // the winning lane drops its head (ids are distinct)
        const bool win = key[b][0] == bk[b];
#pragma unroll
        for (int n = 0; n + 1 < NT; ++n) key[b][n] = win ? key[b][n + 1] : key[b][n];
        key[b][NT - 1] = win ? none : key[b][NT - 1];
      }
    }
  }
}

static_assert(GEMV_MAX_ROWS == 2, "GEMV variants cover 1 and 2 rows");

template <typename T, int RT, int NT, bool PAIR, int VR>
static bool gemm_epi(const GemmLaunch &g, hipStream_t s) {
  if (g.kw < 1 || 64 * g.kw > gemm_max_threads<RT, NT>()) return false;
  dim3 grid(g.m.n_tiles / NT);
  size_t lds = (size_t)((g.kw - 1) * NT * RT * 64) * sizeof(f32x4) +
               (size_t)64 * g.kw * sizeof(float);
  if (VR > 0) lds += (size_t)VR * g.m.K * sizeof(float);
  if constexpr (VR > 0) {
    if (g.epi == EPI_NORM && g.gx.embed) {
      hipLaunchKernelGGL((k_gemm<T, RT, NT, PAIR, EPI_NORM_GATHER, VR>), grid, dim3(64 * g.kw), lds, s, g);
      return true;
    }
  }
  if (g.epi == EPI_NORM) hipLaunchKernelGGL((k_gemm<T, RT, NT, PAIR, EPI_NORM, VR>), grid, dim3(64 * g.kw), lds, s, g);
  else if (g.epi == EPI_SWIGLU) hipLaunchKernelGGL((k_gemm<T, RT, NT, PAIR, EPI_SWIGLU, VR>), grid, dim3(64 * g.kw), lds, s, g);
  else if constexpr (NT <= 2) hipLaunchKernelGGL((k_gemm<T, RT, NT, PAIR, EPI_QKV, VR>), grid, dim3(64 * g.kw), lds, s, g);
  else return false;   // the planner keeps QKV off the 4- and 8-tile unsplit variants
  return true;
}

// Products over more rows than the 16-row-tile kernels take (tree-scoring
// passes of up to ROWGRP_MAX_ROWS rows, bf16).  A workgroup takes 4 RG_NT
// output tiles (RG_NT per wave) against one group of ROWGRP_ROWS rows over
// one K slice.  The row group's hi and lo B fragments of each
// k-block are staged in LDS once for the 4 waves (two buffers, one barrier
// per k-block), so each weight fragment feeds 4 row tiles x 2 planes from
// registers and LDS.  The row groups of one (tile group, slice) pair take
// workgroup ids 8 apart: the hardware's round-robin places them on one XCD
// and dispatches them together, and the later ones find the weights in that
// XCD's L2.  Slice partial sums go to part[s][r][n] as in k_gemm_split, and
// k_gemm_finish applies the epilogue.
constexpr int RG_RT = 4, RG_D = 2;
static_assert(16 * RG_RT == ROWGRP_ROWS, "row-group tiling");
template <int RG_NT>
__device__ __forceinline__ void gemm_rows_body(const GemmLaunch &g) {
  __shared__ u32x4 xs[2][2 * RG_RT][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const TiledMat &m = g.m;
  const int n_rg = (g.R + ROWGRP_ROWS - 1) / ROWGRP_ROWS;
  const int n_xg = (m.n_tiles + 4 * RG_NT - 1) / (4 * RG_NT);
  const int S = g.split;
  const int id = blockIdx.x, blk = id / (8 * n_rg), in = id % (8 * n_rg);
  const int pair = blk * 8 + in % 8, yg = in / 8;
  if (pair >= n_xg * S) return;               // padding workgroup (uniform)
  const int xg = pair % n_xg, sl = pair / n_xg;
  const int t0 = (xg * 4 + wave) * RG_NT;
  const bool live = t0 < m.n_tiles;           // the wave's first tile exists
  const int r0 = yg * ROWGRP_ROWS;
  const int nk = m.nkb - g.kb_lo;
  // S <= nk (host check): every slice has at least one k-block
  const int kb0 = g.kb_lo + (int)((long)sl * nk / S), kb1 = g.kb_lo + (int)((long)(sl + 1) * nk / S);
  const u32x4 z4 = {0, 0, 0, 0};
  // staging: wave w loads the hi and lo fragments of row tiles w, w + 4, ...
  // A row past the last one stages row 0 instead: B column j of the product
  // only reaches output row j, which is not stored
  constexpr int SJ = RG_RT / 4;
  const bf16_t *sh[SJ], *sw[SJ];
#pragma unroll
  for (int j = 0; j < SJ; ++j) {
    const int sr = r0 + 16 * (wave + 4 * j) + (lane & 15);
    sh[j] = (const bf16_t *)g.x.hi + (size_t)(sr < g.R ? sr : 0) * g.x.ld + 8 * (lane >> 4);
    sw[j] = (const bf16_t *)g.x.lo + (size_t)(sr < g.R ? sr : 0) * g.x.ld + 8 * (lane >> 4);
  }
  const u32x4 *wp[RG_NT];
#pragma unroll
  for (int n = 0; n < RG_NT; ++n) {   // a tile past the end streams the wave's first (discarded)
    const int t = t0 + n < m.n_tiles ? t0 + n : (live ? t0 : 0);
    wp[n] = (const u32x4 *)m.w + (size_t)t * m.nkb * 64 + lane;
  }
  u32x4 a[RG_D][RG_NT], sv[RG_D][SJ][2];
#pragma unroll
  for (int u = 0; u < RG_D; ++u) {
    const int k = min(kb0 + u, kb1 - 1);
#pragma unroll
    for (int j = 0; j < SJ; ++j) {
      sv[u][j][0] = *(const u32x4 *)(sh[j] + (size_t)k * 32);
      sv[u][j][1] = *(const u32x4 *)(sw[j] + (size_t)k * 32);
    }
#pragma unroll
    for (int n = 0; n < RG_NT; ++n) a[u][n] = wp[n][(size_t)k * 64];
  }
#pragma unroll
  for (int j = 0; j < SJ; ++j) {
    xs[0][2 * (wave + 4 * j)][lane] = sv[0][j][0];
    xs[0][2 * (wave + 4 * j) + 1][lane] = sv[0][j][1];
  }
  __syncthreads();
  f32x4 acc[RG_NT][RG_RT];
#pragma unroll
  for (int n = 0; n < RG_NT; ++n)
#pragma unroll
    for (int rt = 0; rt < RG_RT; ++rt) acc[n][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // the slice in whole pairs of k-blocks: an odd slice ends with a k-block
  // of zero activations (its weight loads re-read the last one), so that
  // the loop has no exit in its middle and the accumulators stay in place
  const int kb_end = kb0 + ((kb1 - kb0 + 1) & ~1);
  for (int kb = kb0; kb < kb_end; kb += RG_D) {
#pragma unroll
    for (int u = 0; u < RG_D; ++u) {
      const int k = kb + u;                   // staged in buffer u (kb - kb0 is even)
      // every global load below is unconditional (a wave past the last tile
      // streams tile 0 and discards it), so that the compiler can count the
      // loads in flight and wait only for the ones each step consumes.  (The
      // products sit in a branch: without it the compiler rotated the
      // accumulators through other registers and copied them back every
      // iteration.)
      if (live) {
        u32x4 bx[2 * RG_RT];
#pragma unroll
        for (int i = 0; i < 2 * RG_RT; ++i) bx[i] = xs[u][i][lane];
#pragma unroll
        for (int rt = 0; rt < RG_RT; ++rt) {
#pragma unroll
          for (int n = 0; n < RG_NT; ++n) {
            acc[n][rt] = Ty<bf16_t>::mma(a[u][n], bx[2 * rt], acc[n][rt]);
            acc[n][rt] = Ty<bf16_t>::mma(a[u][n], bx[2 * rt + 1], acc[n][rt]);
          }
        }
      }
      // k-block k + 1 (loaded RG_D - 1 steps ago; zeros past the slice) into
      // the other buffer, which every wave has read before the last barrier;
      // k-block k + RG_D into the registers this one leaves (loads past the
      // slice re-read its last k-block)
      const int un = (u + 1) % RG_D;          // a constant once the loop is unrolled
#pragma unroll
      for (int j = 0; j < SJ; ++j) {
        xs[u ^ 1][2 * (wave + 4 * j)][lane] = sv[un][j][0];
        xs[u ^ 1][2 * (wave + 4 * j) + 1][lane] = sv[un][j][1];
      }
      if (k + 1 == kb1) {                     // uniform: the zero k-block of an odd slice
#pragma unroll
        for (int j = 0; j < SJ; ++j) {
          xs[u ^ 1][2 * (wave + 4 * j)][lane] = z4;
          xs[u ^ 1][2 * (wave + 4 * j) + 1][lane] = z4;
        }
      }
      const int kn = min(k + RG_D, kb1 - 1);
#pragma unroll
      for (int j = 0; j < SJ; ++j) {
        sv[u][j][0] = *(const u32x4 *)(sh[j] + (size_t)kn * 32);
        sv[u][j][1] = *(const u32x4 *)(sw[j] + (size_t)kn * 32);
      }
#pragma unroll
      for (int n = 0; n < RG_NT; ++n) a[u][n] = wp[n][(size_t)kn * 64];   // cached: shared
      __syncthreads();
    }
  }
  if (!live) return;
  const int q4 = lane >> 4;
#pragma unroll
  for (int rt = 0; rt < RG_RT; ++rt) {
    const int r = r0 + 16 * rt + (lane & 15);
    if (r >= g.R) continue;
    if (g.part) {   // slice partials for the finish pass
#pragma unroll
      for (int n = 0; n < RG_NT; ++n) {
        if (t0 + n >= m.n_tiles) continue;
        *(f32x4 *)(g.part + ((size_t)sl * g.R + r) * m.N + (t0 + n) * 16 + 4 * q4) = acc[n][rt];
      }
    } else {        // one slice, the epilogue here (row scales precomputed)
      const float sc = g.norm.scale ? g.norm.scale[r] : 1.f;
#pragma unroll
      for (int n = 0; n < RG_NT; ++n) {
        if (t0 + n >= m.n_tiles) continue;
        if (g.epi == EPI_SWIGLU) {   // z = SiLU(gate) * up; no shuffles, r < R
          (void)epilogue_tile<bf16_t, EPI_SWIGLU>(g, t0 + n, r, acc[n][rt], sc, -1, 0);
        } else {                     // EPI_STORE (the LM head): y[r][n] = scale[r] acc
          const f32x4 v = acc[n][rt];
          *(f32x4 *)(g.y + (size_t)r * g.ldy + (t0 + n) * 16 + 4 * q4) =
              f32x4{v.x * sc, v.y * sc, v.z * sc, v.w * sc};
        }
      }
    }
  }
}

// The products: 4 tiles per wave (ROWGRP_TILES per workgroup), up to 3
// workgroups per CU.
static_assert(4 * 4 == ROWGRP_TILES, "row-group tiling");
__global__ __launch_bounds__(256) void k_gemm_rows(GemmLaunch g) { gemm_rows_body<4>(g); }

// The LM head (one slice, EPI_STORE): 8 tiles per wave, which halves the LDS
// reads per MFMA; its 128 accumulators leave room for two waves per SIMD
// only if they share the VGPRs (LM head of the 8B scoring pass 504 -> 454 us).
constexpr int LMR_NT = 8;
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_lmhead_rows(GemmLaunch g) { gemm_rows_body<LMR_NT>(g); }

// the finish pass of a K-split product: one wave per (tile, 16 rows)
template <typename T>
static void finish_launch(const GemmLaunch &g, hipStream_t s) {
  const int ft = finish_tiles(g.m.n_tiles, g.epi);
  const dim3 fg(g.m.n_tiles / ft, (g.R + 15) / 16), fb(64 * ft);
  if (g.epi == EPI_NORM) hipLaunchKernelGGL((k_gemm_finish<T, EPI_NORM>), fg, fb, 0, s, g);
  else if (g.epi == EPI_SWIGLU) hipLaunchKernelGGL((k_gemm_finish<T, EPI_SWIGLU>), fg, fb, 0, s, g);
  else hipLaunchKernelGGL((k_gemm_finish<T, EPI_QKV>), fg, fb, 0, s, g);
}

// Whether a row-group product applies its epilogue in the kernel: the LM
// head's store, and a SwiGLU product of one slice (its row scales
// precomputed); the others write slice partials for the finish pass.
static bool rows_direct(const GemmLaunch &g) {
  return g.epi == EPI_STORE || (g.epi == EPI_SWIGLU && g.split == 1);
}

// Row-group product and, with slice partials, its finish pass.  false
// (nothing launched): rows or slices out of the kernel's range, a token
// resolution it does not do, or a direct epilogue without its operands.
static bool gemm_rows_launch(GemmLaunch g, hipStream_t s) {
  const int nk = g.m.nkb - g.kb_lo;
  const bool direct = rows_direct(g);
  if (g.R < 1 || g.R > ROWGRP_MAX_ROWS || g.split < 1 || g.split > nk || g.tok_out || !g.x.lo ||
      (direct && (g.split != 1 || (g.epi == EPI_STORE && !g.y) ||
                  (g.epi == EPI_SWIGLU && (!g.z.hi || (g.norm.n_parts > 0 && !g.norm.scale))))) ||
      (!direct && !g.part))
    return false;
  if (direct) g.part = nullptr;
  const bool lm = g.epi == EPI_STORE;
  const int tiles = lm ? 4 * LMR_NT : ROWGRP_TILES;   // per workgroup
  const long n_xg = (g.m.n_tiles + tiles - 1) / tiles;
  const long n_rg = (g.R + ROWGRP_ROWS - 1) / ROWGRP_ROWS;
  const long pairs = n_xg * g.split;
  const dim3 grid((unsigned)((pairs + 7) / 8 * 8 * n_rg));
  if (lm) hipLaunchKernelGGL(k_lmhead_rows, grid, dim3(256), 0, s, g);
  else hipLaunchKernelGGL(k_gemm_rows, grid, dim3(256), 0, s, g);
  if (!direct) finish_launch<bf16_t>(g, s);
  return true;
}

template <typename T, int RT, int NT, bool PAIR>
static void gemm_split_launch(const GemmLaunch &g, hipStream_t s) {
  const int groups = g.m.n_tiles / NT;
  const dim3 grid((groups + 3) / 4, g.split);
  bool staged = false;
  if constexpr (sizeof(T) == 2 && RT <= 2) {
    const int nk = g.m.nkb - g.kb_lo;
    const int nk_max = (nk + g.split - 1) / g.split;   // the longest slice
    if (nk_max * 2 * RT <= SPLIT_LDS_FRAGS) {
      hipLaunchKernelGGL((k_gemm_split_lds<RT, NT>), grid, dim3(256),
                         (size_t)nk_max * 2 * RT * 64 * sizeof(u32x4), s, g);
      staged = true;
    }
  }
  if (!staged) hipLaunchKernelGGL((k_gemm_split<T, RT, NT, PAIR>), grid, dim3(256), 0, s, g);
  finish_launch<T>(g, s);
}

template <typename T, bool PAIR>
static bool gemm_rt(const GemmLaunch &g, hipStream_t s) {
  if (g.rowgrp) {
    if constexpr (sizeof(T) == 2) return gemm_rows_launch(g, s);
    return false;
  }
  if (g.R > MAX_ROWS) return false;   // the kernels below hold at most 4 row tiles
  if (g.split > 0) {
    if (g.nt == 8) {
      if (g.R <= 16) gemm_split_launch<T, 1, 8, PAIR>(g, s);
      else if (g.R <= 32) gemm_split_launch<T, 2, 8, PAIR>(g, s);
      else gemm_split_launch<T, 4, 8, PAIR>(g, s);
    } else if (g.nt == 4) {
      if (g.R <= 16) gemm_split_launch<T, 1, 4, PAIR>(g, s);
      else if (g.R <= 32) gemm_split_launch<T, 2, 4, PAIR>(g, s);
      else gemm_split_launch<T, 4, 4, PAIR>(g, s);
    } else if (g.nt == 2) {
      if (g.R <= 16) gemm_split_launch<T, 1, 2, PAIR>(g, s);
      else if (g.R <= 32) gemm_split_launch<T, 2, 2, PAIR>(g, s);
      else gemm_split_launch<T, 4, 2, PAIR>(g, s);
    } else {
      if (g.R <= 16) gemm_split_launch<T, 1, 1, PAIR>(g, s);
      else if (g.R <= 32) gemm_split_launch<T, 2, 1, PAIR>(g, s);
      else gemm_split_launch<T, 4, 1, PAIR>(g, s);
    }
    return true;
  }
  if constexpr (sizeof(T) == 2) {
    if (g.gemv) {
      if (g.R <= 1) return gemm_epi<T, 1, 1, PAIR, 1>(g, s);
      return gemm_epi<T, 1, 1, PAIR, 2>(g, s);   // R <= GEMV_MAX_ROWS
    }
  }
  if (g.nt == 7) {          // gate/up shapes whose tile count is a multiple of 7 * 256
    if (g.R <= 16) return gemm_epi<T, 1, 7, PAIR, 0>(g, s);
    if (g.R <= 32) return gemm_epi<T, 2, 7, PAIR, 0>(g, s);
    return false;
  }
  if (g.nt == 8) {          // batched rows, many tiles: no K slices
    if (g.R <= 16) return gemm_epi<T, 1, 8, PAIR, 0>(g, s);
    if (g.R <= 32) return gemm_epi<T, 2, 8, PAIR, 0>(g, s);
    return false;
  }
  if (g.nt == 4) {
    if (g.R <= 16) return gemm_epi<T, 1, 4, PAIR, 0>(g, s);
    if (g.R <= 32) return gemm_epi<T, 2, 4, PAIR, 0>(g, s);
    return false;
  }
  if (g.nt == 2) {
    if (g.R <= 16) return gemm_epi<T, 1, 2, PAIR, 0>(g, s);
    if (g.R <= 32) return gemm_epi<T, 2, 2, PAIR, 0>(g, s);
    return gemm_epi<T, 4, 2, PAIR, 0>(g, s);
  }
  if (g.R <= 16) return gemm_epi<T, 1, 1, PAIR, 0>(g, s);
  if (g.R <= 32) return gemm_epi<T, 2, 1, PAIR, 0>(g, s);
  return gemm_epi<T, 4, 1, PAIR, 0>(g, s);
}

bool launch_gemm(bool bf16, const GemmLaunch &g, hipStream_t s) {
  if (bf16) return gemm_rt<bf16_t, true>(g, s);
  return gemm_rt<float, false>(g, s);
}

int lm_workgroups(int n_tiles, int nt) { return (n_tiles / nt + 3) / 4; }

int gemm_ss_parts(const GemmLaunch &g) {
  return g.split > 0 ? g.m.n_tiles / finish_tiles(g.m.n_tiles, g.epi) : g.m.n_tiles;
}

bool gemm_own_scales(const GemmLaunch &g, int n_parts) {
  if (g.rowgrp && rows_direct(g)) return false;   // no finish pass: scales precomputed
  if (g.split > 0) return scales_fit(64 * finish_tiles(g.m.n_tiles, g.epi), g.R < 16 ? g.R : 16, n_parts);
  return g.R <= MAX_ROWS && scales_fit(64 * g.kw, g.R, n_parts);
}

bool lm_own_scales(int R, int n_parts) { return R <= MAX_ROWS && scales_fit(256, R, n_parts); }

template <typename T, bool PAIR>
static void lm_rt(const LmLaunch &g, hipStream_t s) {
  const dim3 grid(g.n_wg), blk(256);
  if constexpr (sizeof(T) == 2) {
    if (g.gemv) {
      const size_t lds = gemv_lds_bytes(g.R, g.m.K);
      // one row (LM_GEMV_MAX_ROWS): more rows take the MFMA tiles
      if (g.nt == 4) hipLaunchKernelGGL((k_lmhead<T, 1, 4, PAIR, 1>), grid, blk, lds, s, g);
      else hipLaunchKernelGGL((k_lmhead<T, 1, 1, PAIR, 1>), grid, blk, lds, s, g);
      return;
    }
  }
  if (g.nt == 8) {   // eight tiles per wave share each B fragment
    if (g.R <= 16) hipLaunchKernelGGL((k_lmhead<T, 1, 8, PAIR, 0>), grid, blk, 0, s, g);
    else if (g.R <= 32) hipLaunchKernelGGL((k_lmhead<T, 2, 8, PAIR, 0>), grid, blk, 0, s, g);
    else hipLaunchKernelGGL((k_lmhead<T, 4, 8, PAIR, 0>), grid, blk, 0, s, g);
    return;
  }
  if (g.nt == 4) {   // four tiles per wave share each B fragment (batched rows)
    if (g.R <= 16) hipLaunchKernelGGL((k_lmhead<T, 1, 4, PAIR, 0>), grid, blk, 0, s, g);
    else if (g.R <= 32) hipLaunchKernelGGL((k_lmhead<T, 2, 4, PAIR, 0>), grid, blk, 0, s, g);
    else hipLaunchKernelGGL((k_lmhead<T, 4, 4, PAIR, 0>), grid, blk, 0, s, g);
    return;
  }
  if (g.nt == 2) {
    if (g.R <= 16) hipLaunchKernelGGL((k_lmhead<T, 1, 2, PAIR, 0>), grid, blk, 0, s, g);
    else if (g.R <= 32) hipLaunchKernelGGL((k_lmhead<T, 2, 2, PAIR, 0>), grid, blk, 0, s, g);
    else hipLaunchKernelGGL((k_lmhead<T, 4, 2, PAIR, 0>), grid, blk, 0, s, g);
  } else {
    if (g.R <= 16) hipLaunchKernelGGL((k_lmhead<T, 1, 1, PAIR, 0>), grid, blk, 0, s, g);
    else if (g.R <= 32) hipLaunchKernelGGL((k_lmhead<T, 2, 1, PAIR, 0>), grid, blk, 0, s, g);
    else hipLaunchKernelGGL((k_lmhead<T, 4, 1, PAIR, 0>), grid, blk, 0, s, g);
  }
}

void launch_lmhead(bool bf16, const LmLaunch &g, hipStream_t s) {
  if (bf16) lm_rt<bf16_t, true>(g, s);
  else lm_rt<float, false>(g, s);
}

// LM head over many rows at once, logits only (the target's tree-scoring
// pass: up to LMR_MAX_ROWS rows in one launch): the row-group product with
// one K slice, its epilogue storing logits[r][v] = scale[r] * acc (the final
// RMSNorm's row scale comes precomputed).
bool lmhead_rows_fits(const TiledMat &m, int R) {
  return R >= 1 && R <= LMR_MAX_ROWS && R <= ROWGRP_MAX_ROWS && m.nkb >= 1;
}

void launch_lmhead_rows(const LmRowsArgs &a, hipStream_t s) {
  GemmLaunch g{};
  g.m = a.m;
  g.x = a.x;
  g.R = a.R;
  g.split = 1;
  g.rowgrp = 1;
  g.epi = EPI_STORE;         // the kernel stores y itself
  g.y = a.logits;
  g.ldy = a.ld_logits;
  g.norm.scale = a.scale;
  gemm_rows_launch(g, s);
}

// Embedding half of a fusion FC for every token: T[v][n] = sum_{k < H}
// W[n][k] E[v][k].  Wave w of workgroup (x, y) takes feature tile 4 x + w
// against vocab rows 64 y .. 64 y + 63: W's tiled blocks are the A operand
// as stored, E's rows the B operand, fp32 accumulation.  Runs at load time.
__global__ __launch_bounds__(256) void k_embed_table(const u32x4 *__restrict__ w, int nkb_w,
                                                     int kb_n, const bf16_t *__restrict__ E, int V,
                                                     int H, int N, float *__restrict__ T) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, q4 = lane >> 4;
  const int tile = blockIdx.x * 4 + wave;
  const int v0 = blockIdx.y * 64;
  const u32x4 *wp = w + (size_t)tile * nkb_w * 64 + lane;
  const bf16_t *er[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int v = min(v0 + 16 * j + col, V - 1);
    er[j] = E + (size_t)v * H + 8 * q4;
  }
  f32x4 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int kb = 0; kb < kb_n; ++kb) {
    const u32x4 a = wp[(size_t)kb * 64];
    u32x4 b[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) b[j] = *(const u32x4 *)(er[j] + (size_t)kb * 32);
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = Ty<bf16_t>::mma(a, b[j], acc[j]);
  }
  // lane (col, q4) holds features 16 tile + 4 q4 + i of vocab row col
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int v = v0 + 16 * j + col;
    if (v < V) *(f32x4 *)(T + (size_t)v * N + 16 * tile + 4 * q4) = acc[j];
  }
}

void launch_embed_table(const TiledMat &w, const void *embed, int V, int H, float *T, hipStream_t s) {
  const dim3 grid(w.N / 64, (V + 63) / 64);
  hipLaunchKernelGGL(k_embed_table, grid, dim3(256), 0, s, (const u32x4 *)w.w, w.nkb, H / 32,
                     (const bf16_t *)embed, V, H, w.N, T);
}

// Repack a row-major [n_src_rows, K] matrix into the tiled layout: source row
// i goes to destination row i*row_stride + row_offset (used to concatenate
// q/k/v and to interleave gate/up); destination rows below rot_rows belong to
// rotated heads of size d and use the pair-aligned permutation.  One thread
// per 16-byte destination fragment.
template <typename T>
__global__ void k_repack(const T *__restrict__ src, int n_src_rows, int K, int row_stride,
                         int row_offset, int rot_rows, int d, u32x4 *__restrict__ dst, int n_tiles,
                         int nkb) {
  constexpr int E = Ty<T>::E, KB = Ty<T>::KB;
  const size_t total = (size_t)n_tiles * nkb * 64;
  for (size_t f = (size_t)blockIdx.x * blockDim.x + threadIdx.x; f < total;
       f += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(f & 63);
    const size_t tj = f >> 6;
    const int j = (int)(tj % nkb);
    const int t = (int)(tj / nkb);
    const int i = lane & 15;
    int drow = t * 16 + i;
    if (drow < rot_rows) {
      // tile jj of head h: rows 0..7 -> dims 8jj..8jj+7, rows 8..15 -> d/2 + 8jj..
      const int h = (t * 16) / d, jj = ((t * 16) % d) / 16;
      drow = h * d + (i < 8 ? 8 * jj + i : d / 2 + 8 * jj + (i - 8));
    }
    const int rel = drow - row_offset;
    if (rel < 0 || rel % row_stride) continue;
    const int srow = rel / row_stride;
    if (srow >= n_src_rows) continue;
    const int k0 = j * KB + (lane >> 4) * E;
    dst[f] = *(const u32x4 *)(src + (size_t)srow * K + k0);
  }
}

void launch_repack(bool bf16, const void *src, int n_src_rows, int K, int row_stride,
                   int row_offset, int rot_rows, int d, TiledMat &dst, hipStream_t s) {
  const size_t total = (size_t)dst.n_tiles * dst.nkb * 64;
  const int blocks = (int)((total + 255) / 256 < 65536 ? (total + 255) / 256 : 65536);
  if (bf16)
    hipLaunchKernelGGL(k_repack<bf16_t>, dim3(blocks), dim3(256), 0, s, (const bf16_t *)src,
                       n_src_rows, K, row_stride, row_offset, rot_rows, d, (u32x4 *)dst.w,
                       dst.n_tiles, dst.nkb);
  else
    hipLaunchKernelGGL(k_repack<float>, dim3(blocks), dim3(256), 0, s, (const float *)src,
                       n_src_rows, K, row_stride, row_offset, rot_rows, d, (u32x4 *)dst.w,
                       dst.n_tiles, dst.nkb);
}

}  // namespace prism
