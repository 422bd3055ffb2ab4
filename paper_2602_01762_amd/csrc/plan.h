// Launch plans of the streamed products and the tree attention's row
// groups (host code, plain C++).
//
// The runtime plans every product with these functions, and the product
// kernels take their __launch_bounds__ from product_max_waves, so a plan
// and the kernel it launches agree by construction.  Nothing here includes a
// HIP header, so a host unit test compiles this header with g++ and checks
// the plans of every configured shape.
#pragma once
#include <stddef.h>

namespace prism {

// Rows up to which bf16 products take the VALU GEMV main loop (LM head: one
// row); above it the staged-activation LDS reads, which grow with the rows,
// cost more than the MFMA path's fixed 16-row tiles.
constexpr int GEMV_MAX_ROWS = 2;
constexpr int LM_GEMV_MAX_ROWS = 1;
constexpr int MAX_ROWS = 64;
constexpr int MAX_KW = 16;      // waves of one workgroup splitting K

// 16-row tiles of the batch (the MFMA B operand) a product instantiation
// holds: 1 up to 16 rows, 2 up to 32, else 4.
constexpr int row_tiles(int R) { return R <= 16 ? 1 : (R <= 32 ? 2 : 4); }

// Waves per workgroup a product instantiation allows (its __launch_bounds__
// / 64).  Variants with more accumulators (row tiles x tiles per wave >= 2)
// run at most 8 waves, which leaves them 256 VGPRs.
constexpr int product_max_waves(int rt, int nt) { return rt * nt >= 2 ? MAX_KW / 2 : MAX_KW; }

// Waves per workgroup of the K-sliced batched product (k_gemm_split).
constexpr int SPLIT_WAVES = 4;

// LDS of the staged activations of the GEMV main loop (fp32, one or two rows)
inline size_t gemv_lds_bytes(int R, int K) {
  const int vr = R <= 1 ? 1 : 2;
  return (size_t)vr * K * sizeof(float);
}

struct ProductPlan {
  int kw = 1;      // waves of one workgroup splitting K
  int nt = 1;      // output tiles per wave
  int split = 0;   // > 0: K slices across workgroups (batched path, then a finish pass)
  int gemv = 0;    // 1: VALU GEMV main loop (bf16, at most GEMV_MAX_ROWS rows)
  int rowgrp = 0;  // 1: row-group kernel (more than MAX_ROWS rows, bf16), K slices, finish pass
};

// Products over more than MAX_ROWS rows (tree-scoring passes of whole trees,
// bf16, up to ROWGRP_MAX_ROWS rows): workgroups of 4 waves take
// ROWGRP_TILES output tiles against one group of ROWGRP_ROWS rows over one K
// slice.  Slices: about ROWGRP_WGS workgroups in all (two per CU), at least
// 4 k-blocks each.
constexpr int ROWGRP_MAX_ROWS = 256;
constexpr int ROWGRP_TILES = 16;
constexpr int ROWGRP_ROWS = 64;
constexpr int ROWGRP_WGS = 512;
inline int rowgrp_split(int n_tiles, int nkb, int R) {
  const int base = (n_tiles + ROWGRP_TILES - 1) / ROWGRP_TILES * ((R + ROWGRP_ROWS - 1) / ROWGRP_ROWS);
  int sp = (ROWGRP_WGS + base / 2) / base;
  if (sp > nkb / 4) sp = nkb / 4;
  return sp < 1 ? 1 : sp;
}

// K slices of a batched product at nt tiles per wave: at most one workgroup
// of 4 waves per CU (longer slices stream better than more of them, and a
// grid just above the CU count leaves a few CUs with twice the work), at
// least 4 k-blocks per slice, and fp32 slice partials of at most 1/4 of the
// weight bytes (split * R * N * 4 <= N * K * 2 / 4; at 32 rows the tighter
// 1/8 cap left the 4096-wide products on 64-128 workgroups: tree 2.695 ->
// 2.662 ms; a 1/2 cap was 1.5% slower on the tree).
inline int batched_split(int n_tiles, int nt, int nkb, int K, int R) {
  const int wgs = (n_tiles / nt + SPLIT_WAVES - 1) / SPLIT_WAVES;
  int sp = 256 / wgs;
  if (sp > nkb / 4) sp = nkb / 4;
  if (sp > K / (8 * R)) sp = K / (8 * R);
  return sp < 1 ? 1 : sp;
}

// Batched products (more than GEMV_MAX_ROWS rows): tiles per wave (B
// fragment reuse: 4, or 8 at 17-32 rows, so that the activation fragments a
// wave loads stay within twice its weight fragments) and K slices across
// workgroups.  At 17-32 rows 8 tiles are taken unless the slice cap leaves
// their grid smaller than the 4-tile one (the tree's 4096-wide products:
// 128 workgroups at 8 tiles, 256 at 4; tree 2.342 -> 2.313 ms; at 70B both
// fill the chip, and 4 tiles there were 2.5% slower).
inline void plan_batched(int n_tiles, int nkb, int K, int R, int &nt, int &split) {
  nt = n_tiles % 4 == 0 ? 4 : (n_tiles % 2 == 0 ? 2 : 1);
  split = batched_split(n_tiles, nt, nkb, K, R);
  if (R > 16 && n_tiles % 8 == 0) {
    const int s8 = batched_split(n_tiles, 8, nkb, K, R);
    const long w8 = (long)(n_tiles / 8 + SPLIT_WAVES - 1) / SPLIT_WAVES * s8;
    const long w4 = (long)(n_tiles / nt + SPLIT_WAVES - 1) / SPLIT_WAVES * split;
    if (w8 >= w4) {
      nt = 8;
      split = s8;
    }
  }
}

// Rounds of a grid of `groups` workgroups over the 256 CUs, times the tiles
// each one streams: the relative time of an unsplit product at nt tiles per
// wave.
inline int unsplit_cost(int n_tiles, int nt) { return (n_tiles / nt + 255) / 256 * nt; }

// Plan of a product of an [N = 16 n_tiles, K] matrix over R rows.  nkb and K
// are those of the planned k range (the fusion FC may cover its feature
// columns only); K_full is the width of the staged operand; qkv: the QKV
// product (its epilogue runs on at most 2 tiles per wave); lds_limit: LDS
// bytes one workgroup may use.
inline ProductPlan plan_product(int n_tiles, int nkb, int K, int K_full, int R, bool qkv,
                                bool bf16, size_t lds_limit) {
  ProductPlan p;
  const int rt = row_tiles(R);
  if (R > MAX_ROWS) {   // the row-group kernel (bf16 only: fp32 passes stay within MAX_ROWS)
    p.rowgrp = bf16 ? 1 : 0;
    p.nt = 4;
    p.split = rowgrp_split(n_tiles, nkb, R);
    return p;
  }
  if (R > GEMV_MAX_ROWS) {
    plan_batched(n_tiles, nkb, K, R, p.nt, p.split);
    const int groups = n_tiles / p.nt;
    if (groups >= 200 && (p.nt == 4 || p.nt == 8) && rt <= 2 && !qkv) {
      // enough tile groups to fill the chip: K split across the waves of a
      // workgroup (LDS reduction, epilogue in the kernel), no finish pass;
      // about 1024 waves in all, within the instantiation's bound.  7 tiles
      // per wave where that fills whole rounds of the CUs and 4 or 8 do not
      // (gate/up, 1792 and 3584 tiles: 256 and 512 groups instead of 224 and
      // 448; batch 16 1.813 -> 1.790 ms, 70B 5.873 -> 5.838, tree -0.4%)
      p.split = 0;
      if (n_tiles % 7 == 0 && unsplit_cost(n_tiles, 7) < unsplit_cost(n_tiles, p.nt)) p.nt = 7;
      const int groups = n_tiles / p.nt;
      int kw = 1024 / groups;
      if (kw > product_max_waves(rt, p.nt)) kw = product_max_waves(rt, p.nt);
      while (kw > 1 && ((kw - 1) * p.nt * rt > 48 || kw > nkb / 4)) --kw;
      p.kw = kw < 1 ? 1 : kw;
    }
    return p;
  }
  // 1-2 rows: enough waves to cover HBM latency (about 16 per CU), at least
  // 4 k-blocks (4 KiB of W) per wave
  const int groups = n_tiles / p.nt;
  int kw = (4096 + groups - 1) / groups;
  if (kw > product_max_waves(rt, p.nt)) kw = product_max_waves(rt, p.nt);
  // up to 2 workgroups per CU: keep them co-resident (16 waves per CU) so
  // that a grid of, e.g., 1.5 workgroups per CU runs in one round
  if (groups <= 512 && groups > 256 && kw > 8) kw = 8;
  if (kw > nkb / 4) kw = nkb / 4;
  if (kw < 1) kw = 1;
  // LDS for the cross-wave sum: (kw - 1) * nt * rt KiB
  while (kw > 1 && (kw - 1) * p.nt * rt > 48) --kw;
  p.kw = kw;
  // GEMV main loop (bf16) when the staged activations fit in the
  // workgroup's LDS next to the cross-wave partial sums
  const size_t lds = gemv_lds_bytes(R, K_full) + (size_t)(kw - 1) * 64 * 16 + (size_t)64 * kw * 4;
  p.gemv = bf16 && lds <= lds_limit ? 1 : 0;
  if (p.gemv) p.nt = 1;
  return p;
}

// fp32 words of the K-slice partial sums ([split][rows][N]) that any
// batched product of an [N = 16 n_tiles, K] matrix (nkb k-blocks) writes at
// GEMV_MAX_ROWS + 1 .. rows_max rows.  The slices depend on the row count
// and the tiles per wave and do not shrink as K grows, so the full K bounds
// the fusion FC's feature-column products too.
inline size_t product_partial_floats(int n_tiles, int nkb, int K, int rows_max) {
  size_t most = 0;
  const size_t N = (size_t)16 * n_tiles;
  for (int rr = GEMV_MAX_ROWS + 1; rr <= rows_max; ++rr) {
    int sp = 0;
    if (rr > MAX_ROWS) {
      sp = rowgrp_split(n_tiles, nkb, rr);
    } else {
      for (int nt = 1; nt <= 8; nt *= 2) {
        if (n_tiles % nt) continue;
        const int s = batched_split(n_tiles, nt, nkb, K, rr);
        if (s > sp) sp = s;
      }
    }
    if ((size_t)rr * sp * N > most) most = (size_t)rr * sp * N;
  }
  return most;
}

// Whether a plan's workgroup fits the instantiation it launches (the
// launcher refuses a plan that does not).
inline bool plan_fits(const ProductPlan &p, int R) {
  if (p.split > 0) return true;   // SPLIT_WAVES per workgroup
  const int rt = p.gemv ? 1 : row_tiles(R);
  return p.kw >= 1 && p.kw <= product_max_waves(rt, p.gemv ? 1 : p.nt);
}

// Rows per workgroup of the grouped tree attention (rows of one sequence
// at tree width w): the largest divisor of w whose query rows, g = nq / nkv
// heads each, fit the 16 score columns of the MFMA tile; 1 = no grouping
// (fp32 caches and head dims other than 64 and 128 run ungrouped).
inline int attention_group(bool bf16, int nq, int nkv, int d, int w) {
  if (!bf16 || (d != 64 && d != 128) || nkv <= 0 || nq % nkv) return 1;
  const int g = nq / nkv;
  int gs = 1;
  for (int k = 2; k <= w && k * g <= 16; ++k)
    if (w % k == 0) gs = k;
  return gs;
}

constexpr int ATT_STEP = 64;          // KV slots per attention step
constexpr int ATT_MAX_SUB = 16;       // steps per attention workgroup
constexpr int ATT_MAX_CHUNKS = 1024;  // chunks per row the attention merge takes

// Chunks (of nsub steps) that cover max_slots slots.
inline int attention_chunks(int max_slots, int nsub) {
  return (max_slots + ATT_STEP * nsub - 1) / (ATT_STEP * nsub);
}

// Steps per workgroup of a pass with `units` workgroups per KV head and
// chunk (rows, or row groups): the fewest (a power of two up to ATT_MAX_SUB)
// that keep the grid at about 512 workgroups at capacity (two resident per
// CU), so that each streams several steps after its dependent lookups.  A
// pass with few rows gets short chunks and still fills the chip.
inline int attention_nsub(int units, int nkv, int max_slots) {
  int nsub = 1;
  while (nsub < ATT_MAX_SUB && (long)units * nkv * attention_chunks(max_slots, nsub) > 512) nsub *= 2;
  return nsub;
}

// Rows per workgroup of the tree-scoring attention (grouped from each
// tree's first row, the tree's last group possibly shorter): as many rows
// as fit the 16 score columns at g = nq / nkv query heads each; 1 = no
// grouping (fp32 caches and head dims other than 64 and 128).
inline int score_attention_group(bool bf16, int nq, int nkv, int d) {
  if (!bf16 || (d != 64 && d != 128) || nkv <= 0 || nq % nkv) return 1;
  const int g = nq / nkv;
  return g >= 16 ? 1 : 16 / g;
}

// Rows x chunks of the attention partials that any pass of 1..rows_max rows
// writes, single rows or in groups of grp or grp2 rows, and the most chunks
// of any one row; the partial buffers are sized from the first, and the
// second must not exceed ATT_MAX_CHUNKS.  A pass of R rows in groups of gs
// has at least ceil(R / gs) workgroup rows (more where groups restart at
// each tree), and the chunks per row do not grow with them.
inline long attention_partial_rows(int rows_max, int grp, int grp2, int nkv, int max_slots,
                                   int &max_chunks) {
  long most = 0;
  max_chunks = 0;
  for (int R = 1; R <= rows_max; ++R) {
    const int groups[3] = {1, grp, grp2};   // rows per workgroup
    for (int gs : groups) {
      if (gs < 1) continue;
      const int ch = attention_chunks(max_slots, attention_nsub((R + gs - 1) / gs, nkv, max_slots));
      if ((long)R * ch > most) most = (long)R * ch;
      if (ch > max_chunks) max_chunks = ch;
    }
  }
  return most;
}

}  // namespace prism
