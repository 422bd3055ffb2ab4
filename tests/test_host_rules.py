"""Host unit tests of the library's plain-C++ rules, compiled with g++ (no GPU).

* tree_order.h: the candidate order of the draft tree (as a comparison and as
  integer keys) and the ancestor walk, on NaN, infinity and tie inputs.  The kernels rank candidates by it, so
  ranks must form a permutation whatever the scores are.  If they do not,
  two candidates share a slot and another slot is never written.
* plan.h: the launch plan of every product of every configured shape and row
  count fits the kernel instantiation that it selects, and the tree
  attention's row groups divide the tree width and fit the 16 score columns.
"""
import itertools
import math
import os
import struct
import subprocess

import pytest

from synth import CONFIGS, SMALL_BF16_CHAIN, SMALL_BF16_TREE, SMALL_F32_CHAIN

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2602_01762_amd", "csrc")

DRIVER = r"""
#define __host__
#define __device__
#include <cstdio>
#include <cstring>
#include <cstdint>
#include "tree_order.h"
#include "plan.h"
using namespace prism;

static float f_of(uint32_t u) { float f; std::memcpy(&f, &u, 4); return f; }

int main() {
  char cmd[16];
  while (std::scanf("%15s", cmd) == 1) {
    if (!std::strcmp(cmd, "rank")) {          // n, then n float bit patterns
      int n; std::scanf("%d", &n);
      float s[4096];
      for (int i = 0; i < n; ++i) { unsigned u; std::scanf("%x", &u); s[i] = f_of(u); }
      for (int i = 0; i < n; ++i) {
        int r = 0;
        for (int j = 0; j < n; ++j) r += tree_before(s[j], j, s[i], i);
        std::printf("%d ", r);
      }
      std::printf("\n");
    } else if (!std::strcmp(cmd, "rankk")) {  // the same ranks by the integer keys
      int n; std::scanf("%d", &n);
      uint64_t k[4096];
      for (int i = 0; i < n; ++i) { unsigned u; std::scanf("%x", &u); k[i] = tree_rank_key(f_of(u), i); }
      for (int i = 0; i < n; ++i) {
        int r = 0;
        for (int j = 0; j < n; ++j) r += k[j] > k[i] ? 1 : 0;
        std::printf("%d ", r);
      }
      std::printf("\n");
    } else if (!std::strcmp(cmd, "anc")) {    // n, then n parents
      int n; std::scanf("%d", &n);
      int par[64];
      for (int i = 0; i < n; ++i) std::scanf("%d", &par[i]);
      for (int i = 0; i < n; ++i) std::printf("%llx ", (unsigned long long)tree_ancestor_bits(par, i));
      std::printf("\n");
    } else if (!std::strcmp(cmd, "plan")) {   // n_tiles nkb K K_full R qkv bf16 lds
      int nt, nkb, K, Kf, R, qkv, bf; long lds;
      std::scanf("%d %d %d %d %d %d %d %ld", &nt, &nkb, &K, &Kf, &R, &qkv, &bf, &lds);
      ProductPlan p = plan_product(nt, nkb, K, Kf, R, qkv != 0, bf != 0, (size_t)lds);
      const int rt = p.gemv ? 1 : row_tiles(R);
      std::printf("%d %d %d %d %d %d %d\n", p.kw, p.nt, p.split, p.gemv, plan_fits(p, R) ? 1 : 0,
                  product_max_waves(rt, p.gemv ? 1 : p.nt), p.rowgrp);
    } else if (!std::strcmp(cmd, "grp")) {    // bf16 nq nkv d w
      int bf, nq, nkv, d, w;
      std::scanf("%d %d %d %d %d", &bf, &nq, &nkv, &d, &w);
      std::printf("%d\n", attention_group(bf != 0, nq, nkv, d, w));
    } else if (!std::strcmp(cmd, "nsub")) {   // units nkv max_slots
      int u, nkv, ms;
      std::scanf("%d %d %d", &u, &nkv, &ms);
      const int ns = attention_nsub(u, nkv, ms);
      std::printf("%d %d\n", ns, attention_chunks(ms, ns));
    } else if (!std::strcmp(cmd, "part")) {   // rows_max grp grp2 nkv max_slots
      int rm, gp, gp2, nkv, ms, mc;
      std::scanf("%d %d %d %d %d", &rm, &gp, &gp2, &nkv, &ms);
      const long p = attention_partial_rows(rm, gp, gp2, nkv, ms, mc);
      std::printf("%ld %d\n", p, mc);
    } else if (!std::strcmp(cmd, "pfl")) {    // n_tiles nkb K rows_max
      int nt, nkb, K, rm;
      std::scanf("%d %d %d %d", &nt, &nkb, &K, &rm);
      std::printf("%zu\n", product_partial_floats(nt, nkb, K, rm));
    } else if (!std::strcmp(cmd, "sgrp")) {   // bf16 nq nkv d
      int bf, nq, nkv, d;
      std::scanf("%d %d %d %d", &bf, &nq, &nkv, &d);
      std::printf("%d\n", score_attention_group(bf != 0, nq, nkv, d));
    }
  }
  return 0;
}
"""


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    d = tmp_path_factory.mktemp("rules")
    src = d / "rules.cpp"
    src.write_text(DRIVER)
    exe = d / "rules"
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", "-Wno-unused-result", "-I", CSRC, str(src), "-o",
                    str(exe)], check=True)

    def run(text):
        return subprocess.run([str(exe)], input=text, check=True, capture_output=True,
                              text=True).stdout.split("\n")
    return run


def bits(x):
    return "%08x" % struct.unpack("<I", struct.pack("<f", x))[0]


def ranks(driver, scores, cmd="rank"):
    line = "%s %d %s\n" % (cmd, len(scores), " ".join(bits(s) for s in scores))
    return [int(t) for t in driver(line)[0].split()]


def expected_ranks(scores):
    """Rank of each candidate by sorting (score desc, index asc) with NaN last."""
    key = lambda i: (1, 0.0, i) if math.isnan(scores[i]) else (0, -scores[i], i)
    order = sorted(range(len(scores)), key=key)
    r = [0] * len(scores)
    for pos, i in enumerate(order):
        r[i] = pos
    return r


NAN, INF = float("nan"), float("inf")
NEG_NAN = struct.unpack("<f", struct.pack("<I", 0xffc00001))[0]


@pytest.mark.parametrize("scores", [
    [0.0, -1.0, -0.5, -1.0, -2.0],                 # exact tie
    [NAN, -1.0, NAN, 0.0],                         # NaN last, among them by index
    [NAN] * 7,                                     # every score NaN
    [-INF, NAN, -INF, -3.0, INF],                  # infinities around NaN
    [-0.0, 0.0, -0.0],                             # signed zeros compare equal
    [NEG_NAN, NAN, -INF],                          # NaN of either sign
    [1e-45, -1e-45, 0.0, 3.4e38, -3.4e38],         # denormals, extremes
])
@pytest.mark.parametrize("cmd", ["rank", "rankk"])
def test_tree_order_is_a_total_order(driver, scores, cmd):
    got = ranks(driver, scores, cmd)
    assert sorted(got) == list(range(len(scores))), "ranks must be a permutation"
    assert got == expected_ranks(scores)


def test_tree_order_random_with_nan_and_ties(driver):
    import numpy as np
    rng = np.random.default_rng(0)
    for trial in range(20):
        n = int(rng.integers(1, 400))
        s = rng.choice([-1.0, -0.5, 0.0, NAN, -INF], size=n).astype(np.float32)
        s = np.where(rng.random(n) < 0.5, s, rng.normal(size=n).astype(np.float32))
        scores = [float(x) for x in s]
        want = expected_ranks(scores)
        assert ranks(driver, scores) == want
        assert ranks(driver, scores, "rankk") == want


def test_ancestor_walk_is_bounded_and_exact(driver):
    # a valid tree: 0 and 1 under the root, 2 under 0, 3 under 2, 4 under 1
    out = driver("anc 5 -1 -1 0 2 1\n")[0].split()
    assert [int(x, 16) for x in out] == [0b1, 0b10, 0b101, 0b1101, 0b10010]
    # corrupt parents (self loop, cycle, forward link, out of range) stop the walk
    out = driver("anc 5 0 2 1 7 -9\n")[0].split()
    assert [int(x, 16) for x in out] == [0b1, 0b10, 0b110, 0b1000, 0b10000]


def _products(cfg):
    """(n_tiles, nkb, K, K_full, qkv) of every product a pass of cfg runs."""
    bf = cfg.dtype == "bf16"
    kq = 32 if bf else 16
    H, I = cfg.hidden, cfg.ffn
    tab = bf and H % 64 == 0
    out = []
    for F in {cfg.feat_width, H}:
        lo = H // kq if tab else 0
        out.append((H // 16, (H + F) // kq - lo, H + F - lo * kq, H + F, False))
    out.append((cfg.qkv_dim // 16, H // kq, H, H, True))
    out.append((H // 16, cfg.n_q_heads * cfg.head_dim // kq, cfg.n_q_heads * cfg.head_dim,
                cfg.n_q_heads * cfg.head_dim, False))
    out.append((2 * I // 16, H // kq, H, H, False))
    out.append((H // 16, I // kq, I, I, False))
    return out


def test_every_plan_fits_its_kernel(driver):
    cfgs = list(CONFIGS.values()) + [SMALL_BF16_CHAIN, SMALL_BF16_TREE, SMALL_F32_CHAIN]
    # the parity tests' wide-FFN and odd-hidden variants
    cfgs += [SMALL_BF16_CHAIN.with_(ffn=6400), SMALL_BF16_CHAIN.with_(ffn=12800),
             SMALL_BF16_CHAIN.with_(hidden=480, feat_width=1440)]
    lines, cases = [], []
    for cfg in cfgs:
        bf = 1 if cfg.dtype == "bf16" else 0
        for (nt, nkb, K, Kf, qkv), R, lds in itertools.product(
                _products(cfg), range(1, 65), (65536, 163840)):
            lines.append("plan %d %d %d %d %d %d %d %d" % (nt, nkb, K, Kf, R, qkv, bf, lds))
            cases.append((cfg.name, nt, nkb, R, qkv, lds))
    out = driver("\n".join(lines) + "\n")
    assert len([o for o in out if o]) == len(cases)
    for case, o in zip(cases, out):
        kw, nt, split, gemv, fits, maxw, rowgrp = (int(x) for x in o.split())
        assert fits == 1 and 1 <= kw <= maxw and rowgrp == 0, (case, o)
        if split == 0 and not gemv:
            assert 64 * kw <= 64 * maxw
            # instantiations the launcher dispatches unsplit
            assert nt in (1, 2, 4, 7, 8), (case, o)
            if nt in (4, 7, 8):
                assert case[3] <= 32 and not case[4], (case, o)
        if split > 0:
            assert nt in (1, 2, 4, 8), (case, o)
        if gemv:
            assert case[3] <= 2 and nt == 1


def test_tree_attention_groups(driver):
    cfgs = list(CONFIGS.values()) + [SMALL_BF16_TREE, SMALL_BF16_CHAIN]
    cases = [(1 if c.dtype == "bf16" else 0, c.n_q_heads, c.n_kv_heads, c.head_dim, w)
             for c in cfgs for w in range(1, 17)]
    cases += [(1, 32, 8, 256, 8), (0, 32, 8, 128, 8), (1, 64, 8, 128, 6), (1, 32, 32, 64, 12)]
    out = driver("".join("grp %d %d %d %d %d\n" % c for c in cases))
    for (bf, nq, nkv, d, w), o in zip(cases, out):
        gs = int(o)
        g = nq // nkv
        assert gs >= 1 and w % gs == 0 and gs * g <= 16 or gs == 1, (bf, nq, nkv, d, w, gs)
        if not bf or d not in (64, 128):
            assert gs == 1
        else:   # the largest such divisor
            best = max(k for k in range(1, w + 1) if w % k == 0 and (k * g <= 16 or k == 1))
            assert gs == best, (nq, nkv, d, w, gs)
    # the workloads' trees: 4 rows of 4 query heads per workgroup
    assert driver("grp 1 32 8 128 8\n")[0] == "4"
    t = SMALL_BF16_TREE
    assert driver("grp 1 %d %d %d %d\n" % (t.n_q_heads, t.n_kv_heads, t.head_dim,
                                           t.tree_width))[0] == "4"


@pytest.mark.parametrize("rows_max,grp,grp2,nkv,max_slots", [
    (32, 4, 4, 8, 1152), (4, 1, 4, 8, 1152), (1, 1, 1, 8, 4096), (32, 1, 4, 8, 4096),
    (16, 1, 16, 8, 4096), (2, 4, 1, 2, 448), (64, 2, 4, 8, 131072), (8, 8, 1, 1, 64),
    (32, 4, 4, 8, 16), (256, 4, 4, 8, 1152), (256, 1, 16, 32, 4096), (256, 2, 2, 8, 131072)])
def test_attention_partials_cover_every_pass(driver, rows_max, grp, grp2, nkv, max_slots):
    """Steps per workgroup: a power of two up to 16, the fewest that keep a
    pass at most 512 workgroups; the partial buffers hold rows x chunks of
    every pass of 1..rows_max rows: single rows, groups of grp or grp2 rows,
    and runs of rps rows (trees) grouped from each run's first row."""
    part, most_ch = (int(x) for x in driver("part %d %d %d %d %d\n" % (
        rows_max, grp, grp2, nkv, max_slots))[0].split())

    def chunks(units):
        ns, ch = (int(x) for x in driver("nsub %d %d %d\n" % (units, nkv, max_slots))[0].split())
        assert ns in (1, 2, 4, 8, 16)
        assert ch == -(-max_slots // (64 * ns))
        assert units * nkv * ch <= 512 or ns == 16
        if ns > 1:   # the fewest such steps
            assert units * nkv * -(-max_slots // (64 * (ns // 2))) > 512
        return ch

    seen_rc, seen_ch = 0, 0
    for R in range(1, rows_max + 1):
        for gs in {1, grp, grp2}:
            ch = chunks(-(-R // gs))
            assert R * ch <= part
            seen_rc, seen_ch = max(seen_rc, R * ch), max(seen_ch, ch)
    assert (part, most_ch) == (seen_rc, seen_ch)
    # runs of rps rows (trees of rps - 1 nodes) in groups of grp2: more
    # workgroup rows than ceil(R / grp2), never more chunks per row
    for rps in (2, 5, 17, 61, 64):
        for n_runs in range(1, rows_max // rps + 1, 3):
            R = n_runs * rps
            units = n_runs * -(-rps // grp2)
            assert R * chunks(units) <= part


def test_gate_up_tiles_fill_whole_rounds(driver):
    """The 8B gate/up (1792 tiles) at 16 and 32 rows and the 70B one (3584
    tiles) at 32 rows run unsplit at 7 tiles per wave: 256 and 512 tile
    groups, whole rounds of the 256 CUs."""
    for n_tiles, K, R, groups in ((1792, 4096, 16, 256), (1792, 4096, 32, 256),
                                  (3584, 8192, 32, 512)):
        o = driver("plan %d %d %d %d %d 0 1 163840\n" % (n_tiles, K // 32, K, K, R))[0]
        kw, nt, split, gemv, fits, maxw, rowgrp = (int(x) for x in o.split())
        assert (nt, split, gemv, fits, rowgrp) == (7, 0, 0, 1, 0), o
        assert n_tiles // nt == groups


def test_row_group_plans_for_scoring_passes(driver):
    """Passes of more than 64 rows (tree scoring, whole trees up to 256 rows)
    take the row-group kernel in bf16: at least one K slice, at most a
    quarter of the k-blocks (so every slice has k-blocks), about 512
    workgroups of 16 tiles x 64 rows in all.  fp32 contexts never plan them
    (their passes stay within 64 rows; the launcher refuses such a plan)."""
    cfgs = list(CONFIGS.values()) + [SMALL_BF16_CHAIN, SMALL_BF16_TREE, SMALL_F32_CHAIN,
                                     SMALL_BF16_CHAIN.with_(hidden=480, feat_width=1440)]
    lines, cases = [], []
    for cfg in cfgs:
        bf = 1 if cfg.dtype == "bf16" else 0
        for (nt, nkb, K, Kf, qkv), R in itertools.product(_products(cfg), (65, 100, 183, 244, 256)):
            lines.append("plan %d %d %d %d %d %d %d 163840" % (nt, nkb, K, Kf, R, qkv, bf))
            cases.append((cfg.name, bf, nt, nkb, R))
    out = driver("\n".join(lines) + "\n")
    for (name, bf, n_tiles, nkb, R), o in zip(cases, out):
        kw, nt, split, gemv, fits, maxw, rowgrp = (int(x) for x in o.split())
        assert rowgrp == bf and gemv == 0, (name, n_tiles, nkb, R, o)
        if not bf:
            continue
        assert 1 <= split <= max(1, nkb // 4), (name, n_tiles, nkb, R, o)
        base = -(-n_tiles // 16) * -(-R // 64)
        if nkb // 4 >= split + 1:   # not capped by the k-blocks: the nearest count to 512
            assert abs(base * split - 512) <= base / 2 + 1e-9, (name, n_tiles, nkb, R, o)
    # the 8B scoring passes (4 trees of 61 rows): FC 8, QKV 5, O 8, gate/up 1, down 8 slices
    o = [driver("plan %d %d %d %d 244 %d 1 163840\n" % c)[0].split()[2] for c in (
        (256, 384, 12288, 16384, 0), (384, 128, 4096, 4096, 1), (256, 128, 4096, 4096, 0),
        (1792, 128, 4096, 4096, 0), (256, 448, 14336, 14336, 0))]
    assert o == ["8", "5", "8", "1", "8"]


@pytest.mark.parametrize("bf,nq,nkv,d,want", [
    (1, 32, 8, 128, 4), (1, 32, 32, 128, 16), (1, 64, 8, 128, 2), (1, 24, 8, 64, 5),
    (1, 32, 8, 256, 1), (0, 32, 8, 128, 1), (1, 32, 2, 128, 1), (1, 30, 8, 128, 1)])
def test_scoring_attention_groups(driver, bf, nq, nkv, d, want):
    """Tree-scoring rows per attention workgroup: as many rows of g = nq / nkv
    query heads as fit the 16 score columns (bf16, head dims 64 and 128)."""
    gs = int(driver("sgrp %d %d %d %d\n" % (bf, nq, nkv, d))[0])
    assert gs == want
    if gs > 1:
        assert gs * (nq // nkv) <= 16 < (gs + 1) * (nq // nkv)


def test_partial_buffer_holds_every_plan(driver):
    """The K-slice partial buffer (sized at creation by
    product_partial_floats over the full K of each matrix) holds split x rows
    x N floats for the plan of every product at every batched row count: up
    to 256 rows for bf16 (tree-scoring passes), 64 for fp32, the fusion FC
    planned over its feature columns only."""
    cfgs = list(CONFIGS.values()) + [SMALL_BF16_CHAIN, SMALL_BF16_TREE, SMALL_F32_CHAIN,
                                     SMALL_BF16_CHAIN.with_(ffn=6400),
                                     SMALL_BF16_CHAIN.with_(hidden=480, feat_width=1440)]
    for cfg in cfgs:
        bf = 1 if cfg.dtype == "bf16" else 0
        kq = 32 if bf else 16
        rows_max = 256 if bf else 64
        prods = _products(cfg)
        sizes = driver("".join("pfl %d %d %d %d\n" % (nt, Kf // kq, Kf, rows_max)
                               for (nt, nkb, K, Kf, qkv) in prods))
        size = max(int(x) for x in sizes if x)
        lines, cases = [], []
        for (nt, nkb, K, Kf, qkv), R in itertools.product(prods, range(3, rows_max + 1)):
            lines.append("plan %d %d %d %d %d %d %d 163840" % (nt, nkb, K, Kf, R, qkv, bf))
            cases.append((nt, R))
        out = driver("\n".join(lines) + "\n")
        for (nt, R), o in zip(cases, out):
            split = int(o.split()[2])
            assert split * R * 16 * nt <= size, (cfg.name, nt, R, split, size)


def test_plans_on_random_shapes(driver):
    """Seeded random product shapes (tile counts, k-block counts, rows up to
    256, both dtypes, with and without a feature-column range): every plan
    fits its kernel, row-group plans appear exactly above 64 rows (bf16),
    every slice count leaves each slice at least one k-block, and the
    partial buffer sized for the shape holds split x rows x N."""
    import numpy as np
    rng = np.random.default_rng(1234)
    lines, cases = [], []
    for _ in range(300):
        bf = int(rng.integers(0, 2))
        kq = 32 if bf else 16
        nt = int(rng.integers(1, 2049))
        nkb_full = int(rng.integers(1, 900))
        lo = int(rng.integers(0, nkb_full)) if rng.random() < 0.3 else 0
        nkb = nkb_full - lo
        R = int(rng.integers(3, 257 if bf else 65))
        qkv = int(rng.random() < 0.2)
        lines.append("plan %d %d %d %d %d %d %d 163840" % (nt, nkb, nkb * kq, nkb_full * kq, R, qkv, bf))
        lines.append("pfl %d %d %d %d" % (nt, nkb_full, nkb_full * kq, 256 if bf else 64))
        cases.append((bf, nt, nkb, R))
    out = [o for o in driver("\n".join(lines) + "\n") if o]
    assert len(out) == 2 * len(cases)
    for i, (bf, nt, nkb, R) in enumerate(cases):
        kw, tiles, split, gemv, fits, maxw, rowgrp = (int(x) for x in out[2 * i].split())
        size = int(out[2 * i + 1])
        assert fits == 1, (bf, nt, nkb, R, out[2 * i])
        assert rowgrp == (1 if bf and R > 64 else 0), (bf, nt, nkb, R, out[2 * i])
        if split > 0:
            assert split <= nkb, (bf, nt, nkb, R, split)
            assert split * R * 16 * nt <= size, (bf, nt, nkb, R, split, size)
