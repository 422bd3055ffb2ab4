// Candidate order and ancestor walk of the draft tree.
//
// Plain C++ marked __host__ __device__: the tree kernels use these, and a
// host unit test compiles the same header with g++ (defining both markers
// empty) to check NaN, infinity and tie inputs on the CPU.  Nothing here
// includes a HIP header.
#pragma once
#include <stdint.h>

namespace prism {

// Order-preserving image of a score: a larger float gives a larger key,
// -0 and +0 give the same key, and NaN (any sign or payload) gives 0, below
// the key of -inf (0x007fffff).  So the order is total.
__host__ __device__ inline uint32_t tree_score_key(float s) {
  uint32_t u = __builtin_bit_cast(uint32_t, s + 0.0f);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return s != s ? 0u : u;
}

// Whether candidate j comes before candidate i: larger score first (NaN
// last), equal scores (two NaN included) by the lower creation index.  For
// n distinct indices the number of candidates before each one is a
// permutation of 0..n-1, whatever the scores.  So each rank slot below the
// cut gets exactly one writer.
__host__ __device__ inline bool tree_before(float sj, int j, float si, int i) {
  const uint32_t kj = tree_score_key(sj), ki = tree_score_key(si);
  return kj > ki || (kj == ki && j < i);
}

// The same order as one integer compare: tree_before(sj, j, si, i) holds
// exactly when tree_rank_key(sj, j) > tree_rank_key(si, i) (score key in the
// high half; the complemented index in the low half, so that of two equal
// scores the lower index compares higher).  i >= 0.
__host__ __device__ inline uint64_t tree_rank_key(float s, int i) {
  return ((uint64_t)tree_score_key(s) << 32) | (uint64_t)(~(uint32_t)i);
}

// Ancestor bitset of output node i (i < 64): bit i and the bit of every
// node on its path to the root.  par[n] is the output position of n's
// parent (-1: the root).  A selected tree has par[n] < n, because a parent
// never comes after its child in the order above: its score is at least
// the child's (a log-probability is <= 0, and a NaN parent makes the child
// NaN), and it was created first.  The walk follows only links that
// decrease, so it takes at most i steps whatever par holds.
__host__ __device__ inline uint64_t tree_ancestor_bits(const int *par, int i) {
  uint64_t m = 1ull << i;
  int n = i;
  while (true) {
    const int p = par[n];
    if (p < 0 || p >= n) break;
    m |= 1ull << p;
    n = p;
  }
  return m;
}

}  // namespace prism
