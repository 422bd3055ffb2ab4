// Device helpers for the gfx950 kernels: bf16 conversion, wave64 reductions,
// MFMA fragments.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <math.h>

#include "internal.h"

namespace prism {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

// round-to-nearest-even fp32 -> bf16 (NaN stays NaN)
__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

template <typename T> struct Ty;
template <> struct Ty<float> {
  static constexpr int E = 4;    // elements per 16-byte lane fragment
  static constexpr int KB = 16;  // k per tiled k-block
  __device__ static float ld(const float *p, size_t i) { return p[i]; }
  __device__ static void st(float *p, size_t i, float v) { p[i] = v; }
  // 4 MFMA 16x16x4 fp32 steps; element e of each lane is k-slot (lane>>4) of step e
  __device__ static f32x4 mma(u32x4 a, u32x4 b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
};
template <> struct Ty<bf16_t> {
  static constexpr int E = 8;
  static constexpr int KB = 32;
  __device__ static float ld(const bf16_t *p, size_t i) { return bf2f(p[i]); }
  __device__ static void st(bf16_t *p, size_t i, float v) { p[i] = (bf16_t)f2bf(v); }
  // one MFMA 16x16x32 bf16 step: lane l holds k = 8*(l>>4) .. +7 of row/col (l & 15)
  __device__ static f32x4 mma(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                    __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};

// ---- wave64 reductions (every lane ends with the same value, the same
// operation order on every run).  Partners within a row of 16 lanes come by
// DPP (quad permutes, then the half-row and row mirrors), which the VALU
// executes without the LDS permute unit; the four row results are then read
// as scalars and combined in row order. ----------------------------------
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, 0xf, 0xf, false);
}
constexpr int DPP_QUAD_XOR1 = 0xB1;      // quad_perm [1, 0, 3, 2]
constexpr int DPP_QUAD_XOR2 = 0x4E;      // quad_perm [2, 3, 0, 1]
constexpr int DPP_ROW_MIRROR = 0x140;    // lane i of a row <- lane 15 - i
constexpr int DPP_HALF_MIRROR = 0x141;   // lane i of a half-row <- lane 7 - i
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __uint_as_float(dpp_u32<CTRL>(__float_as_uint(v)));
}
__device__ __forceinline__ float readlane_f32(float v, int l) {
  return __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(v), l));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f32<DPP_QUAD_XOR1>(v));
  v = fmaxf(v, dpp_f32<DPP_QUAD_XOR2>(v));
  v = fmaxf(v, dpp_f32<DPP_HALF_MIRROR>(v));
  v = fmaxf(v, dpp_f32<DPP_ROW_MIRROR>(v));
  return fmaxf(fmaxf(readlane_f32(v, 0), readlane_f32(v, 16)),
               fmaxf(readlane_f32(v, 32), readlane_f32(v, 48)));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f32<DPP_QUAD_XOR1>(v);
  v += dpp_f32<DPP_QUAD_XOR2>(v);
  v += dpp_f32<DPP_HALF_MIRROR>(v);
  v += dpp_f32<DPP_ROW_MIRROR>(v);
  return (readlane_f32(v, 0) + readlane_f32(v, 16)) + (readlane_f32(v, 32) + readlane_f32(v, 48));
}
// Value of lane l ^ 32 / l ^ 16 by the gfx950 permlane swaps (VALU, no LDS).
// permlane32_swap(v, v) returns {v of lanes 0-31 in both halves, v of lanes
// 32-63 in both halves}; permlane16_swap(v, v) does the same for the even
// and odd rows of 16 within each half.
__device__ __forceinline__ float xor32_f(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}
__device__ __forceinline__ float xor16_f(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __uint_as_float((threadIdx.x & 16) ? r[0] : r[1]);
}
// larger value wins; equal values: lower id wins
__device__ __forceinline__ bool better(float v, int id, float ov, int oid) {
  // bitwise, not short-circuit: lane masks combine without exec-mask branches
  return (v > ov) | ((v == ov) & (id < oid));
}

// The same over N independent values (the results equal N separate calls;
// the DPP steps of different values are independent, so the compiler
// interleaves them)
template <int N>
__device__ __forceinline__ void wave_max_n(float (&v)[N]) {
#pragma unroll
  for (int b = 0; b < N; ++b) v[b] = wave_max(v[b]);
}
template <int N>
__device__ __forceinline__ void wave_sum_n(float (&v)[N]) {
#pragma unroll
  for (int b = 0; b < N; ++b) v[b] = wave_sum(v[b]);
}

// (value, id) candidates as one 64-bit key whose unsigned order is the
// candidate order above: larger value wins, equal values -> lower id.  The
// high word is the value mapped to an order-preserving unsigned integer (-0
// taken as +0, NaN lowest), the low word the complemented id.
__device__ __forceinline__ uint64_t cand_key(float v, int id) {
  uint32_t u = __float_as_uint(v + 0.0f);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  u = v != v ? 0u : u;
  return ((uint64_t)u << 32) | (uint64_t)(~(uint32_t)id);
}
__device__ __forceinline__ float key_value(uint64_t k) {
  const uint32_t u = (uint32_t)(k >> 32);
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u);
}
__device__ __forceinline__ int key_id(uint64_t k) { return (int)~(uint32_t)k; }
// Maxima of N keys at once; every lane ends with each maximum.  Within each
// row of 16 lanes the partners come by DPP (quad permutes, then the half-row
// and row mirrors), which the VALU executes; the four row maxima are then
// read as scalars.  No LDS permute is involved: a wave's 64-bit arg-max
// costs about 30 VALU operations instead of 12 dependent LDS permutes.
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_key(uint64_t k) {
  return ((uint64_t)dpp_u32<CTRL>((uint32_t)(k >> 32)) << 32) | dpp_u32<CTRL>((uint32_t)k);
}
__device__ __forceinline__ uint64_t readlane_key(uint64_t k, int l) {
  return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(k >> 32), l) << 32) |
         (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)k, l);
}
template <int N>
__device__ __forceinline__ void wave_max_key_n(uint64_t (&k)[N]) {
#pragma unroll
  for (int b = 0; b < N; ++b) { const uint64_t t = dpp_key<DPP_QUAD_XOR1>(k[b]); k[b] = t > k[b] ? t : k[b]; }
#pragma unroll
  for (int b = 0; b < N; ++b) { const uint64_t t = dpp_key<DPP_QUAD_XOR2>(k[b]); k[b] = t > k[b] ? t : k[b]; }
#pragma unroll
  for (int b = 0; b < N; ++b) { const uint64_t t = dpp_key<DPP_HALF_MIRROR>(k[b]); k[b] = t > k[b] ? t : k[b]; }
#pragma unroll
  for (int b = 0; b < N; ++b) { const uint64_t t = dpp_key<DPP_ROW_MIRROR>(k[b]); k[b] = t > k[b] ? t : k[b]; }
#pragma unroll
  for (int b = 0; b < N; ++b) {
    const uint64_t r0 = readlane_key(k[b], 0), r1 = readlane_key(k[b], 16);
    const uint64_t r2 = readlane_key(k[b], 32), r3 = readlane_key(k[b], 48);
    const uint64_t m01 = r1 > r0 ? r1 : r0, m23 = r3 > r2 ? r3 : r2;
    k[b] = m23 > m01 ? m23 : m01;
  }
}

// Arg-max of (value, id) over the wave by the same order as `better`
// (larger value wins, equal values -> lower id), on candidate keys; every
// lane ends with the winner.  (NaN ranks lowest here.)
__device__ __forceinline__ void wave_argmax(float &v, int &id) {
  uint64_t k[1] = {cand_key(v, id)};
  wave_max_key_n<1>(k);
  v = key_value(k[0]);
  id = key_id(k[0]);
}

// block-wide (256 threads = 4 waves) reductions through LDS, fixed order
__device__ __forceinline__ float block_sum(float v, float *sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
  const int nw = blockDim.x >> 6;
  for (int i = 0; i < nw; ++i) t += sh[i];
  return t;
}
__device__ __forceinline__ float block_max(float v, float *sh) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float t = -INFINITY;
  const int nw = blockDim.x >> 6;
  for (int i = 0; i < nw; ++i) t = fmaxf(t, sh[i]);
  return t;
}
__device__ __forceinline__ void block_argmax(float &v, int &id, float *shv, int *shi) {
  wave_argmax(v, id);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) { shv[w] = v; shi[w] = id; }
  __syncthreads();
  const int nw = blockDim.x >> 6;
  v = shv[0];
  id = shi[0];
  for (int i = 1; i < nw; ++i)
    if (better(shv[i], shi[i], v, id)) { v = shv[i]; id = shi[i]; }
}

// order a wave's LDS writes before its later reads (and the reverse) when
// the data is private to the wave, so no workgroup barrier is needed
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ float silu(float y) { return y / (1.0f + expf(-y)); }

// Token of row r from the LM head's top-1 partials (larger logit wins, ties
// -> lower id).  Every thread of the block calls it (block reduction) and
// gets the result; shv / shi hold one entry per wave.
constexpr int TOK_UNROLL = 4;
__device__ __forceinline__ int token_from_lm(const TokFromLm &t, int r, float *shv, int *shi) {
  float bv = -INFINITY;
  int bid = 0x7fffffff;
  const float *pv = t.pval + (size_t)r * t.n_wg;
  const int *pi = t.pid + (size_t)r * t.n_wg;
  for (int i0 = 0; i0 < t.n_wg; i0 += TOK_UNROLL * (int)blockDim.x) {
    float v[TOK_UNROLL];
    int id[TOK_UNROLL];
#pragma unroll
    for (int u = 0; u < TOK_UNROLL; ++u) {   // all loads first, then the compares
      const int i = i0 + u * blockDim.x + threadIdx.x;
      v[u] = i < t.n_wg ? pv[i] : -INFINITY;
      id[u] = i < t.n_wg ? pi[i] : 0x7fffffff;
    }
#pragma unroll
    for (int u = 0; u < TOK_UNROLL; ++u)
      if (better(v[u], id[u], bv, bid)) { bv = v[u]; bid = id[u]; }
  }
  block_argmax(bv, bid, shv, shi);
  return bid;
}

// The same resolved by one wave on its own (no workgroup barrier), in two
// halves so that the partials' loads can be issued ahead of other loads:
// the first PRE * 64 entries go out in issue_tok, the rest (larger grids)
// are read in finish_tok, which returns the token in every lane.
template <int PRE>
struct TokLoads {
  float v[PRE];
  int id[PRE];
};
template <int PRE>
__device__ __forceinline__ TokLoads<PRE> issue_tok(const TokFromLm &t, int r) {
  const int lane = threadIdx.x & 63;
  const float *pv = t.pval + (size_t)r * t.n_wg;
  const int *pi = t.pid + (size_t)r * t.n_wg;
  TokLoads<PRE> l;
#pragma unroll
  for (int u = 0; u < PRE; ++u) {
    const int i = u * 64 + lane;
    l.v[u] = i < t.n_wg ? pv[i] : -INFINITY;
    l.id[u] = i < t.n_wg ? pi[i] : 0x7fffffff;
  }
  return l;
}
template <int PRE>
__device__ __forceinline__ int finish_tok(const TokFromLm &t, int r, const TokLoads<PRE> &l) {
  const int lane = threadIdx.x & 63;
  float bv = -INFINITY;
  int bid = 0x7fffffff;
#pragma unroll
  for (int u = 0; u < PRE; ++u)
    if (better(l.v[u], l.id[u], bv, bid)) { bv = l.v[u]; bid = l.id[u]; }
  const float *pv = t.pval + (size_t)r * t.n_wg;
  const int *pi = t.pid + (size_t)r * t.n_wg;
  for (int i = PRE * 64 + lane; i < t.n_wg; i += 64)
    if (better(pv[i], pi[i], bv, bid)) { bv = pv[i]; bid = pi[i]; }
  wave_argmax(bv, bid);
  return bid;
}

}  // namespace prism
