// Skinny GEMMs of the drafting step on MFMA: Y[R, N] = X[R, K] . W[N, K]^T
// with R <= 64 rows (batch rows or tree nodes) and N, K in the thousands.
//
// These products are HBM-bound (a weight byte feeds 2R flops), so the design
// is about streaming W: W is pre-tiled so that every wave-wide load is one
// contiguous KiB (see TiledMat), each wave keeps U such loads in flight, and
// K is split across the waves of a workgroup (and across workgroups) until
// the grid holds enough waves to cover HBM latency.  The MFMA treats 16 rows
// of W as the M side and 16 rows of X as the N side; for R = 1 most of the
// B fragment is zero, which costs MFMA cycles that are idle anyway.
#include "device.h"

namespace prism {

constexpr int U = 8;  // k-blocks in flight per wave

template <typename T, int RT>
__device__ __forceinline__ void wave_mma(const u32x4 *__restrict__ wp, const T *__restrict__ X,
                                         int ldx, int R, int kb0, int kb1, f32x4 (&acc)[RT]) {
  constexpr int E = Ty<T>::E, KB = Ty<T>::KB;
  const int lane = threadIdx.x & 63;
  const int col = lane & 15, kq = lane >> 4;
  const T *xr[RT];
  bool ok[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = col + 16 * rt;
    ok[rt] = r < R;
    xr[rt] = X + (size_t)(ok[rt] ? r : 0) * ldx + kq * E;
  }
  wp += (size_t)kb0 * 64 + lane;
  int kb = kb0;
  for (; kb + U <= kb1; kb += U) {
    u32x4 a[U];
    u32x4 b[U][RT];
#pragma unroll
    for (int u = 0; u < U; ++u) a[u] = __builtin_nontemporal_load(wp + u * 64);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        b[u][rt] = ok[rt] ? *(const u32x4 *)(xr[rt] + (size_t)(kb + u) * KB) : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt] = Ty<T>::mma(a[u], b[u][rt], acc[rt]);
    wp += U * 64;
  }
  for (; kb < kb1; ++kb) {
    const u32x4 a = __builtin_nontemporal_load(wp);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const u32x4 b = ok[rt] ? *(const u32x4 *)(xr[rt] + (size_t)kb * KB) : u32x4{0, 0, 0, 0};
      acc[rt] = Ty<T>::mma(a, b, acc[rt]);
    }
    wp += 64;
  }
}

// Workgroup = 4 waves.  kw waves split the K range of one tile (summed in
// LDS in wave order), so a workgroup covers 4/kw tiles; grid.y = splits
// splits K further across workgroups (partials summed later in split order).
template <typename T, int RT, int EPI>
__global__ __launch_bounds__(256) void k_gemm(GemmLaunch g) {
  const TiledMat &m = g.m;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int tpw = 4 / g.kw;
  const int tile = blockIdx.x * tpw + wave / g.kw;
  const int ks = blockIdx.y * g.kw + wave % g.kw;
  const int nsl = g.splits * g.kw;
  const int kb0 = (int)((long)ks * m.nkb / nsl);
  const int kb1 = (int)((long)(ks + 1) * m.nkb / nsl);
  const bool live = tile < m.n_tiles;
  f32x4 acc[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (live)
    wave_mma<T, RT>((const u32x4 *)m.w + (size_t)tile * m.nkb * 64, (const T *)g.X, g.ldx, g.R,
                    kb0, kb1, acc);
  if (g.kw > 1) {
    __shared__ f32x4 red[4][RT][64];
    if (wave % g.kw) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) red[wave][rt][lane] = acc[rt];
    }
    __syncthreads();
    if (wave % g.kw == 0) {
      for (int j = 1; j < g.kw; ++j)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[rt] += red[wave + j][rt][lane];
    }
  }
  if (!live || (wave % g.kw) != 0) return;
  // lane holds output features n0..n0+3 of batch rows (lane & 15) + 16 rt
  const int n0 = tile * 16 + 4 * (lane >> 4);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = (lane & 15) + 16 * rt;
    if (r >= g.R) continue;
    if (EPI == EPI_PARTIAL) {
      *(f32x4 *)(g.part + ((size_t)blockIdx.y * g.R + r) * m.N + n0) = acc[rt];
    } else {
      // rows are interleaved (gate c, up c, gate c+1, up c+1)
      const int c = n0 >> 1;
      T *z = (T *)g.Z + (size_t)r * g.ldz + c;
      Ty<T>::st(z, 0, silu(acc[rt].x) * acc[rt].y);
      Ty<T>::st(z, 1, silu(acc[rt].z) * acc[rt].w);
    }
  }
}

// LM head: one wave per 16-row vocab tile over the full K, a workgroup per
// 64 vocab ids.  The epilogue reduces the workgroup's logits of each batch
// row to partials: max, sum of exp(logit - max), and the top-k
// (logit desc, id asc); optional fp32 logits store.
template <typename T, int RT>
__global__ __launch_bounds__(256) void k_lmhead(LmLaunch g) {
  const TiledMat &m = g.m;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int tile = blockIdx.x * 4 + wave;
  const bool live = tile < m.n_tiles;
  f32x4 acc[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (live)
    wave_mma<T, RT>((const u32x4 *)m.w + (size_t)tile * m.nkb * 64, (const T *)g.X, g.ldx, g.R,
                    0, m.nkb, acc);
  __shared__ float sl[RT * 16][65];
  const int q = lane >> 4;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = (lane & 15) + 16 * rt;
    if (r >= g.R) continue;
    const float v[4] = {acc[rt].x, acc[rt].y, acc[rt].z, acc[rt].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) sl[r][wave * 16 + 4 * q + i] = v[i];
    if (live && g.logits)
      *(f32x4 *)(g.logits + (size_t)r * g.ld_logits + tile * 16 + 4 * q) = acc[rt];
  }
  __syncthreads();
  for (int r = wave; r < g.R; r += 4) {
    const int id0 = blockIdx.x * 64 + lane;
    const bool valid = id0 < g.V;
    float v = valid ? sl[r][lane] : -INFINITY;
    int id = valid ? id0 : 0x7fffffff;
    const float mx = wave_max(v);
    const float s = wave_sum(valid ? expf(v - mx) : 0.f);
    const size_t pi = (size_t)r * g.n_wg + blockIdx.x;
    if (lane == 0) {
      g.pmax[pi] = mx;
      g.psum[pi] = s;
    }
    for (int j = 0; j < g.topk; ++j) {
      float bv = v;
      int bid = id;
      wave_argmax(bv, bid);
      if (lane == 0) {
        g.pval[pi * g.topk + j] = bv;
        g.pid[pi * g.topk + j] = bid;
      }
      if (id == bid) { v = -INFINITY; id = 0x7fffffff; }
    }
  }
}

template <typename T, int EPI>
static void gemm_rt(const GemmLaunch &g, hipStream_t s) {
  const int tpw = 4 / g.kw;
  dim3 grid((g.m.n_tiles + tpw - 1) / tpw, g.splits);
  if (g.R <= 16) hipLaunchKernelGGL((k_gemm<T, 1, EPI>), grid, dim3(256), 0, s, g);
  else if (g.R <= 32) hipLaunchKernelGGL((k_gemm<T, 2, EPI>), grid, dim3(256), 0, s, g);
  else hipLaunchKernelGGL((k_gemm<T, 4, EPI>), grid, dim3(256), 0, s, g);
}

void launch_gemm(bool bf16, int epi, const GemmLaunch &g, hipStream_t s) {
  if (bf16) {
    if (epi == EPI_PARTIAL) gemm_rt<bf16_t, EPI_PARTIAL>(g, s);
    else gemm_rt<bf16_t, EPI_SWIGLU>(g, s);
  } else {
    if (epi == EPI_PARTIAL) gemm_rt<float, EPI_PARTIAL>(g, s);
    else gemm_rt<float, EPI_SWIGLU>(g, s);
  }
}

int lm_workgroups(int n_tiles) { return (n_tiles + 3) / 4; }

template <typename T>
static void lm_rt(const LmLaunch &g, hipStream_t s) {
  dim3 grid(g.n_wg);
  if (g.R <= 16) hipLaunchKernelGGL((k_lmhead<T, 1>), grid, dim3(256), 0, s, g);
  else if (g.R <= 32) hipLaunchKernelGGL((k_lmhead<T, 2>), grid, dim3(256), 0, s, g);
  else hipLaunchKernelGGL((k_lmhead<T, 4>), grid, dim3(256), 0, s, g);
}

void launch_lmhead(bool bf16, const LmLaunch &g, hipStream_t s) {
  if (bf16) lm_rt<bf16_t>(g, s);
  else lm_rt<float>(g, s);
}

// Repack a row-major [n_src_rows, K] matrix into the tiled layout: source row
// i goes to destination row i*row_stride + row_offset (used to concatenate
// q/k/v and to interleave gate/up).  One thread per 16-byte destination
// fragment.
template <typename T>
__global__ void k_repack(const T *__restrict__ src, int n_src_rows, int K, int row_stride,
                         int row_offset, u32x4 *__restrict__ dst, int n_tiles, int nkb) {
  constexpr int E = Ty<T>::E, KB = Ty<T>::KB;
  const size_t total = (size_t)n_tiles * nkb * 64;
  for (size_t f = (size_t)blockIdx.x * blockDim.x + threadIdx.x; f < total;
       f += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(f & 63);
    const size_t tj = f >> 6;
    const int j = (int)(tj % nkb);
    const int t = (int)(tj / nkb);
    const int drow = t * 16 + (lane & 15);
    const int rel = drow - row_offset;
    if (rel < 0 || rel % row_stride) continue;
    const int srow = rel / row_stride;
    if (srow >= n_src_rows) continue;
    const int k0 = j * KB + (lane >> 4) * E;
    dst[f] = *(const u32x4 *)(src + (size_t)srow * K + k0);
  }
}

void launch_repack(bool bf16, const void *src, int n_src_rows, int K, int row_stride,
                   int row_offset, TiledMat &dst, hipStream_t s) {
  const size_t total = (size_t)dst.n_tiles * dst.nkb * 64;
  const int blocks = (int)((total + 255) / 256 < 65536 ? (total + 255) / 256 : 65536);
  if (bf16)
    hipLaunchKernelGGL(k_repack<bf16_t>, dim3(blocks), dim3(256), 0, s, (const bf16_t *)src,
                       n_src_rows, K, row_stride, row_offset, (u32x4 *)dst.w, dst.n_tiles, dst.nkb);
  else
    hipLaunchKernelGGL(k_repack<float>, dim3(blocks), dim3(256), 0, s, (const float *)src,
                       n_src_rows, K, row_stride, row_offset, (u32x4 *)dst.w, dst.n_tiles, dst.nkb);
}

}  // namespace prism
