// Decode attention of the drafting step over the paged draft KV cache, with
// causal or tree visibility, and the fused QKV epilogue (RoPE + cache append).
//
// Visibility of row r (sequence b, prior context L_b):
//   tree bits given:  slots [0, L_b)  plus  L_b + j for every set bit j
//   no tree bits:     slots [0, slot[r]]  (causal)
// Split-KV: a workgroup takes one (row, KV head, chunk of C slots) and all
// g = n_q/n_kv query heads that share the KV head; partial softmax states
// (max, sum, unnormalised output) are merged by a second kernel in chunk
// order, so the result does not depend on scheduling.
#include "device.h"

namespace prism {

constexpr int ATT_C = 256;     // slots per chunk = threads per workgroup
constexpr int ATT_MAXG = 8;    // query heads per KV head
constexpr int ATT_MAXD = 256;

struct AttnArgs {
  const void *q;              // [R, nq*d] storage dtype, RoPE applied
  const int32_t *seq, *slot;
  const uint64_t *bits;
  KvArgs kv;
  int R, nq, nkv, d, nch;     // nch: chunks per row in the partial buffers
  float scale;
  float *pm, *pl, *po;        // [R, nq, nch] / [R, nq, nch, d]
  void *o;                    // [R, nq*d]
  uint32_t *err;
};

__device__ __forceinline__ void row_range(const AttnArgs &a, int r, int &b, int &L, int &prefix,
                                          int &total, uint64_t &bits) {
  b = a.seq[r];
  if (b < 0 || b >= a.kv.n_seq) {   // invalid row: nothing visible (flagged)
    b = -1;
    L = prefix = total = 0;
    bits = 0ull;
    return;
  }
  L = a.kv.ctx_lens[b];
  bits = a.bits ? a.bits[r] : 0ull;
  if (a.bits) {
    prefix = L;
    total = L + (bits ? 64 - __clzll((long long)bits) : 0);
  } else {
    prefix = a.slot[r] + 1;
    total = prefix;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_attn_partial(AttnArgs a) {
  const int c = blockIdx.x, j = blockIdx.y, r = blockIdx.z;
  const int tid = threadIdx.x;
  int b, L, prefix, total;
  uint64_t bits;
  row_range(a, r, b, L, prefix, total, bits);
  if (b < 0) {
    if (c == 0 && j == 0 && tid == 0) atomicOr(a.err, ERRF_CAPACITY);
    return;
  }
  const int t0 = c * ATT_C;
  if (t0 >= total) return;
  const int t1 = min(t0 + ATT_C, total);
  const int d = a.d, g = a.nq / a.nkv;

  __shared__ float qs[ATT_MAXG * ATT_MAXD];
  __shared__ float ps[ATT_MAXG][ATT_C];
  __shared__ long offs[ATT_C];
  __shared__ float red[4096];

  const T *q = (const T *)a.q + (size_t)r * a.nq * d + (size_t)j * g * d;
  for (int e = tid; e < g * d; e += 256) qs[e] = Ty<T>::ld(q, e);

  // locate this thread's slot
  const int t = t0 + tid;
  long off = -1;
  if (t < t1) {
    bool vis = t < prefix || (a.bits && t >= L && ((bits >> (t - L)) & 1ull));
    if (vis) {
      const int bi = t / a.kv.bs;
      const int blk = bi < a.kv.mbps ? a.kv.block_table[(size_t)b * a.kv.mbps + bi] : -1;
      if (blk < 0 || blk >= a.kv.n_blocks) {
        atomicOr(a.err, ERRF_CAPACITY);
      } else {
        // pool layout [block, kv head, slot in block, d]
        off = ((long)blk * a.nkv + j) * a.kv.bs * d + (long)(t % a.kv.bs) * d;
      }
    }
  }
  offs[tid] = off;
  __syncthreads();

  // scores
  float s[ATT_MAXG];
#pragma unroll
  for (int h = 0; h < ATT_MAXG; ++h) s[h] = 0.f;
  if (off >= 0) {
    const T *kp = (const T *)a.kv.k_pool + off;
    constexpr int E = Ty<T>::E;
    for (int e0 = 0; e0 < d; e0 += E) {
      const u32x4 raw = *(const u32x4 *)(kp + e0);
      float kv[E];
      if constexpr (E == 8) {
        const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          kv[2 * i] = __uint_as_float(w4[i] << 16);
          kv[2 * i + 1] = __uint_as_float(w4[i] & 0xffff0000u);
        }
      } else {
        kv[0] = __uint_as_float(raw.x);
        kv[1] = __uint_as_float(raw.y);
        kv[2] = __uint_as_float(raw.z);
        kv[3] = __uint_as_float(raw.w);
      }
#pragma unroll
      for (int h = 0; h < ATT_MAXG; ++h) {
        if (h < g) {
#pragma unroll
          for (int i = 0; i < E; ++i) s[h] += qs[h * d + e0 + i] * kv[i];
        }
      }
    }
  }
#pragma unroll
  for (int h = 0; h < ATT_MAXG; ++h)
    if (h < g) ps[h][tid] = off >= 0 ? s[h] * a.scale : -INFINITY;
  __syncthreads();

  // softmax state per head: wave w handles heads w, w+4
  const int wave = tid >> 6, lane = tid & 63;
  for (int h = wave; h < g; h += 4) {
    float v0 = ps[h][lane], v1 = ps[h][lane + 64], v2 = ps[h][lane + 128], v3 = ps[h][lane + 192];
    const float m = wave_max(fmaxf(fmaxf(v0, v1), fmaxf(v2, v3)));
    float l;
    if (m == -INFINITY) {
      ps[h][lane] = ps[h][lane + 64] = ps[h][lane + 128] = ps[h][lane + 192] = 0.f;
      l = 0.f;
    } else {
      v0 = expf(v0 - m); v1 = expf(v1 - m); v2 = expf(v2 - m); v3 = expf(v3 - m);
      ps[h][lane] = v0; ps[h][lane + 64] = v1; ps[h][lane + 128] = v2; ps[h][lane + 192] = v3;
      l = wave_sum((v0 + v1) + (v2 + v3));
    }
    if (lane == 0) {
      const size_t pi = ((size_t)r * a.nq + j * g + h) * a.nch + c;
      a.pm[pi] = m;
      a.pl[pi] = l;
    }
  }
  __syncthreads();

  // P V: thread = (dim pair, slot group)
  const int npair = d >> 1, G = 256 / npair;
  const int pi2 = tid % npair, grp = tid / npair;
  float acc[ATT_MAXG][2];
#pragma unroll
  for (int h = 0; h < ATT_MAXG; ++h) acc[h][0] = acc[h][1] = 0.f;
  if (grp < G) {
    for (int tt = grp; tt < t1 - t0; tt += G) {
      const long o2 = offs[tt];
      if (o2 < 0) continue;
      const T *vp = (const T *)a.kv.v_pool + o2 + 2 * pi2;
      float v0, v1;
      if constexpr (sizeof(T) == 2) {
        const uint32_t w = *(const uint32_t *)vp;
        v0 = __uint_as_float(w << 16);
        v1 = __uint_as_float(w & 0xffff0000u);
      } else {
        v0 = vp[0];
        v1 = vp[1];
      }
#pragma unroll
      for (int h = 0; h < ATT_MAXG; ++h) {
        if (h < g) {
          const float p = ps[h][tt];
          acc[h][0] += p * v0;
          acc[h][1] += p * v1;
        }
      }
    }
  }
  // reduce over slot groups in group order
  if (grp < G) {
#pragma unroll
    for (int h = 0; h < ATT_MAXG; ++h)
      if (h < g) {
        red[(grp * g + h) * d + 2 * pi2] = acc[h][0];
        red[(grp * g + h) * d + 2 * pi2 + 1] = acc[h][1];
      }
  }
  __syncthreads();
  for (int e = tid; e < g * d; e += 256) {
    const int h = e / d, dim = e % d;
    float sum = 0.f;
    for (int gg = 0; gg < G; ++gg) sum += red[(gg * g + h) * d + dim];
    a.po[(((size_t)r * a.nq + j * g + h) * a.nch + c) * d + dim] = sum;
  }
}

template <typename T>
__global__ void k_attn_combine(AttnArgs a) {
  const int h = blockIdx.x, r = blockIdx.y, dim = threadIdx.x;
  int b, L, prefix, total;
  uint64_t bits;
  row_range(a, r, b, L, prefix, total, bits);
  if (total > a.nch * ATT_C) {
    if (h == 0 && dim == 0) atomicOr(a.err, ERRF_CAPACITY);
  }
  const int nch = min((total + ATT_C - 1) / ATT_C, a.nch);
  const size_t base = ((size_t)r * a.nq + h) * a.nch;
  float M = -INFINITY;
  for (int c = 0; c < nch; ++c) M = fmaxf(M, a.pm[base + c]);
  float lsum = 0.f, o = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float l = a.pl[base + c];
    if (l == 0.f) continue;
    const float w = expf(a.pm[base + c] - M);
    lsum += l * w;
    if (dim < a.d) o += a.po[(base + c) * a.d + dim] * w;
  }
  if (dim < a.d) Ty<T>::st((T *)a.o, (size_t)r * a.nq * a.d + (size_t)h * a.d + dim, o / lsum);
}

void launch_attention(bool bf16, int R, int nq, int nkv, int d, const void *q, const RowsIn &in,
                      const KvArgs &kv, int max_slots, int chunk, float *pm, float *pl, float *po,
                      void *o_out, uint32_t *err, hipStream_t s) {
  (void)chunk;
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
  a.nch = (max_slots + ATT_C - 1) / ATT_C;
  a.scale = 1.0f / sqrtf((float)d);
  a.pm = pm;
  a.pl = pl;
  a.po = po;
  a.o = o_out;
  a.err = err;
  dim3 g1(a.nch, nkv, R), g2(nq, R);
  const int th = d <= 64 ? 64 : (d <= 128 ? 128 : 256);
  if (bf16) {
    hipLaunchKernelGGL(k_attn_partial<bf16_t>, g1, dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_attn_combine<bf16_t>, g2, dim3(th), 0, s, a);
  } else {
    hipLaunchKernelGGL(k_attn_partial<float>, g1, dim3(256), 0, s, a);
    hipLaunchKernelGGL(k_attn_combine<float>, g2, dim3(th), 0, s, a);
  }
}

// ---------------------------------------------------------------------------
// QKV epilogue: sum the split-K partials of row r, rotate q and k (rotate-half
// pairs (i, i + d/2) by pos * theta^(-2i/d); angle in fp64, cos/sin rounded to
// fp32), write q in the storage dtype and k, v into the cache slot.
struct QkvArgs {
  const float *part;
  int splits, R, nq, nkv, d;
  RowsIn in;
  KvArgs kv;
  const double *inv_freq;   // [d/2]
  void *q_out;
  uint32_t *err;
};

template <typename T>
__global__ __launch_bounds__(256) void k_qkv_fin(QkvArgs a) {
  extern __shared__ float sh[];
  const int r = blockIdx.x, tid = threadIdx.x;
  const int d = a.d, half = d >> 1;
  const int N = (a.nq + 2 * a.nkv) * d;
  float *row = sh;             // [N]
  float *cs = sh + N;          // [half] cos, [half] sin
  for (int n = tid; n < N; n += blockDim.x) {
    float v = 0.f;
    for (int sp = 0; sp < a.splits; ++sp) v += a.part[((size_t)sp * a.R + r) * N + n];
    row[n] = v;
  }
  const int pos = a.in.pos[r];
  for (int i = tid; i < half; i += blockDim.x) {
    const double ang = (double)pos * a.inv_freq[i];
    cs[i] = (float)cos(ang);
    cs[half + i] = (float)sin(ang);
  }
  __syncthreads();
  // cache location of this row's slot
  const int b = a.in.seq[r];
  const int slot = a.in.slot[r];
  const int bi = slot / a.kv.bs;
  long base = -1;
  if (b >= 0 && b < a.kv.n_seq && slot >= 0 && bi < a.kv.mbps) {
    const int blk = a.kv.block_table[(size_t)b * a.kv.mbps + bi];
    if (blk >= 0 && blk < a.kv.n_blocks) base = (long)blk * a.nkv * a.kv.bs * d + (long)(slot % a.kv.bs) * d;
  }
  if (base < 0 && tid == 0) atomicOr(a.err, ERRF_CAPACITY);
  T *qo = (T *)a.q_out + (size_t)r * a.nq * d;
  const int nrot = (a.nq + a.nkv) * half;
  for (int e = tid; e < nrot; e += blockDim.x) {
    const int h = e / half, i = e % half;
    const float x1 = row[h * d + i], x2 = row[h * d + i + half];
    const float c = cs[i], sn = cs[half + i];
    const float y1 = x1 * c - x2 * sn;
    const float y2 = x2 * c + x1 * sn;
    if (h < a.nq) {
      Ty<T>::st(qo, (size_t)h * d + i, y1);
      Ty<T>::st(qo, (size_t)h * d + i + half, y2);
    } else if (base >= 0) {
      T *kp = (T *)a.kv.k_pool + base + (long)(h - a.nq) * a.kv.bs * d;
      Ty<T>::st(kp, i, y1);
      Ty<T>::st(kp, i + half, y2);
    }
  }
  if (base >= 0) {
    for (int e = tid; e < a.nkv * d; e += blockDim.x) {
      const int jh = e / d, dim = e % d;
      T *vp = (T *)a.kv.v_pool + base + (long)jh * a.kv.bs * d;
      Ty<T>::st(vp, dim, row[(a.nq + a.nkv) * d + e]);
    }
  }
}

void launch_qkv_fin(bool bf16, int R, int nq, int nkv, int d, const float *part, int splits,
                    const RowsIn &in, const KvArgs &kv, const double *inv_freq, void *q_out,
                    uint32_t *err, hipStream_t s) {
  QkvArgs a;
  a.part = part;
  a.splits = splits;
  a.R = R;
  a.nq = nq;
  a.nkv = nkv;
  a.d = d;
  a.in = in;
  a.kv = kv;
  a.inv_freq = inv_freq;
  a.q_out = q_out;
  a.err = err;
  const size_t lds = ((size_t)(nq + 2 * nkv) * d + d) * sizeof(float);
  if (bf16) hipLaunchKernelGGL(k_qkv_fin<bf16_t>, dim3(R), dim3(256), lds, s, a);
  else hipLaunchKernelGGL(k_qkv_fin<float>, dim3(R), dim3(256), lds, s, a);
}

}  // namespace prism
