// RMSNorm into projection operands, RoPE angle table and the per-row output
// statistics of the float32 LM head.
#include "internal.h"

namespace ssm {

// ---- RMSNorm: y = x / sqrt(mean(x^2) + eps) * g ----------------------------
// Vector form, one workgroup of 256 threads per row: thread t holds float4
// number t + 256 i of the row (i < NV) and the matching four gains, all
// loaded before the reduction, so a row costs one round trip to memory.
template <typename T> struct Gain4;
template <> struct Gain4<float> {
  __device__ __forceinline__ static float4 ld(const float* g) { return *(const float4*)g; }
};
template <> struct Gain4<bf16_t> {
  __device__ __forceinline__ static float4 ld(const bf16_t* g) {
    const uint2 u = *(const uint2*)g;
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
  }
};

template <typename T, int NV>
__global__ void __launch_bounds__(256) norm_vec_kernel(const float* __restrict__ x, int d,
                                                       const T* __restrict__ g, float eps,
                                                       ActOut y, int per, int stride, int off) {
  __shared__ float red[4];
  const int o = blockIdx.x, tid = threadIdx.x;
  const int nv4 = d >> 2;
  const float4* xr = (const float4*)(x + ((size_t)(o / per) * stride + off + o % per) * d);
  float4 v[NV], gv[NV];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int j = tid + 256 * i;
    if (j < nv4) {
      v[i] = xr[j];
      gv[i] = Gain4<T>::ld(g + 4 * j);
    } else {
      v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      gv[i] = v[i];
    }
  }
#pragma unroll
  for (int i = 0; i < NV; ++i) ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  ss = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int j = tid + 256 * i;
    if (j >= nv4) continue;
    const int c = 4 * j;
    const float r[4] = {v[i].x * inv * gv[i].x, v[i].y * inv * gv[i].y, v[i].z * inv * gv[i].z,
                        v[i].w * inv * gv[i].w};
    if constexpr (std::is_same<T, float>::value) {
      *(float4*)((float*)y.hi + (size_t)o * y.ld + c) = make_float4(r[0], r[1], r[2], r[3]);
    } else {
      uint16_t hi[4], lo[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        hi[e] = f2bf(r[e]);
        lo[e] = f2bf(r[e] - bf2f(hi[e]));
      }
      const size_t idx = frag_index(o, c, y.G);   // 4 consecutive columns share a chunk
      *(uint2*)((bf16_t*)y.hi + idx) = *(const uint2*)hi;
      if (y.lo) *(uint2*)(y.lo + idx) = *(const uint2*)lo;
    }
  }
}

// Any width: two passes, element by element.
template <typename T>
__global__ void __launch_bounds__(256) norm_kernel(const float* __restrict__ x, int d,
                                                   const T* __restrict__ g, float eps, ActOut y,
                                                   int n_rows, int per, int stride, int off) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + wave;
  if (o >= n_rows) return;
  const float* xr = x + ((size_t)(o / per) * stride + off + o % per) * d;
  float ss = 0.f;
  for (int c = lane; c < d; c += 64) ss += xr[c] * xr[c];
  ss = wave_sum(ss);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int c = lane; c < d; c += 64) y.store<T>(o, c, xr[c] * inv * ldf(g + c));
}

template <typename T>
static hipError_t norm_dispatch(const float* x, int d, const T* g, float eps, const ActOut& y,
                                int n_rows, int per, int stride, int off, hipStream_t st) {
  const bool aligned = ((uintptr_t)x & 15) == 0 && ((uintptr_t)g & (sizeof(T) * 4 - 1)) == 0;
  if (aligned && d % 4 == 0 && d <= 4 * 256 * 8) {
    const int nv = ceil_div(d / 4, 256);
    switch (nv) {
#define NORM_CASE(NV) \
  case NV: launch((norm_vec_kernel<T, NV>), dim3(n_rows), dim3(256), 0, st, x, d, g, eps, y, per, stride, off); return hipGetLastError();
      NORM_CASE(1) NORM_CASE(2) NORM_CASE(3) NORM_CASE(4) NORM_CASE(5) NORM_CASE(6)
      NORM_CASE(7) NORM_CASE(8)
#undef NORM_CASE
      default: break;
    }
  }
  launch(norm_kernel<T>, dim3(ceil_div(n_rows, 4)), dim3(256), 0, st, x, d, g, eps, y,
                     n_rows, per, stride, off);
  return hipGetLastError();
}

hipError_t launch_norm(int dtype, const float* x, int d, const void* g, float eps,
                       const ActOut& y, int n_rows, int per, int stride, int off, hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  if (dtype == 0) return norm_dispatch(x, d, (const float*)g, eps, y, n_rows, per, stride, off, st);
  return norm_dispatch(x, d, (const bf16_t*)g, eps, y, n_rows, per, stride, off, st);
}

// ---- RoPE table (rotate-half form), float64 arithmetic -------------------
// Table t (blockIdx.y) holds the angles of sequence t's positions pos[r] -
// pad[t]; padding rows (negative positions) take position 0.
__global__ void rope_table_kernel(const int32_t* __restrict__ pos, int n_rows, int half, int dh,
                                  double base, float2* __restrict__ tab, Pads pads) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n_rows * half) return;
  const int r = idx / half, i = idx % half, t = blockIdx.y;
  const int p = pos[r] - pads.of(t);
  const double inv_freq = 1.0 / pow(base, (2.0 * i) / (double)dh);
  const double a = (double)(p < 0 ? 0 : p) * inv_freq;
  tab[(size_t)t * n_rows * half + idx] = make_float2((float)cos(a), (float)sin(a));
}

hipError_t launch_rope_table(const int32_t* pos, int n_rows, int dh, float base, float2* tab,
                             int batch, const Pads& pads, hipStream_t st) {
  const int half = dh / 2, n = n_rows * half;
  if (n == 0) return hipSuccess;
  launch(rope_table_kernel, dim3(ceil_div(n, 256), pads.any ? batch : 1), dim3(256), 0, st, pos,
         n_rows, half, dh, (double)base, tab, pads);
  return hipGetLastError();
}

// ---- per-row statistics ----------------------------------------------------
// Candidate order: larger value first, then lower id.
__device__ __forceinline__ bool better(float v, int i, float w, int j) {
  return v > w || (v == w && i < j);
}

constexpr int KMAX = 8;

// Inserts (v, i) into the descending list (tv, ti) of length KMAX.
__device__ __forceinline__ void topk_insert(float (&tv)[KMAX], int (&ti)[KMAX], float v, int i) {
#pragma unroll
  for (int q = 0; q < KMAX; ++q) {
    const bool gt = better(v, i, tv[q], ti[q]);
    const float ov = tv[q];
    const int oi = ti[q];
    tv[q] = gt ? v : ov;
    ti[q] = gt ? i : oi;
    v = gt ? ov : v;
    i = gt ? oi : i;
  }
}

// One workgroup (256 threads) per row.  Deterministic: every reduction
// combines partial results in a fixed order.
__global__ void __launch_bounds__(256) rowstats_kernel(const float* __restrict__ logits, int V,
                                                       int ldl, int mask_id, int k,
                                                       int32_t* __restrict__ argmax,
                                                       float* __restrict__ conf,
                                                       int32_t* __restrict__ topk_ids,
                                                       float* __restrict__ topk_w) {
  __shared__ float s_m[256];
  __shared__ float s_s[256];
  __shared__ float s_v[4];
  __shared__ int s_i[4];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* L = logits + (size_t)row * ldl;
  float tv[KMAX];
  int ti[KMAX];
#pragma unroll
  for (int q = 0; q < KMAX; ++q) { tv[q] = -INFINITY; ti[q] = 0x7fffffff; }
  float m = -INFINITY, s = 0.f;
  for (int v = tid; v < V; v += 256) {
    if (v == mask_id) continue;
    const float x = L[v];
    if (x > m) { s = s * expf(m - x) + 1.0f; m = x; }
    else s += expf(x - m);
    if (better(x, v, tv[KMAX - 1], ti[KMAX - 1])) topk_insert(tv, ti, x, v);
  }
  // softmax normaliser: max, then rescaled sums, combined in thread order
  s_m[tid] = m;
  s_s[tid] = s;
  __syncthreads();
  if (tid == 0) {
    float M = -INFINITY;
    for (int t = 0; t < 256; ++t) M = fmaxf(M, s_m[t]);
    float S = 0.f;
    for (int t = 0; t < 256; ++t)
      if (s_s[t] > 0.f) S += s_s[t] * expf(s_m[t] - M);
    s_m[0] = M;
    s_s[0] = S;
  }
  __syncthreads();
  const float S = s_s[0];
  // top-k merge: KMAX rounds of a block-wide arg-best over the list heads
  float best_v[KMAX];
  int best_i[KMAX];
  for (int q = 0; q < KMAX; ++q) {
    float v = tv[0];
    int i = ti[0];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(v, o, 64);
      const int oi = __shfl_xor(i, o, 64);
      if (better(ov, oi, v, i)) { v = ov; i = oi; }
    }
    __syncthreads();
    if (lane == 0) { s_v[wave] = v; s_i[wave] = i; }
    __syncthreads();
    v = s_v[0];
    i = s_i[0];
    for (int w = 1; w < 4; ++w)
      if (better(s_v[w], s_i[w], v, i)) { v = s_v[w]; i = s_i[w]; }
    best_v[q] = v;
    best_i[q] = i;
    if (ti[0] == i && tv[0] == v) {  // the owner pops its head (ids are unique)
#pragma unroll
      for (int t = 0; t < KMAX - 1; ++t) { tv[t] = tv[t + 1]; ti[t] = ti[t + 1]; }
      tv[KMAX - 1] = -INFINITY;
      ti[KMAX - 1] = 0x7fffffff;
    }
  }
  if (tid == 0) {
    argmax[row] = best_i[0];
    conf[row] = 1.0f / S;   // exp(max - max) / sum exp(x - max)
    float z = 0.f;
    for (int q = 0; q < KMAX; ++q)
      if (q < k) z += expf(best_v[q] - best_v[0]);
    for (int q = 0; q < KMAX; ++q) {
      if (q < k) {
        topk_ids[(size_t)row * k + q] = best_i[q];
        topk_w[(size_t)row * k + q] = expf(best_v[q] - best_v[0]) / z;
      }
    }
  }
}

hipError_t launch_rowstats(const float* logits, int rows, int V, int ldl, int mask_id, int k,
                           int32_t* argmax, float* conf, int32_t* topk_ids, float* topk_w,
                           hipStream_t st) {
  if (rows == 0) return hipSuccess;
  launch(rowstats_kernel, dim3(rows), dim3(256), 0, st, logits, V, ldl, mask_id, k,
                     argmax, conf, topk_ids, topk_w);
  return hipGetLastError();
}

}  // namespace ssm
