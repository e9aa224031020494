// RoPE angle table and the per-row output statistics of the LM head.
#include "internal.h"

namespace ssm {

// ---- RoPE table (rotate-half form), float64 arithmetic -------------------
__global__ void rope_table_kernel(const int32_t* __restrict__ pos, int n_rows, int half, int dh,
                                  double base, float2* __restrict__ tab) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n_rows * half) return;
  const int r = idx / half, i = idx % half;
  const double inv_freq = 1.0 / pow(base, (2.0 * i) / (double)dh);
  const double a = (double)pos[r] * inv_freq;
  tab[idx] = make_float2((float)cos(a), (float)sin(a));
}

hipError_t launch_rope_table(const int32_t* pos, int n_rows, int dh, float base, float2* tab,
                             hipStream_t st) {
  const int half = dh / 2, n = n_rows * half;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_table_kernel, dim3(ceil_div(n, 256)), dim3(256), 0, st, pos, n_rows,
                     half, dh, (double)base, tab);
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
  hipLaunchKernelGGL(rowstats_kernel, dim3(rows), dim3(256), 0, st, logits, V, ldl, mask_id, k,
                     argmax, conf, topk_ids, topk_w);
  return hipGetLastError();
}

}  // namespace ssm
