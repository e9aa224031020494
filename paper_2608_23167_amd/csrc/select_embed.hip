// Compacted row list of the sparse input (Section 3.2, Eq. 1-5) and the
// soft suffix embedding of its rows (Section 3.2, Eq. 6-8).
#include "internal.h"
#include "dcheck.h"

namespace ssm {

// Row r of sequence s gathers the token at its own position pos[r] - pad[s]
// (-1 for padding rows, whose position is negative).
__global__ void __launch_bounds__(256) select_kernel(SelectLayout L, const int32_t* __restrict__ tokens,
                                                     int seq_len, int32_t* __restrict__ pos,
                                                     int32_t* __restrict__ tok_c,
                                                     int8_t* __restrict__ region, int cap, Pads pads) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= L.n_rows) return;
  int p, g;
  row_position(L, r, p, g);
  SSM_DCHECK(r < cap && p >= 0 && p < seq_len);
  const int s = blockIdx.y;
  if (s == 0) {
    pos[r] = p;
    if (region) region[r] = (int8_t)g;
  }
  const int q = p - pads.of(s);
  tok_c[(size_t)s * cap + r] = (q >= 0 && q < seq_len) ? tokens[(size_t)s * seq_len + q] : -1;
}

hipError_t launch_select(const SelectLayout& L, int batch, int seq_len, const int32_t* tokens,
                         int32_t* pos, int32_t* tok_c, int8_t* region, int cap, const Pads& pads,
                         hipStream_t st) {
  if (L.n_rows == 0) return hipSuccess;
  dim3 grid(ceil_div(L.n_rows, 256), batch);
  launch(select_kernel, grid, dim3(256), 0, st, L, tokens, seq_len, pos, tok_c,
                     region, cap, pads);
  return hipGetLastError();
}

// One workgroup per (row, sequence).  An out-of-range id or position makes
// the row NaN instead of reading outside the tables; a padding row (its
// position pos[r] - pad[s] below zero) is the [MASK] embedding.
template <typename T>
__global__ void __launch_bounds__(256) embed_kernel(
    const T* __restrict__ E, int d, int vocab, int mask_id, int seq_len,
    const int32_t* __restrict__ tok_c, int tok_stride, const int32_t* __restrict__ pos,
    const int8_t* __restrict__ region, int n_rows, const int32_t* __restrict__ pred_ids,
    const float* __restrict__ pred_w, const int32_t* __restrict__ pred_step, int prev_step, int k,
    float alpha, float* __restrict__ x, Pads pads) {
  const int r = blockIdx.x, s = blockIdx.y;
  float* out = x + ((size_t)s * n_rows + r) * d;
  const int p = pos[r] - pads.of(s);
  const bool pad = pos[r] >= 0 && p < 0;
  const bool pos_ok = p >= 0 && p < seq_len;
  const size_t sp = (size_t)s * seq_len + (pos_ok ? p : 0);
  const bool soft = pos_ok && region[r] >= 2 && prev_step >= 0 && pred_step[sp] == prev_step;
  SSM_DCHECK(k >= 1 && k <= 8 && (pos_ok || pad));
  if (!soft) {
    const int tok = pad ? mask_id : tok_c[(size_t)s * tok_stride + r];
    const bool ok = (pos_ok || pad) && tok >= 0 && tok < vocab;
    SSM_DCHECK(ok);
    const T* e = E + (size_t)(ok ? tok : 0) * d;
    for (int c = threadIdx.x; c < d; c += blockDim.x) out[c] = ok ? ldf(e + c) : __builtin_nanf("");
    return;
  }
  int ids[8];
  float w[8];
  bool ok = true;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    ids[i] = 0;
    w[i] = 0.f;
    if (i < k) {
      ids[i] = pred_ids[sp * k + i];
      w[i] = pred_w[sp * k + i];
      ok = ok && ids[i] >= 0 && ids[i] < vocab;
    }
  }
  SSM_DCHECK(ok);
  const T* em = E + (size_t)mask_id * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float acc = 0.f;  // Eq. 7: sum_i w_i e_{id_i}, in the stored order
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (i < k) acc = acc + w[i] * ldf(E + (size_t)(ok ? ids[i] : 0) * d + c);
    const float v = (1.0f - alpha) * ldf(em + c) + alpha * acc;  // Eq. 8
    out[c] = ok ? v : __builtin_nanf("");
  }
}

// Vector form for d a multiple of 8 and 16-byte aligned tables and output:
// thread t handles columns 8c .. 8c + 7 (c = t, t + 256, ...), 16-byte table
// loads and two 16-byte stores; per element the same arithmetic in the same
// order as embed_kernel.
__device__ __forceinline__ void load8f(const bf16_t* p, float (&v)[8]) {
  const u32x4_t w = *(const u32x4_t*)p;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[2 * j] = __uint_as_float(w[j] << 16);
    v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8f(const float* p, float (&v)[8]) {
  const float4 a = ((const float4*)p)[0], b = ((const float4*)p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

template <typename T>
__global__ void __launch_bounds__(256) embed8_kernel(
    const T* __restrict__ E, int d, int vocab, int mask_id, int seq_len,
    const int32_t* __restrict__ tok_c, int tok_stride, const int32_t* __restrict__ pos,
    const int8_t* __restrict__ region, int n_rows, const int32_t* __restrict__ pred_ids,
    const float* __restrict__ pred_w, const int32_t* __restrict__ pred_step, int prev_step, int k,
    float alpha, float* __restrict__ x, Pads pads) {
  const int r = blockIdx.x, s = blockIdx.y, d8 = d >> 3;
  float* out = x + ((size_t)s * n_rows + r) * d;
  const int p = pos[r] - pads.of(s);
  const bool pad = pos[r] >= 0 && p < 0;
  const bool pos_ok = p >= 0 && p < seq_len;
  const size_t sp = (size_t)s * seq_len + (pos_ok ? p : 0);
  const bool soft = pos_ok && region[r] >= 2 && prev_step >= 0 && pred_step[sp] == prev_step;
  const float qnan = __builtin_nanf("");
  SSM_DCHECK(k >= 1 && k <= 8 && (pos_ok || pad));
  if (!soft) {
    const int tok = pad ? mask_id : tok_c[(size_t)s * tok_stride + r];
    const bool ok = (pos_ok || pad) && tok >= 0 && tok < vocab;
    SSM_DCHECK(ok);
    const T* e = E + (size_t)(ok ? tok : 0) * d;
    for (int c = threadIdx.x; c < d8; c += blockDim.x) {
      float v[8];
      load8f(e + 8 * c, v);
      if (!ok) {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = qnan;
      }
      ((float4*)(out + 8 * c))[0] = make_float4(v[0], v[1], v[2], v[3]);
      ((float4*)(out + 8 * c))[1] = make_float4(v[4], v[5], v[6], v[7]);
    }
    return;
  }
  int ids[8];
  float w[8];
  bool ok = true;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    ids[i] = 0;
    w[i] = 0.f;
    if (i < k) {
      ids[i] = pred_ids[sp * k + i];
      w[i] = pred_w[sp * k + i];
      ok = ok && ids[i] >= 0 && ids[i] < vocab;
    }
  }
  SSM_DCHECK(ok);
  const T* em = E + (size_t)mask_id * d;
  for (int c = threadIdx.x; c < d8; c += blockDim.x) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};   // Eq. 7, in the stored order
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i < k) {
        float e[8];
        load8f(E + (size_t)(ok ? ids[i] : 0) * d + 8 * c, e);
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = acc[j] + w[i] * e[j];
      }
    }
    float m[8], v[8];
    load8f(em + 8 * c, m);
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = ok ? (1.0f - alpha) * m[j] + alpha * acc[j] : qnan;   // Eq. 8
    ((float4*)(out + 8 * c))[0] = make_float4(v[0], v[1], v[2], v[3]);
    ((float4*)(out + 8 * c))[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
}

hipError_t launch_embed(int dtype, const void* E, int d, int vocab, int mask_id, int batch,
                        int seq_len, const int32_t* tok_c, int tok_stride, const int32_t* pos,
                        const int8_t* region, int n_rows, const int32_t* pred_ids,
                        const float* pred_w, const int32_t* pred_step, int prev_step, int k,
                        float alpha, float* x, const Pads& pads, hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  dim3 grid(n_rows, batch);
  const bool vec = d % 8 == 0 && ((uintptr_t)E & 15) == 0 && ((uintptr_t)x & 15) == 0;
  if (vec && dtype == 0)
    launch(embed8_kernel<float>, grid, dim3(256), 0, st, (const float*)E, d, vocab, mask_id,
           seq_len, tok_c, tok_stride, pos, region, n_rows, pred_ids, pred_w, pred_step,
           prev_step, k, alpha, x, pads);
  else if (vec)
    launch(embed8_kernel<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)E, d, vocab, mask_id,
           seq_len, tok_c, tok_stride, pos, region, n_rows, pred_ids, pred_w, pred_step,
           prev_step, k, alpha, x, pads);
  else if (dtype == 0)
    launch(embed_kernel<float>, grid, dim3(256), 0, st, (const float*)E, d, vocab,
                       mask_id, seq_len, tok_c, tok_stride, pos, region, n_rows, pred_ids, pred_w,
                       pred_step, prev_step, k, alpha, x, pads);
  else
    launch(embed_kernel<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)E, d, vocab,
                       mask_id, seq_len, tok_c, tok_stride, pos, region, n_rows, pred_ids, pred_w,
                       pred_step, prev_step, k, alpha, x, pads);
  return hipGetLastError();
}

// ---- row gather of activations -------------------------------------------
// One thread per 16-byte chunk: out[s, i, 8c .. 8c + 7] = src[s, pos[i], ...];
// positions outside [0, src_rows) give zeros.
__global__ void __launch_bounds__(256) gather_rows_kernel(const bf16_t* __restrict__ src,
                                                          int src_rows, int width,
                                                          const int32_t* __restrict__ pos,
                                                          int n_rows, bf16_t* __restrict__ dst) {
  const int c8n = width >> 3, s = blockIdx.y;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (size_t)n_rows * c8n) return;
  const int i = (int)(idx / c8n), c = (int)(idx % c8n);
  const int p = pos[i];
  u32x4_t v = {0u, 0u, 0u, 0u};
  if (p >= 0 && p < src_rows) v = *(const u32x4_t*)(src + ((size_t)s * src_rows + p) * width + c * 8);
  *(u32x4_t*)(dst + ((size_t)s * n_rows + i) * width + c * 8) = v;
}

hipError_t launch_gather_rows(int batch, int src_rows, int width, const bf16_t* src,
                              const int32_t* pos, int n_rows, bf16_t* dst, hipStream_t st) {
  const size_t n = (size_t)n_rows * (width / 8);
  if (n == 0 || batch == 0) return hipSuccess;
  launch(gather_rows_kernel, dim3((unsigned)((n + 255) / 256), batch), dim3(256), 0, st, src,
         src_rows, width, pos, n_rows, dst);
  return hipGetLastError();
}

}  // namespace ssm
