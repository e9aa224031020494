// Internal launcher interfaces of the SSM HIP library.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <type_traits>

#include "common.h"

namespace ssm {

// ---- kernel launches -------------------------------------------------------
// With launch profiling on, prof_next hands out a pair of HIP events recorded
// under the current operation tag and the kernel's ordinal within that
// operation; it returns false when profiling is off.
bool prof_next(hipEvent_t* start, hipEvent_t* stop);

// Every kernel of the library is launched here; a profiled launch is
// bracketed by its own pair of events (created without the system-scope
// fence, so recording them does not write back the caches between kernels).
// Arguments are converted to the kernel's parameter types first.
template <typename... KArgs, typename... Args>
inline void launch(void (*kernel)(KArgs...), dim3 grid, dim3 block, uint32_t shmem,
                   hipStream_t st, Args&&... args) {
  static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel argument count");
  hipEvent_t a, b;
  const bool timed = prof_next(&a, &b);
  if (timed) hipEventRecord(a, st);
  hipLaunchKernelGGL(kernel, grid, block, shmem, st, static_cast<KArgs>(args)...);
  if (timed) hipEventRecord(b, st);
}

// Left padding of each sequence of a batch whose prompts differ in length.
// The batch shares one row layout, that of its longest prompt; sequence s,
// whose prompt is pad[s] tokens shorter, sits pad[s] positions to the left
// in it: row r of the layout is position pos[r] - pad[s] of that sequence,
// and rows whose position falls below zero are padding (embedded as [MASK],
// never read as keys).  The retained suffix of every sequence is that of the
// longest prompt shifted by pad[s] (its suffix regions are measured from its
// own block), so one position list serves the whole batch.  Passed to the
// kernels by value; `any` = 0 for a batch without padding.
constexpr int MAX_PAD_BATCH = 64;
struct Pads {
  int32_t v[MAX_PAD_BATCH];
  int32_t any;
  __host__ __device__ __forceinline__ int of(int s) const { return any ? v[s] : 0; }
};

// Closed-form layout of the compacted rows of one step (Section 3.2, Eq. 1-5).
struct SelectLayout {
  int n_prefix;      // prefix rows included (0 on a cached step)
  int P;             // first position of the current block
  int b;             // block size
  int s0;            // first suffix position
  int n_local;       // local tokens [s0, s0 + n_local)
  int mid_lo, mid_len, n_mid, mid_mode;
  int mid_first;     // block modes: the first kept middle position
  int mid_alt;       // start+end mode: 1 if that position is a block end (the
                     // first middle block is cut by the local region)
  int tail_lo, tail_len, n_tail, tail_mode;
  int n_suffix, n_rows;
};

// Row r of [prefix; block; local; middle; tail] -> (position, region).  Every
// row is computed independently in closed form, so the kernel is a pure
// coalesced map over rows.
__host__ __device__ inline void row_position(const SelectLayout& L, int r, int& p, int& g) {
  if (r < L.n_prefix) { p = r; g = 0; return; }
  r -= L.n_prefix;
  if (r < L.b) { p = L.P + r; g = 1; return; }
  r -= L.b;
  if (r < L.n_local) { p = L.s0 + r; g = 2; return; }
  r -= L.n_local;
  if (r < L.n_mid) {
    if (L.mid_mode == 0) {
      p = L.mid_lo + (int)(((long long)r * L.mid_len) / L.n_mid);
    } else if (L.mid_mode != 3) {            // block starts or block ends
      p = L.mid_first + r * L.b;
    } else if (L.mid_alt && r == 0) {        // the end of a block cut by the local region
      p = L.mid_first;
    } else {                                 // start, end of each block in turn
      const int q = r - L.mid_alt;
      p = L.mid_first + L.mid_alt + (q >> 1) * L.b + (q & 1) * (L.b - 1);
    }
    g = 3;
    return;
  }
  r -= L.n_mid;
  if (L.tail_mode == 1) p = L.tail_lo;
  else if (L.n_tail == 1) p = L.tail_lo + L.tail_len - 1;
  else p = L.tail_lo + (int)(((long long)r * (L.tail_len - 1)) / (L.n_tail - 1));
  g = 4;
}

hipError_t launch_select(const SelectLayout& L, int batch, int seq_len, const int32_t* tokens,
                         int32_t* pos, int32_t* tok_c, int8_t* region, int cap, const Pads& pads,
                         hipStream_t st);

// out[s, i, :] = src[s, pos[i], :] for bfloat16 rows of `width` elements.
hipError_t launch_gather_rows(int batch, int src_rows, int width, const bf16_t* src,
                              const int32_t* pos, int n_rows, bf16_t* dst, hipStream_t st);

hipError_t launch_embed(int dtype, const void* E, int d, int vocab, int mask_id, int batch,
                        int seq_len, const int32_t* tok_c, int tok_stride, const int32_t* pos,
                        const int8_t* region, int n_rows, const int32_t* pred_ids,
                        const float* pred_w, const int32_t* pred_step, int prev_step, int k,
                        float alpha, float* x, const Pads& pads, hipStream_t st);

// cos/sin of pos[r] * base^(-2i/dh) computed in float64, stored as float2
// [n_rows, dh / 2]; with padding, one table per sequence ([batch, n_rows,
// dh / 2]) at positions pos[r] - pad[s] (padding rows at position 0).
hipError_t launch_rope_table(const int32_t* pos, int n_rows, int dh, float base, float2* tab,
                             int batch, const Pads& pads, hipStream_t st);

// Per-row statistics of float32 logits [rows, ldl]: argmax, max probability,
// top-k ids and their renormalised weights, [MASK] excluded.
hipError_t launch_rowstats(const float* logits, int rows, int V, int ldl, int mask_id, int k,
                           int32_t* argmax, float* conf, int32_t* topk_ids, float* topk_w,
                           hipStream_t st);

// ---- projections -------------------------------------------------------
struct QKVOut {
  void* q;           // [B, H, n_rows, dh]
  void* kc;          // layer slice of the K cache [B, Hkv, cap, dh]
  void* vc;
  int cap, n_cached, n_rows;
  const float2* rope;
  int rope_per_seq;  // 1: one RoPE table per sequence (padded batch)
};

// Workspace for split-K partial sums, float32.
struct SplitWs {
  float* part;
  size_t floats;
};

// bfloat16 projection operands are stored in MFMA fragment order.  The
// matrix [M, K] (K a multiple of 64) is cut into 16-row groups and 64-column
// K-steps; each (K-step, group) pair owns two 1 KB halves of 16 rows x 32
// columns, and inside a half the 8-element chunk of row r, columns
// 8q .. 8q + 7, sits at chunk position 16q + r.  One 16-byte load per lane
// (lane 16q + r) then reads a whole half contiguously, already in the
// A-operand layout of v_mfma_f32_16x16x32_bf16; a row-major operand would
// touch 16 cache lines per load instruction instead of 8.  G is the number
// of row groups of the allocation; rows past M are padding, never stored
// back by any epilogue.
__host__ __device__ __forceinline__ size_t frag_index(int m, int k, int G) {
  return ((((size_t)(k >> 6) * G + (m >> 4)) * 2 + ((k >> 5) & 1)) * 64 + ((k >> 3) & 3) * 16 +
          (m & 15)) * 8 + (k & 7);
}
__host__ __device__ __forceinline__ int row_groups(int M) { return (M + 15) >> 4; }

// Activation operand of a projection: for bfloat16 models a bfloat16 array
// (hi) in fragment order with G row groups, plus an optional second
// bfloat16 part (lo) in the same order so that hi + lo carries the float32
// value; for float32 models `hi` is a row-major float32 array with row
// stride ld and lo is null.
struct ActIn {
  const void* hi;
  const bf16_t* lo;
  int ld;
  int G;
};

// Destination of an activation written by an epilogue, in the layout of
// ActIn: float32 row-major for float32 models; for bfloat16 models
// hi = bf16(v) and, if lo is not null, lo = bf16(v - hi), in fragment order;
// with f32 set, a bfloat16 kernel writes float32 row-major (row stride ld)
// instead (outputs handed back to a caller).
struct ActOut {
  void* hi;
  bf16_t* lo;
  int ld;
  int G;
  int f32;
  template <typename T>
  __device__ __forceinline__ void store(int m, int k, float v) const {
    if (std::is_same<T, float>::value || f32) {
      ((float*)hi)[(size_t)m * ld + k] = v;
    } else {
      const size_t i = frag_index(m, k, G);
      const bf16_t h = f2bf(v);
      ((bf16_t*)hi)[i] = h;
      if (lo) lo[i] = f2bf(v - bf2f(h));
    }
  }
  // columns k .. k + 7 of row m, k a multiple of 8: one chunk of the fragment
  // order, so one 16-byte store per part
  template <typename T>
  __device__ __forceinline__ void store8(int m, int k, const float (&v)[8]) const {
    if (std::is_same<T, float>::value || f32) {
      float* p = (float*)hi + (size_t)m * ld + k;
      *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
      *(float4*)(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
    } else {
      const size_t i = frag_index(m, k, G);
      uint16_t h[8], l[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        h[e] = f2bf(v[e]);
        l[e] = f2bf(v[e] - bf2f(h[e]));
      }
      *(u32x4_t*)((bf16_t*)hi + i) = *(const u32x4_t*)h;
      if (lo) *(u32x4_t*)(lo + i) = *(const u32x4_t*)l;
    }
  }
};

// RMSNorm of float32 rows into a projection operand: output row o reads
// input row (o / per) * stride + off + o % per.
hipError_t launch_norm(int dtype, const float* x, int d, const void* g, float eps,
                       const ActOut& y, int n_rows, int per, int stride, int off, hipStream_t st);

hipError_t gemm_qkv(int dtype, const ActIn& a, int M, int d, const void* wq, const void* wk,
                    const void* wv, int H, int Hkv, int dh, const QKVOut& out, SplitWs ws,
                    hipStream_t st);
// RMSNorm applied to the residual stream right after a residual projection:
// y = resid / rms(resid) * g, written as the next projection's operand.
struct NormTo {
  const void* g;
  float eps;
  ActOut y;
};
// resid += a * w^T; with `nrm`, the updated rows are also normalised into
// nrm->y (fused with the split-K completion when the projection splits K).
hipError_t gemm_resid(int dtype, const char* kind, const ActIn& a, int M, int K, const void* w,
                      int N, float* resid, SplitWs ws, hipStream_t st, const NormTo* nrm);
hipError_t gemm_swiglu(int dtype, const ActIn& a, int M, int d, const void* wg, const void* wu,
                       int F, const ActOut& act, SplitWs ws, hipStream_t st);
hipError_t gemm_store_f32(const ActIn& a, int M, int K, const void* w, int N, float* c, int ldc,
                          SplitWs ws, hipStream_t st);
size_t gemm_split_ws_floats(int M, int max_n);

// bfloat16 LM head with the row statistics fused into the GEMM epilogue
// (per half tile) and merged by a second kernel; logits stored only if
// `logits` is not null.  N must be a multiple of 128.
size_t lm_stats_ws_bytes(int M, int N);
hipError_t lm_head_stats(const ActIn& a, int M, int K, const void* w, int N, int mask_id, int k,
                         void* stats_ws, float* logits, int32_t* argmax, float* conf,
                         int32_t* topk_ids, float* topk_w, hipStream_t st);

// ---- attention -----------------------------------------------------------
struct AttnWs {
  float* opart;      // [S, B*H, Mq, dh]
  float* ml;         // [S, B*H, Mq, 2]
  int max_splits;
};
// Operand types of attention(): float32 (the float32 model), bfloat16, or
// float16 (the bfloat16 model's q, k, v).  The output is the float32 rows or
// the bfloat16 operand of the output projection, as `out` says.
enum { ATTN_F32 = 0, ATTN_BF16 = 1, ATTN_F16 = 2 };
// Number of key-range splits attention() uses for these sizes (at most
// max_splits); with more than one, ws receives S * B * H * Mq float32 rows of
// dh partial outputs and S * B * H * Mq (max, sum) pairs, each written before
// the merge reads it.  keys_per_split (may be null) receives the split width.
int attention_splits(int dtype, int B, int H, int Mq, int Nk, int max_splits, int* keys_per_split);
// out: [B * Mq, H * dh] activation operand of the output projection
// Sequence s reads keys [pads.of(s), Nk): its first pads.of(s) slots are padding.
hipError_t attention(int dtype, const void* q, const void* kc, const void* vc, int B, int H,
                     int Hkv, int dh, int Mq, int Nk, int cap, const ActOut& out, AttnWs ws,
                     const Pads& pads, hipStream_t st);

// ---- unmasking ------------------------------------------------------------
hipError_t launch_unmask(int32_t* tokens, int batch, int seq_len, int block_start, int b,
                         int mask_id, int rule, int n_per_step, float threshold,
                         const int32_t* argmax, const float* conf, const int32_t* topk_ids,
                         const float* topk_w, int k, int n_out, const int32_t* pos_out, int step,
                         int32_t* pred_ids, float* pred_w, int32_t* pred_step, uint8_t* selected,
                         int32_t* masked_left, const Pads& pads, hipStream_t st);
hipError_t launch_early_stop(int32_t* tokens, int batch, int seq_len, int block_start, int b,
                             int eos_id, int32_t* done, const Pads& pads, hipStream_t st);

}  // namespace ssm
