// Internal launcher interfaces of the SSM HIP library.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.h"

namespace ssm {

// Closed-form layout of the compacted rows of one step (Section 3.2, Eq. 1-5).
struct SelectLayout {
  int n_prefix;      // prefix rows included (0 on a cached step)
  int P;             // first position of the current block
  int b;             // block size
  int s0;            // first suffix position
  int n_local;       // local tokens [s0, s0 + n_local)
  int mid_lo, mid_len, n_mid, mid_mode, mid_first;
  int tail_lo, tail_len, n_tail;
  int n_suffix, n_rows;
};

hipError_t launch_select(const SelectLayout& L, int batch, int seq_len, const int32_t* tokens,
                         int32_t* pos, int32_t* tok_c, int8_t* region, int cap, hipStream_t st);

hipError_t launch_embed(int dtype, const void* E, int d, int vocab, int mask_id, int batch,
                        int seq_len, const int32_t* tok_c, int tok_stride, const int32_t* pos,
                        const int8_t* region, int n_rows, const int32_t* pred_ids,
                        const float* pred_w, const int32_t* pred_step, int prev_step, int k,
                        float alpha, float* x, hipStream_t st);

// cos/sin of pos[r] * base^(-2i/dh) computed in float64, stored as float2.
hipError_t launch_rope_table(const int32_t* pos, int n_rows, int dh, float base, float2* tab,
                             hipStream_t st);

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
};

// Workspace for split-K partial sums, float32.
struct SplitWs {
  float* part;
  size_t floats;
};

// float32 activation operand of a projection, with the fused RMSNorm scales:
// A[m, k] = a[row(m) * lda + k] * rscale[m] * cscale[k] (a null scale is 1),
// row(m) = (m / per) * stride + off + m % per.
struct GemmA {
  const float* a;
  int lda;
  const float* rscale;
  const void* cscale;     // model dtype
  int per, stride, off;
};

inline GemmA plain_a(const float* a, int lda, int M) { return GemmA{a, lda, nullptr, nullptr, M, 0, 0}; }

hipError_t launch_row_rms(const float* x, int d, float eps, float* inv, int n_rows, int per,
                          int stride, int off, hipStream_t st);
hipError_t gemm_qkv(int dtype, bool split, const GemmA& a, int M, int d, const void* wq,
                    const void* wk, const void* wv, int H, int Hkv, int dh, const QKVOut& out,
                    SplitWs ws, hipStream_t st);
hipError_t gemm_resid(int dtype, bool split, const char* kind, const GemmA& a, int M, int K,
                      const void* w, int N, float* resid, SplitWs ws, hipStream_t st);
hipError_t gemm_swiglu(int dtype, bool split, const GemmA& a, int M, int d, const void* wg,
                       const void* wu, int F, float* act, SplitWs ws, hipStream_t st);
hipError_t gemm_store(int dtype, bool split, const GemmA& a, int M, int K, const void* w, int N,
                      float* c, int ldc, SplitWs ws, hipStream_t st);
size_t gemm_split_ws_floats(int M, int max_n);

// bfloat16 LM head with the row statistics fused into the GEMM epilogue
// (per half tile) and merged by a second kernel; logits stored only if
// `logits` is not null.  N must be a multiple of 128.
size_t lm_stats_ws_bytes(int M, int N);
hipError_t lm_head_stats(bool split, const GemmA& a, int M, int K, const void* w, int N,
                         int mask_id, int k, void* stats_ws, float* logits, int32_t* argmax,
                         float* conf, int32_t* topk_ids, float* topk_w, hipStream_t st);

// ---- attention -----------------------------------------------------------
struct AttnWs {
  float* opart;      // [S, B*H, Mq, dh]
  float* ml;         // [S, B*H, Mq, 2]
  int max_splits;
};
// out: float32 [B * Mq, H * dh]
hipError_t attention(int dtype, const void* q, const void* kc, const void* vc, int B, int H,
                     int Hkv, int dh, int Mq, int Nk, int cap, float* out, AttnWs ws,
                     hipStream_t st);

// ---- unmasking ------------------------------------------------------------
hipError_t launch_unmask(int32_t* tokens, int batch, int seq_len, int block_start, int b,
                         int mask_id, int rule, int n_per_step, float threshold,
                         const int32_t* argmax, const float* conf, const int32_t* topk_ids,
                         const float* topk_w, int k, int n_out, const int32_t* pos_out, int step,
                         int32_t* pred_ids, float* pred_w, int32_t* pred_step, uint8_t* selected,
                         int32_t* masked_left, hipStream_t st);

}  // namespace ssm
