// Confidence-based unmasking of the current block (Section 4.2: top-n
// "Vanilla" decoding and threshold "Par." decoding; Section 4.6 (Table 3): margin
// rule) and the update of the per-position prediction state that the next
// step's soft suffix embedding reads (Section 3.2, Eq. 6).
#include "internal.h"
#include "dcheck.h"

namespace ssm {

// One workgroup per sequence; the block (<= 1024 positions) lives in LDS.
__global__ void __launch_bounds__(256) unmask_kernel(
    int32_t* __restrict__ tokens, int seq_len, int block_start, int b, int mask_id, int rule,
    int n_per_step, float threshold, const int32_t* __restrict__ argmax,
    const float* __restrict__ conf, const int32_t* __restrict__ topk_ids,
    const float* __restrict__ topk_w, int k, int n_out, const int32_t* __restrict__ pos_out,
    int step, int32_t* __restrict__ pred_ids, float* __restrict__ pred_w,
    int32_t* __restrict__ pred_step, uint8_t* __restrict__ selected,
    int32_t* __restrict__ masked_left, Pads pads) {
  __shared__ float score[1024];
  __shared__ uint8_t cand[1024];
  __shared__ uint8_t sel[1024];
  __shared__ int n_cand, n_sel, best;
  const int s = blockIdx.x, tid = threadIdx.x;
  SSM_DCHECK(b <= 1024 && k >= 1 && k <= 8 && n_out >= b);
  // a padded sequence's block and suffix positions sit pad[s] to the left
  const int shift = pads.of(s);
  int32_t* tok = tokens + (size_t)s * seq_len + (block_start - shift);
  const size_t ro = (size_t)s * n_out;
  if (tid == 0) { n_cand = 0; n_sel = 0; best = -1; }
  for (int i = tid; i < b; i += blockDim.x) {
    cand[i] = tok[i] == mask_id;
    float sc = conf[ro + i];
    if (rule == 2) {  // p1 - p2, with p2/p1 = w[1]/w[0] of the top-k renormalisation
      const float w0 = topk_w[(ro + i) * k], w1 = topk_w[(ro + i) * k + 1];
      sc = sc * (1.0f - w1 / w0);
    }
    score[i] = sc;
  }
  __syncthreads();
  int my_c = 0, my_s = 0;
  for (int i = tid; i < b; i += blockDim.x) {
    uint8_t chosen = 0;
    if (cand[i]) {
      ++my_c;
      int rank = 0;  // candidates ranked ahead: higher score, then lower position
      for (int j = 0; j < b; ++j)
        rank += cand[j] && (score[j] > score[i] || (score[j] == score[i] && j < i));
      if (rank == 0) best = i;
      chosen = rule == 0 ? (rank < n_per_step) : (score[i] > threshold);
    }
    sel[i] = chosen;
    my_s += chosen;
  }
  atomicAdd(&n_cand, my_c);   // integer counts: order-independent
  atomicAdd(&n_sel, my_s);
  __syncthreads();
  if (rule != 0 && n_sel == 0 && best >= 0) {
    if (tid == 0) sel[best] = 1;
    __syncthreads();
  }
  for (int i = tid; i < b; i += blockDim.x) {
    if (sel[i]) tok[i] = argmax[ro + i];
    if (selected) selected[(size_t)s * b + i] = sel[i];
  }
  if (masked_left && tid == 0) {
    const int chosen = (rule != 0 && n_sel == 0 && best >= 0) ? 1 : n_sel;
    masked_left[s] = n_cand - chosen;
  }
  // prediction state of the retained suffix rows
  for (int r = b + tid; r < n_out; r += blockDim.x) {
    const int p = pos_out[r] - shift;
    SSM_DCHECK(p >= 0 && p < seq_len);
    if (p < 0 || p >= seq_len) continue;
    const size_t sp = (size_t)s * seq_len + p;
    for (int i = 0; i < k; ++i) {
      pred_ids[sp * k + i] = topk_ids[(ro + r) * k + i];
      pred_w[sp * k + i] = topk_w[(ro + r) * k + i];
    }
    pred_step[sp] = step;
  }
}

hipError_t launch_unmask(int32_t* tokens, int batch, int seq_len, int block_start, int b,
                         int mask_id, int rule, int n_per_step, float threshold,
                         const int32_t* argmax, const float* conf, const int32_t* topk_ids,
                         const float* topk_w, int k, int n_out, const int32_t* pos_out, int step,
                         int32_t* pred_ids, float* pred_w, int32_t* pred_step, uint8_t* selected,
                         int32_t* masked_left, const Pads& pads, hipStream_t st) {
  launch(unmask_kernel, dim3(batch), dim3(256), 0, st, tokens, seq_len, block_start, b,
                     mask_id, rule, n_per_step, threshold, argmax, conf, topk_ids, topk_w, k,
                     n_out, pos_out, step, pred_ids, pred_w, pred_step, selected, masked_left,
                     pads);
  return hipGetLastError();
}

// Early termination after a block (Section 3.2, "Early Termination"; the fill
// rule of Section 4.4).  One workgroup per sequence: a sequence not yet done
// whose block holds eos_id gets every later position set to eos_id and is
// marked done.  A padded sequence's block starts pad[s] to the left and its
// sequence ends pad[s] before seq_len.
__global__ void __launch_bounds__(256) early_stop_kernel(int32_t* __restrict__ tokens, int seq_len,
                                                         int block_start, int b, int eos_id,
                                                         int32_t* __restrict__ done, Pads pads) {
  __shared__ int found;
  const int s = blockIdx.x, tid = threadIdx.x;
  if (done[s]) return;                        // uniform over the workgroup
  int32_t* tok = tokens + (size_t)s * seq_len;
  const int shift = pads.of(s);
  block_start -= shift;
  seq_len -= shift;
  if (tid == 0) found = 0;
  __syncthreads();
  int hit = 0;
  for (int i = block_start + tid; i < block_start + b; i += blockDim.x) hit |= tok[i] == eos_id;
  if (hit) found = 1;                         // benign race: every writer stores 1
  __syncthreads();
  if (!found) return;
  for (int i = block_start + b + tid; i < seq_len; i += blockDim.x) tok[i] = eos_id;
  if (tid == 0) done[s] = 1;
}

hipError_t launch_early_stop(int32_t* tokens, int batch, int seq_len, int block_start, int b,
                             int eos_id, int32_t* done, const Pads& pads, hipStream_t st) {
  launch(early_stop_kernel, dim3(batch), dim3(256), 0, st, tokens, seq_len, block_start, b, eos_id,
         done, pads);
  return hipGetLastError();
}

}  // namespace ssm
