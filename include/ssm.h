/*
 * ssm.h -- C ABI of the SSM block-wise denoising step on AMD Instinct MI355X (gfx950).
 *
 * Structured Suffix Modeling (SSM) decodes a masked diffusion language model
 * block by block.  At each denoising step the model input is the prefix (the
 * prompt and every block decoded so far), the current block, and only the
 * suffix tokens retained by the local / middle / tail rules (Section 3.2,
 * Eq. 1-5), each at its original RoPE position ("Sparse Input Construction").
 * Retained suffix tokens are embedded as a mix of the [MASK] embedding and a
 * soft embedding of the previous step's top-k prediction (Eq. 6-8).  The step
 * ends by unmasking the most confident positions of the block (Section 4.2).
 *
 * One step is four calls, in this order:
 *   ssm_select_suffix  -> compacted row list (positions, regions, token ids)
 *   ssm_embed_suffix   -> input embeddings of the compacted rows
 *   ssm_denoise_step   -> transformer forward, LM head, per-row statistics
 *   ssm_unmask         -> decode block positions, record suffix predictions
 *
 * Conventions shared by every call
 *   - "d_" pointers are HIP device memory owned by the caller.  The library
 *     never allocates or frees device memory and keeps no pointer after a
 *     call returns.  Host pointers (structs, output counts) are read or
 *     written synchronously during the call.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Work is enqueued
 *     on it asynchronously and is ordered with the caller's other work on
 *     that stream.
 *   - Arguments are validated on the host before anything is launched; an
 *     invalid call launches nothing and returns a negative SSM_E_* code with
 *     a message available from ssm_last_error() (thread-local).
 *   - No C++ exception crosses the ABI.  Results are deterministic: no
 *     floating-point reduction depends on scheduling order.
 *   - Batched sequences share generation length, block size, budgets and
 *     block schedule.  Their prompts may differ in length: the calls then take
 *     `pad`, a HOST array [batch] (at most 64 sequences) in which pad[s] is
 *     how many tokens shorter sequence s's prompt is than the longest one
 *     (pad = NULL: all prompts equally long).  The batch shares the row
 *     layout of its longest prompt, and sequence s sits pad[s] positions to
 *     the left in it: row r is position pos[r] - pad[s] of sequence s, and
 *     prefix rows whose position falls below zero are padding (embedded as
 *     [MASK], computed, never read as keys).  This is exact rather than an
 *     approximation: with a shared generation length each sequence's suffix
 *     regions (Eq. 1) and retained set R_t are those of the longest prompt
 *     shifted by pad[s], so pos[r] - pad[s] is sequence s's own position
 *     list.  Token and prediction-state arrays keep a stride of the longest
 *     sequence; sequence s uses its first seq_len - pad[s] positions.
 *   - Element types: token ids and positions int32; region tags int8;
 *     probabilities and the residual stream float32; weights and embeddings
 *     in the model's dtype (float32 or bfloat16); the KV cache in float32
 *     for a float32 model and in float16 for a bfloat16 model.
 */
#ifndef SSM_H
#define SSM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
enum {
  SSM_OK = 0,
  SSM_E_INVAL = -1,        /* bad argument value or null required pointer     */
  SSM_E_SHAPE = -2,        /* inconsistent model shape                         */
  SSM_E_CAPACITY = -3,     /* an output or cache buffer is too small           */
  SSM_E_HIP = -4,          /* a HIP runtime or launch error                    */
  SSM_E_UNSUPPORTED = -5   /* valid, but a shape this build has no kernel for  */
};

/* Middle-region retention (Section 3.2, Eq. 3; the middle-region variants of
 * the ablation in Table 2).  The block modes ignore middle_budget. */
enum {
  SSM_MIDDLE_STRIDED = 0,         /* middle_budget tokens at offsets floor(i*len/M')     */
  SSM_MIDDLE_BLOCK_START = 1,     /* the start token of every middle block (Eq. 3)     */
  SSM_MIDDLE_BLOCK_END = 2,       /* the end token of every middle block                */
  SSM_MIDDLE_BLOCK_START_END = 3  /* both (one token if block_size == 1)                */
};

/* Tail-region retention (Section 3.2, Eq. 4; the tail variants of Table 2). */
enum {
  SSM_TAIL_SPREAD = 0,   /* T' = min(tail_budget, len) tokens at offsets floor(i*(len-1)/(T'-1)), */
                         /* both ends first (Eq. 4 is T = 2); T' = 1 keeps the end token         */
  SSM_TAIL_START = 1     /* the start token only (if tail_budget >= 1)                          */
};

/* Unmasking rules (Section 4.2 "Vanilla" / "Par."; Section 4.6 margin rule, Table 3). */
enum {
  SSM_UNMASK_TOPN = 0,         /* the n most confident masked positions             */
  SSM_UNMASK_THRESHOLD = 1,    /* confidence > threshold, at least one per step     */
  SSM_UNMASK_MARGIN = 2        /* top1 - top2 probability > threshold, at least one */
};

/* Element types.  SSM_DT_F32 and SSM_DT_BF16 are model types; SSM_DT_F16 is
 * the type of the attention operands (queries, KV cache) of a bfloat16 model. */
enum { SSM_DT_F32 = 0, SSM_DT_BF16 = 1, SSM_DT_F16 = 2 };

/* Activation precision at the projections of a bfloat16 model. */
enum {
  SSM_ACT_BF16 = 0,     /* each projection input is rounded once to bfloat16                 */
  SSM_ACT_BF16X2 = 1,   /* each projection input is kept as a bfloat16 pair hi + lo and both  */
                        /* parts are multiplied (weights stay bfloat16; twice the MFMA work)  */
  SSM_ACT_BF16X2_FIRST = 2  /* the pair in layers [0, pair_layers) only; the later layers and   */
                            /* the LM head round once.  The residual stream grows with depth,   */
                            /* so a rounding in an early layer weighs far more in the output    */
                            /* than one in a late layer.                                        */
};

/* Region tag of a compacted row. */
enum {
  SSM_REGION_PREFIX = 0, SSM_REGION_BLOCK = 1, SSM_REGION_LOCAL = 2,
  SSM_REGION_MIDDLE = 3, SSM_REGION_TAIL = 4
};

/* Prefix KV cache use in ssm_denoise_step (the "PC." setting, Section 4.8, Table 4). */
enum {
  SSM_CACHE_OFF = 0,    /* every row is an input row; the cache buffers are scratch        */
  SSM_CACHE_WRITE = 1,  /* first step of a block: rows start with the prefix; afterwards   */
                        /* slots [0, prefix) of every layer hold the prefix keys/values     */
  SSM_CACHE_READ = 2    /* later step: keys/values of slots [0, n_cached) are the prefix   */
};

/* ------------------------------------------------------------------------ */
/* Suffix partition and compaction (Section 3.2, Eq. 1-5; sparse input).    */
/* ------------------------------------------------------------------------ */

typedef struct ssm_select_params {
  int32_t prompt_len;      /* P0 >= 0                                                      */
  int32_t gen_len;         /* G > 0, a multiple of block_size                              */
  int32_t block_size;      /* b in [1, 1024]                                               */
  int32_t block_idx;       /* current block j in [0, G/b)                                  */
  int32_t local_budget;    /* tokens kept whole after the block (Eq. 2 with w*b)  >= 0     */
  int32_t middle_budget;   /* strided mode: tokens kept in the middle region      >= 0     */
  int32_t middle_mode;     /* SSM_MIDDLE_*                                                 */
  int32_t tail_budget;     /* tokens kept in the last block, both ends first (Eq. 4) >= 0  */
  int32_t include_prefix;  /* 1: rows start with the prefix [0, P0 + j*b); 0: cached step  */
  int32_t tail_mode;       /* SSM_TAIL_*                                                   */
} ssm_select_params;

/*
 * Row counts of the compacted sequence, in closed form on the host; no GPU
 * work.  n_rows = (include_prefix ? P0 + j*b : 0) + b + n_suffix;
 * first_out_row = the index of the first row of the current block (rows
 * from there on need logits).  Any output pointer may be NULL.
 */
int32_t ssm_select_count(const ssm_select_params* p, int32_t* n_rows, int32_t* n_suffix,
                         int32_t* first_out_row);

/*
 * The position and region lists of ssm_select_suffix computed on the host, by
 * the same closed form the kernel evaluates per row; no GPU work.
 *   pos [cap] int32 and region [cap] int8 (may be NULL) are HOST arrays.
 * SSM_E_CAPACITY if cap < n_rows; n_rows may be NULL.
 */
int32_t ssm_select_positions_host(const ssm_select_params* p, int32_t* pos, int8_t* region,
                                  int32_t cap, int32_t* n_rows);

/*
 * Builds the compacted row list of the sparse input [P; B_t; R_t]: for row r,
 * d_pos[r] is its absolute position (ascending within prefix, block and R_t),
 * d_region[r] its SSM_REGION_* tag, and d_tok_c[s*cap + r] the token id of
 * sequence s at that position (gathered from d_tokens[s*seq_len + pos -
 * pad[s]]; -1 for padding rows).
 *   d_tokens  [batch, seq_len] int32, seq_len == prompt_len + gen_len
 *             (prompt_len: the longest prompt when pad is given)
 *   pad       HOST [batch] or NULL, each in [0, prompt_len]
 *   d_pos     [cap] int32, d_region [cap] int8 (may be NULL), d_tok_c [batch, cap] int32
 * The row counts are returned synchronously (as ssm_select_count).
 * SSM_E_CAPACITY if cap < n_rows.
 */
int32_t ssm_select_suffix(const ssm_select_params* p, int32_t batch, int32_t seq_len,
                          const int32_t* pad, const int32_t* d_tokens, int32_t* d_pos,
                          int32_t* d_tok_c, int8_t* d_region, int32_t cap, int32_t* n_rows,
                          int32_t* n_suffix, int32_t* first_out_row, void* stream);

/* ------------------------------------------------------------------------ */
/* Model description.                                                       */
/* ------------------------------------------------------------------------ */

/* Device pointers of one decoder layer, row-major, in the model's dtype. */
typedef struct ssm_layer {
  const void* attn_norm;   /* [d]                                  */
  const void* wq;          /* [n_heads*head_dim, d]                */
  const void* wk;          /* [n_kv_heads*head_dim, d]             */
  const void* wv;          /* [n_kv_heads*head_dim, d]             */
  const void* wo;          /* [d, n_heads*head_dim]                */
  const void* ffn_norm;    /* [d]                                  */
  const void* w_gate;      /* [ffn_dim, d]                         */
  const void* w_up;        /* [ffn_dim, d]                         */
  const void* w_down;      /* [d, ffn_dim]                         */
} ssm_layer;

/*
 * Bidirectional pre-norm decoder (LLaDA / Dream shape): RMSNorm, attention
 * with rotate-half RoPE and grouped-query heads, SwiGLU FFN, final RMSNorm,
 * untied LM head.  d_model == n_heads*head_dim; n_heads % n_kv_heads == 0.
 */
typedef struct ssm_model {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab, mask_id;
  int32_t dtype;           /* SSM_DT_F32 or SSM_DT_BF16                        */
  float rope_base;         /* e.g. 10000                                       */
  float rms_eps;           /* e.g. 1e-5                                        */
  const void* tok_emb;     /* [vocab, d] device                                */
  const void* final_norm;  /* [d] device                                       */
  const void* lm_head;     /* [vocab, d] device                                */
  const ssm_layer* layers; /* HOST array of n_layers device-pointer sets       */
  int32_t act_mode;        /* SSM_ACT_*; ignored for float32 models            */
  int32_t pair_layers;     /* SSM_ACT_BF16X2_FIRST: leading layers that keep   */
                           /* the pair, in [0, n_layers]; ignored otherwise    */
} ssm_model;

/* Prefix KV cache: k and v are [n_layers, batch, n_kv_heads, capacity, head_dim],
 * float32 for a float32 model and float16 for a bfloat16 model; keys are
 * stored after RoPE.  A bfloat16 model keeps its attention operands (queries,
 * keys, values and the softmax probabilities) in float16: the same MFMA rate
 * and bytes as bfloat16 with three more significand bits.  Rounding them to
 * bfloat16 instead costs about 0.4% relative error per layer over long
 * contexts of distinct tokens (2.4% over 28 layers of 1024 rows); float16
 * brings that rounding down by a factor of about eight.  Values must stay
 * within the float16 range (|x| < 65504). */
typedef struct ssm_kv_cache {
  void* k;
  void* v;
  int32_t capacity;
} ssm_kv_cache;

/* ------------------------------------------------------------------------ */
/* Soft suffix embedding (Section 3.2, Eq. 6-8).                            */
/* ------------------------------------------------------------------------ */

/*
 * d_x[s, r, :] (float32 [batch, n_rows, d]) = the input embedding of row r:
 *   - E[tok] for prefix and block rows (d_region < SSM_REGION_LOCAL);
 *   - for a retained suffix row at position p whose prediction was made at
 *     step prev_step (d_pred_step[s, p] == prev_step >= 0):
 *       (1 - alpha) E[mask] + alpha * sum_i d_pred_w[s, p, i] E[d_pred_ids[s, p, i]]
 *     (Eq. 7-8; the weights are the Eq. 6 renormalised top-k probabilities);
 *   - E[mask] for a retained suffix row without such a prediction.
 *   d_tok_c [batch, tok_stride] int32 (tok_stride >= n_rows: the `cap` of
 *   ssm_select_suffix); d_pos, d_region [n_rows];
 *   d_pred_ids [batch, seq_len, k] int32, d_pred_w [batch, seq_len, k] float32,
 *   d_pred_step [batch, seq_len] int32 (indexed by each sequence's own
 *   position pos[r] - pad[s]; pad HOST [batch] or NULL, each in [0, seq_len]).
 * Padding rows (position below zero) are E[mask].
 * k in [1, 8]; alpha in [0, 1].
 */
int32_t ssm_embed_suffix(const ssm_model* m, int32_t batch, int32_t seq_len, const int32_t* pad,
                         const int32_t* d_tok_c, int32_t tok_stride, const int32_t* d_pos,
                         const int8_t* d_region, int32_t n_rows, const int32_t* d_pred_ids,
                         const float* d_pred_w, const int32_t* d_pred_step, int32_t prev_step,
                         int32_t k, float alpha, float* d_x, void* stream);

/* ------------------------------------------------------------------------ */
/* Transformer forward over the compacted rows, LM head and row statistics. */
/* ------------------------------------------------------------------------ */

/* Bytes of device workspace ssm_denoise_step needs for up to max_rows rows per
 * sequence (256-byte aligned pieces). */
int32_t ssm_workspace_size(const ssm_model* m, int32_t batch, int32_t max_rows, size_t* bytes);

/*
 * Runs every layer over the n_rows compacted rows of each sequence
 * (d_x float32 [batch, n_rows, d], rows at positions d_pos[n_rows]), then the
 * final norm and LM head over the output rows [first_out_row, n_rows)
 * (n_out = n_rows - first_out_row) and writes, per output row (float32 /
 * int32, [batch, n_out(, k)]), with the [MASK] id excluded from the vocabulary:
 *   d_argmax   most probable token (lower id on ties)
 *   d_conf     its softmax probability
 *   d_topk_ids the k most probable tokens, most probable first
 *   d_topk_w   their probabilities renormalised over the k (Eq. 6)
 * Optional debug outputs (NULL to skip): d_logits_dbg float32 [batch, n_out, vocab],
 * d_hidden_dbg float32 [batch, n_rows, d] (residual stream after the last layer).
 * Cache: cache_mode SSM_CACHE_OFF / WRITE require n_cached == 0; READ requires
 * n_cached > 0 prefix slots written by an earlier WRITE step.  This step's keys
 * and values go to slots [n_cached, n_cached + n_rows), so capacity >=
 * n_cached + n_rows.  Attention of every row reads all n_cached + n_rows keys.
 * d_ws: workspace of ws_bytes >= ssm_workspace_size(batch, n_rows).
 * pad (HOST [batch] or NULL): sequence s rotates row r at position pos[r] -
 * pad[s] and its keys start at slot pad[s] (its padding rows and slots are
 * never attended to); each pad[s] is at most the prefix it pads: n_cached
 * for SSM_CACHE_READ, first_out_row otherwise (SSM_E_INVAL).
 * k in [1, 8].  The bfloat16 path needs d_model and ffn_dim to be multiples of
 * 256, vocab a multiple of 128 and head_dim == 128; otherwise SSM_E_UNSUPPORTED.
 */
int32_t ssm_denoise_step(const ssm_model* m, const ssm_kv_cache* cache, int32_t cache_mode,
                         int32_t n_cached, int32_t batch, const int32_t* pad, const int32_t* d_pos,
                         int32_t n_rows, const float* d_x, int32_t first_out_row, int32_t k,
                         int32_t* d_argmax, float* d_conf, int32_t* d_topk_ids, float* d_topk_w,
                         float* d_logits_dbg, float* d_hidden_dbg, void* d_ws, size_t ws_bytes,
                         void* stream);

/* ------------------------------------------------------------------------ */
/* Building blocks of the step, callable alone (measurement and testing).   */
/* ------------------------------------------------------------------------ */

/* Bytes of device workspace ssm_attention needs (split-KV partial results). */
int32_t ssm_attention_workspace_size(int32_t batch, int32_t n_heads, int32_t n_q, size_t* bytes);

/*
 * The non-causal attention of ssm_denoise_step on its own (Section 3.2: every
 * compacted row attends to every key): for sequence s, head h, row i,
 *   out[s, i, 128 h + :] = sum_j softmax_j(q[s,h,i,:] . k[s,h/g,j,:] / sqrt(128)) v[s,h/g,j,:]
 * over keys j < n_keys, g = n_heads / n_kv_heads (grouped-query heads).
 * Inputs of type dtype (SSM_DT_BF16, or SSM_DT_F16 as in the step of a
 * bfloat16 model): d_q [batch, n_heads, n_q, 128]; d_k, d_v [batch,
 * n_kv_heads, capacity, 128] (the KV cache layout, keys already rotated).
 * Output float32 d_out [batch, n_q, n_heads * 128], row-major.  Scores and
 * softmax in float32; the probabilities are rounded to the input type for the
 * P V product (to nearest even for bfloat16, toward zero for float16).
 * SSM_E_INVAL for another dtype; n_keys <= capacity (SSM_E_CAPACITY), n_heads
 * a multiple of n_kv_heads (SSM_E_SHAPE), ws_bytes >=
 * ssm_attention_workspace_size(batch, n_heads, n_q) (SSM_E_CAPACITY).
 */
int32_t ssm_attention(int32_t dtype, int32_t batch, int32_t n_heads, int32_t n_kv_heads,
                      int32_t n_q, int32_t n_keys, int32_t capacity, const void* d_q,
                      const void* d_k, const void* d_v, float* d_out, void* d_ws,
                      size_t ws_bytes, void* stream);

/* Size of the device scratch array behind ssm_attention_static (16 MiB per
 * GPU): 520 bytes per split-KV partial row (128 float32 outputs, max and sum),
 * room for 32263 rows.  The split choice keeps S * batch * n_heads * n_q at
 * or below 32768, so only launches near that edge are refused. */
#define SSM_ATTENTION_STATIC_SCRATCH_BYTES (16 << 20)

/*
 * ssm_attention for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops that forbid allocation): the same
 * arguments without the workspace, the same kernels and split choice, and
 * bit-identical results.  The split-KV partial results go to a file-scope
 * device array of SSM_ATTENTION_STATIC_SCRATCH_BYTES that each GPU the
 * library runs on holds until the process ends; its address is looked up
 * once per device on the first call there.  The call allocates and frees
 * nothing.  SSM_E_CAPACITY if the partials of this launch would exceed the
 * array (only launches that split a long key range over many rows use it;
 * ssm_attention has no such limit); otherwise as ssm_attention.  Calls that
 * overlap on one GPU (other streams or threads) share the array and race:
 * order them on one stream.
 */
int32_t ssm_attention_static(int32_t dtype, int32_t batch, int32_t n_heads, int32_t n_kv_heads,
                             int32_t n_q, int32_t n_keys, int32_t capacity, const void* d_q,
                             const void* d_k, const void* d_v, float* d_out, void* stream);

/*
 * The row gather of the compaction (Section 3.2, sparse input construction)
 * applied to activations: for each sequence s and i < n_rows,
 *   d_dst[s, i, :] = d_src[s, d_pos[i], :]
 * for bfloat16 rows of `width` elements (a multiple of 8); d_src [batch,
 * src_rows, width], d_pos int32 [n_rows], d_dst [batch, n_rows, width].
 * A position outside [0, src_rows) yields a row of zeros.
 */
int32_t ssm_gather_rows(int32_t batch, int32_t src_rows, int32_t width, const void* d_src,
                        const int32_t* d_pos, int32_t n_rows, void* d_dst, void* stream);

/* ------------------------------------------------------------------------ */
/* Confidence-based unmasking and prediction-state update (Section 4.2).    */
/* ------------------------------------------------------------------------ */

/*
 * For each sequence s, among the still-masked positions of the block
 * [block_start, block_start + block_size) of d_tokens [batch, seq_len]:
 *   TOPN:      the n_per_step highest d_conf (lower position on ties);
 *   THRESHOLD: every d_conf > threshold, or the single highest if none;
 *   MARGIN:    every (p1 - p2) > threshold, or the single widest if none,
 *              where p2 = d_conf * d_topk_w[.,1] / d_topk_w[.,0] (needs k >= 2);
 * and writes d_argmax there.  Output rows (d_argmax, d_conf [batch, n_out],
 * d_topk_ids, d_topk_w [batch, n_out, k]) are those of ssm_denoise_step: row i
 * < block_size is block position block_start + i; row i >= block_size is the
 * retained suffix position d_pos_out[i].  For those suffix rows the top-k
 * prediction is stored: d_pred_ids/d_pred_w[s, pos, :] and
 * d_pred_step[s, pos] = step.
 * d_selected (uint8 [batch, block_size], may be NULL) receives the decoded
 * positions, d_masked_left (int32 [batch], may be NULL) the masks left in the block.
 * pad (HOST [batch] or NULL, each in [0, block_start]): sequence s's block
 * starts at block_start - pad[s] and its suffix rows are at d_pos_out[i] - pad[s].
 */
int32_t ssm_unmask(int32_t* d_tokens, int32_t batch, int32_t seq_len, const int32_t* pad,
                   int32_t block_start, int32_t block_size, int32_t mask_id, int32_t rule,
                   int32_t n_per_step, float threshold, const int32_t* d_argmax, const float* d_conf,
                   const int32_t* d_topk_ids, const float* d_topk_w, int32_t k, int32_t n_out,
                   const int32_t* d_pos_out, int32_t step, int32_t* d_pred_ids, float* d_pred_w,
                   int32_t* d_pred_step, uint8_t* d_selected, int32_t* d_masked_left,
                   void* stream);

/* ------------------------------------------------------------------------ */
/* Early termination (Section 3.2, "Early Termination"; the fill rule of    */
/* Section 4.4).                                                             */
/* ------------------------------------------------------------------------ */

/*
 * Called after the last step of a block.  Every sequence s with d_done[s] == 0
 * whose block [block_start, block_start + block_size) holds eos_id gets all
 * later positions [block_start + block_size, seq_len) set to eos_id and
 * d_done[s] = 1; sequences already done are left as they are.
 *   d_tokens [batch, seq_len] int32 (in place), d_done [batch] int32, zeroed by
 *   the caller at the start of a generation.
 * The generation can stop once every d_done[s] is 1 (the caller copies
 * d_done to the host to find out).  With pad (HOST [batch] or NULL, each in
 * [0, block_start]) sequence s's block starts pad[s] to the left and its
 * sequence ends at seq_len - pad[s].  SSM_E_INVAL for a block outside the
 * sequence, eos_id < 0, a pad out of range or a null pointer.
 */
int32_t ssm_early_stop(int32_t* d_tokens, int32_t batch, int32_t seq_len, const int32_t* pad,
                       int32_t block_start, int32_t block_size, int32_t eos_id, int32_t* d_done,
                       void* stream);

/* ------------------------------------------------------------------------ */
/* Launch timing (tracing aid; off by default).                             */
/* ------------------------------------------------------------------------ */

/*
 * on != 0: from now on every kernel launched by the calls above is
 * bracketed by a pair of HIP events on the call's stream (created without
 * the system-scope fence), recorded under a tag naming the operation ("select", "embed",
 * "rope_table", "norm", "gemm_qkv", "attention", "gemm_o", "gemm_gate_up",
 * "gemm_down", "gemm_lm_head", "rowstats", "unmask", "early_stop") and the kernel's
 * ordinal within one call of that operation (0 = the main kernel; split-K
 * reductions and merges come after).  Each call discards earlier records.
 * Not thread-safe; meant for a single profiling thread.
 */
int32_t ssm_profile_enable(int32_t on);

/* Number of recorded kernels under `tag` (all ordinals if kernel < 0, else
 * only that ordinal) and their summed duration in milliseconds; waits for
 * the recorded events to complete. */
int32_t ssm_profile_query(const char* tag, int32_t kernel, int32_t* count, double* total_ms);

/* Message of the last error on this thread ("" if none). */
const char* ssm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SSM_H */
