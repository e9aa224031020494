// C ABI of the SSM library: argument validation, workspace layout and the
// orchestration of one denoising step.  See include/ssm.h for the contract.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "../../include/ssm.h"
#include "internal.h"

using namespace ssm;

namespace {

thread_local std::string g_err;

int32_t fail(int32_t code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int32_t ok() {
  g_err.clear();
  return SSM_OK;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) return fail(SSM_E_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

int32_t layout_of(const ssm_select_params* p, SelectLayout& L) {
  if (!p) return fail(SSM_E_INVAL, "null select params");
  const int P0 = p->prompt_len, G = p->gen_len, b = p->block_size, j = p->block_idx;
  if (P0 < 0) return fail(SSM_E_INVAL, "prompt_len %d < 0", P0);
  if (b < 1 || b > 1024) return fail(SSM_E_INVAL, "block_size %d not in [1, 1024]", b);
  if (G <= 0 || G % b != 0) return fail(SSM_E_INVAL, "gen_len %d not a positive multiple of block_size %d", G, b);
  if (j < 0 || j >= G / b) return fail(SSM_E_INVAL, "block_idx %d not in [0, %d)", j, G / b);
  if (p->local_budget < 0 || p->middle_budget < 0 || p->tail_budget < 0)
    return fail(SSM_E_INVAL, "negative budget");
  if (p->middle_mode < SSM_MIDDLE_STRIDED || p->middle_mode > SSM_MIDDLE_BLOCK_START_END)
    return fail(SSM_E_INVAL, "unknown middle_mode %d", p->middle_mode);
  if (p->tail_mode != SSM_TAIL_SPREAD && p->tail_mode != SSM_TAIL_START)
    return fail(SSM_E_INVAL, "unknown tail_mode %d", p->tail_mode);
  if (p->include_prefix != 0 && p->include_prefix != 1)
    return fail(SSM_E_INVAL, "include_prefix must be 0 or 1");
  if ((long long)P0 + G > 0x3fffffff) return fail(SSM_E_INVAL, "sequence too long");
  // Eq. 1: local = first min(L, n) suffix tokens, tail = last block minus the
  // local part, middle = what lies between.
  L.P = P0 + j * b;
  L.b = b;
  L.n_prefix = p->include_prefix ? L.P : 0;
  L.s0 = L.P + b;
  const int s_end = P0 + G, n = s_end - L.s0;
  L.n_local = p->local_budget < n ? p->local_budget : n;
  const int tail_lo = (L.s0 + L.n_local > s_end - b) ? L.s0 + L.n_local : s_end - b;
  L.mid_lo = L.s0 + L.n_local;
  L.mid_len = tail_lo - L.mid_lo;
  // with one-token blocks a block's start is its end
  L.mid_mode = (p->middle_mode == SSM_MIDDLE_BLOCK_START_END && b == 1) ? SSM_MIDDLE_BLOCK_START
                                                                       : p->middle_mode;
  L.mid_first = 0;
  L.mid_alt = 0;
  if (L.mid_len <= 0) {
    L.n_mid = 0;
  } else if (L.mid_mode == SSM_MIDDLE_STRIDED) {
    L.n_mid = p->middle_budget < L.mid_len ? p->middle_budget : L.mid_len;
  } else {
    // block grid from s0; the middle ends on a block boundary (the tail is the
    // last block) but may start inside a block cut by the local region
    const int off = L.mid_lo - L.s0, mid_hi = L.mid_lo + L.mid_len;
    const int first_start = L.s0 + ((off + b - 1) / b) * b;      // Eq. 3
    const int first_end = L.s0 + (off / b) * b + b - 1;
    const int n_start = first_start < mid_hi ? (mid_hi - first_start) / b : 0;
    const int n_end = first_end < mid_hi ? (mid_hi - first_end + b - 1) / b : 0;
    if (L.mid_mode == SSM_MIDDLE_BLOCK_START) {
      L.mid_first = first_start;
      L.n_mid = n_start;
    } else if (L.mid_mode == SSM_MIDDLE_BLOCK_END) {
      L.mid_first = first_end;
      L.n_mid = n_end;
    } else {   // start and end tokens, in position order
      L.mid_alt = first_end < first_start;
      L.mid_first = L.mid_alt ? first_end : first_start;
      L.n_mid = n_start + n_end;
    }
  }
  L.tail_lo = tail_lo;
  L.tail_len = s_end - tail_lo;
  L.tail_mode = p->tail_mode;
  L.n_tail = p->tail_budget < L.tail_len ? p->tail_budget : L.tail_len;   // Eq. 4
  if (L.tail_mode == SSM_TAIL_START && L.n_tail > 1) L.n_tail = 1;
  L.n_suffix = L.n_local + L.n_mid + L.n_tail;                           // Eq. 5
  L.n_rows = L.n_prefix + b + L.n_suffix;
  return SSM_OK;
}

int32_t check_model(const ssm_model* m) {
  if (!m) return fail(SSM_E_INVAL, "null model");
  if (m->dtype != SSM_DT_F32 && m->dtype != SSM_DT_BF16) return fail(SSM_E_INVAL, "unknown dtype %d", m->dtype);
  if (m->n_layers < 0 || m->d_model <= 0 || m->n_heads <= 0 || m->n_kv_heads <= 0 ||
      m->head_dim <= 0 || m->ffn_dim <= 0 || m->vocab <= 1)
    return fail(SSM_E_SHAPE, "non-positive model dimension");
  if (m->d_model != m->n_heads * m->head_dim)
    return fail(SSM_E_SHAPE, "d_model %d != n_heads %d * head_dim %d", m->d_model, m->n_heads, m->head_dim);
  if (m->n_heads % m->n_kv_heads != 0)
    return fail(SSM_E_SHAPE, "n_heads %d not a multiple of n_kv_heads %d", m->n_heads, m->n_kv_heads);
  if (m->mask_id < 0 || m->mask_id >= m->vocab) return fail(SSM_E_INVAL, "mask_id out of range");
  if (!m->tok_emb || !m->final_norm || !m->lm_head) return fail(SSM_E_INVAL, "null model tensor");
  if (m->n_layers > 0 && !m->layers) return fail(SSM_E_INVAL, "null layer array");
  for (int l = 0; l < m->n_layers; ++l) {
    const ssm_layer& y = m->layers[l];
    if (!y.attn_norm || !y.wq || !y.wk || !y.wv || !y.wo || !y.ffn_norm || !y.w_gate || !y.w_up || !y.w_down)
      return fail(SSM_E_INVAL, "null tensor in layer %d", l);
  }
  if (m->dtype == SSM_DT_BF16 && m->act_mode != SSM_ACT_BF16 && m->act_mode != SSM_ACT_BF16X2 &&
      m->act_mode != SSM_ACT_BF16X2_FIRST)
    return fail(SSM_E_INVAL, "unknown act_mode %d", m->act_mode);
  if (m->dtype == SSM_DT_BF16 && m->act_mode == SSM_ACT_BF16X2_FIRST &&
      (m->pair_layers < 0 || m->pair_layers > m->n_layers))
    return fail(SSM_E_INVAL, "pair_layers %d not in [0, %d]", m->pair_layers, m->n_layers);
  if (m->dtype == SSM_DT_BF16) {
    if (m->head_dim != 128) return fail(SSM_E_UNSUPPORTED, "bf16 path needs head_dim 128 (got %d)", m->head_dim);
    if (m->d_model % 256 || m->ffn_dim % 256 || m->vocab % 128)
      return fail(SSM_E_UNSUPPORTED, "bf16 path needs d_model and ffn_dim multiples of 256, vocab of 128");
  } else {
    if (m->head_dim != 32 && m->head_dim != 64 && m->head_dim != 128)
      return fail(SSM_E_UNSUPPORTED, "fp32 path needs head_dim 32, 64 or 128");
    if (m->d_model % 32 || m->ffn_dim % 32 || m->vocab % 32)
      return fail(SSM_E_UNSUPPORTED, "fp32 path needs d_model, ffn_dim, vocab multiples of 32");
  }
  return SSM_OK;
}

// Host array of per-sequence left padding (null: none) -> the kernels' Pads,
// each entry in [0, max_pad].
int32_t pads_of(const int32_t* pad, int batch, int max_pad, Pads& P) {
  memset(&P, 0, sizeof(P));
  if (!pad) return SSM_OK;
  if (batch > MAX_PAD_BATCH)
    return fail(SSM_E_UNSUPPORTED, "padded batches hold at most %d sequences (got %d)", MAX_PAD_BATCH, batch);
  for (int s = 0; s < batch; ++s) {
    if (pad[s] < 0 || pad[s] > max_pad)
      return fail(SSM_E_INVAL, "pad[%d] = %d not in [0, %d]", s, pad[s], max_pad);
    P.v[s] = pad[s];
    P.any |= pad[s] != 0;
  }
  return SSM_OK;
}

constexpr int ATTN_MAX_SPLITS = 16;

// Scratch memory of ssm_attention_static: the split-KV partial results,
// SSM_ATTENTION_STATIC_SCRATCH_BYTES in a file-scope device array, one copy
// per GPU, held until the process ends.  In host code `scratch` is only a
// stand-in for the symbol: its device address comes from
// hipGetSymbolAddress, once per device with that device current, and only
// that address is handed to kernels.
__device__ __align__(256) unsigned char scratch[SSM_ATTENTION_STATIC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

// ---- launch profiling: HIP events around each launcher, per tag ----------
struct ProfRec {
  const char* tag;
  int ordinal;            // kernel ordinal within one call of the operation
  hipEvent_t a, b;
};
bool g_prof_on = false;
std::vector<ProfRec> g_prof;
std::vector<hipEvent_t> g_event_pool;
const char* g_prof_tag = nullptr;   // operation being launched
int g_prof_ordinal = 0;

hipEvent_t pool_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

void prof_clear() {
  for (auto& r : g_prof) {
    g_event_pool.push_back(r.a);
    g_event_pool.push_back(r.b);
  }
  g_prof.clear();
}

struct ProfScope {
  ProfScope(const char* tag, hipStream_t) {
    g_prof_tag = tag;
    g_prof_ordinal = 0;
  }
  ~ProfScope() { g_prof_tag = nullptr; }
};

}  // namespace

bool ssm::prof_next(hipEvent_t* start, hipEvent_t* stop) {
  if (!g_prof_on || !g_prof_tag) return false;
  ProfRec r{g_prof_tag, g_prof_ordinal++, pool_event(), pool_event()};
  if (!r.a || !r.b) return false;
  g_prof.push_back(r);
  *start = r.a;
  *stop = r.b;
  return true;
}

namespace {

#define PROF_TRY(tag, expr)            \
  do {                                 \
    ProfScope ps_(tag, st);            \
    HIP_TRY(expr);                     \
  } while (0)

struct WsLayout {
  size_t resid, xn, xn_lo, q, attn, attn_lo, act, act_lo, rope, opart, ml, part, logits, lmstats, total;
  size_t part_floats;
};

// Whether the projection inputs of layer l (l == n_layers: the LM head) are
// kept as a bfloat16 pair.
static bool pair_in_layer(const ssm_model* m, int l) {
  if (m->dtype != SSM_DT_BF16) return false;
  if (m->act_mode == SSM_ACT_BF16X2) return true;
  return m->act_mode == SSM_ACT_BF16X2_FIRST && l < m->pair_layers;
}

WsLayout ws_layout(const ssm_model* m, int batch, int max_rows) {
  const size_t es = m->dtype == SSM_DT_BF16 ? 2 : 4;
  const size_t Mt = (size_t)batch * max_rows;
  const size_t d = m->d_model, H = m->n_heads, Hkv = m->n_kv_heads, dh = m->head_dim;
  const size_t F = m->ffn_dim, V = m->vocab;
  const size_t qkv = (H + 2 * Hkv) * dh;
  size_t maxn = qkv;
  if (2 * F > maxn) maxn = 2 * F;
  if (V > maxn) maxn = V;
  WsLayout w{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
  // projection operands: float32 for float32 models, bfloat16 hi (+ lo) otherwise
  // (bfloat16 operands in fragment order: rows padded to whole 16-row groups)
  const size_t lo_es = pair_in_layer(m, 0) ? 2 : 0;
  const size_t Mp = (size_t)row_groups((int)Mt) * 16;
  w.resid = take(Mt * d * 4);
  w.xn = take(Mp * d * es);
  w.xn_lo = take(Mp * d * lo_es);
  w.q = take(Mt * H * dh * es);
  w.attn = take(Mp * H * dh * es);
  w.attn_lo = take(Mp * H * dh * lo_es);
  w.act = take(Mp * F * es);
  w.act_lo = take(Mp * F * lo_es);
  w.rope = take((size_t)batch * max_rows * (dh / 2) * 8);   // one table per sequence when padded
  w.opart = take((size_t)ATTN_MAX_SPLITS * Mt * H * dh * 4);
  w.ml = take((size_t)ATTN_MAX_SPLITS * Mt * H * 2 * 4);
  w.part_floats = gemm_split_ws_floats((int)Mt, (int)maxn);
  w.part = take(w.part_floats * 4);
  w.logits = m->dtype == SSM_DT_BF16 ? take(0) : take(Mt * V * 4);
  w.lmstats = take(m->dtype == SSM_DT_BF16 ? lm_stats_ws_bytes((int)Mt, (int)V) : 0);
  w.total = off;
  return w;
}

}  // namespace

extern "C" {

const char* ssm_last_error(void) { return g_err.c_str(); }

int32_t ssm_select_count(const ssm_select_params* p, int32_t* n_rows, int32_t* n_suffix,
                         int32_t* first_out_row) {
  SelectLayout L;
  int32_t rc = layout_of(p, L);
  if (rc) return rc;
  if (n_rows) *n_rows = L.n_rows;
  if (n_suffix) *n_suffix = L.n_suffix;
  if (first_out_row) *first_out_row = L.n_prefix;
  return ok();
}

int32_t ssm_select_positions_host(const ssm_select_params* p, int32_t* pos, int8_t* region,
                                  int32_t cap, int32_t* n_rows) {
  SelectLayout L;
  int32_t rc = layout_of(p, L);
  if (rc) return rc;
  if (!pos) return fail(SSM_E_INVAL, "null position array");
  if (cap < L.n_rows) return fail(SSM_E_CAPACITY, "cap %d < n_rows %d", cap, L.n_rows);
  for (int r = 0; r < L.n_rows; ++r) {
    int q, g;
    row_position(L, r, q, g);
    pos[r] = q;
    if (region) region[r] = (int8_t)g;
  }
  if (n_rows) *n_rows = L.n_rows;
  return ok();
}

int32_t ssm_select_suffix(const ssm_select_params* p, int32_t batch, int32_t seq_len,
                          const int32_t* pad, const int32_t* d_tokens, int32_t* d_pos,
                          int32_t* d_tok_c, int8_t* d_region, int32_t cap, int32_t* n_rows,
                          int32_t* n_suffix, int32_t* first_out_row, void* stream) {
  SelectLayout L;
  int32_t rc = layout_of(p, L);
  if (rc) return rc;
  if (batch < 1) return fail(SSM_E_INVAL, "batch %d < 1", batch);
  Pads pads;
  if ((rc = pads_of(pad, batch, p->prompt_len, pads))) return rc;
  if (seq_len != p->prompt_len + p->gen_len)
    return fail(SSM_E_INVAL, "seq_len %d != prompt_len + gen_len", seq_len);
  if (!d_tokens || !d_pos || !d_tok_c) return fail(SSM_E_INVAL, "null device pointer");
  if (cap < L.n_rows) return fail(SSM_E_CAPACITY, "cap %d < n_rows %d", cap, L.n_rows);
  if (n_rows) *n_rows = L.n_rows;
  if (n_suffix) *n_suffix = L.n_suffix;
  if (first_out_row) *first_out_row = L.n_prefix;
  hipStream_t st = (hipStream_t)stream;
  PROF_TRY("select", launch_select(L, batch, seq_len, d_tokens, d_pos, d_tok_c, d_region, cap, pads, st));
  return ok();
}

int32_t ssm_embed_suffix(const ssm_model* m, int32_t batch, int32_t seq_len, const int32_t* pad,
                         const int32_t* d_tok_c, int32_t tok_stride, const int32_t* d_pos,
                         const int8_t* d_region, int32_t n_rows, const int32_t* d_pred_ids,
                         const float* d_pred_w, const int32_t* d_pred_step, int32_t prev_step,
                         int32_t k, float alpha, float* d_x, void* stream) {
  if (!m) return fail(SSM_E_INVAL, "null model");
  if (m->dtype != SSM_DT_F32 && m->dtype != SSM_DT_BF16) return fail(SSM_E_INVAL, "unknown dtype");
  if (!m->tok_emb || m->d_model <= 0 || m->vocab <= 1 || m->mask_id < 0 || m->mask_id >= m->vocab)
    return fail(SSM_E_INVAL, "bad embedding table description");
  if (batch < 1 || seq_len < 1 || n_rows < 0 || tok_stride < n_rows)
    return fail(SSM_E_INVAL, "bad sizes (batch %d, seq_len %d, n_rows %d, tok_stride %d)", batch, seq_len, n_rows, tok_stride);
  if (k < 1 || k > 8) return fail(SSM_E_INVAL, "k %d not in [1, 8]", k);
  if (!(alpha >= 0.f && alpha <= 1.f)) return fail(SSM_E_INVAL, "alpha not in [0, 1]");
  if (!d_tok_c || !d_pos || !d_region || !d_pred_ids || !d_pred_w || !d_pred_step || !d_x)
    return fail(SSM_E_INVAL, "null device pointer");
  Pads pads;
  int32_t rc = pads_of(pad, batch, seq_len, pads);
  if (rc) return rc;
  hipStream_t st = (hipStream_t)stream;
  PROF_TRY("embed", launch_embed(m->dtype, m->tok_emb, m->d_model, m->vocab, m->mask_id, batch,
                                 seq_len, d_tok_c, tok_stride, d_pos, d_region, n_rows, d_pred_ids,
                                 d_pred_w, d_pred_step, prev_step, k, alpha, d_x, pads, st));
  return ok();
}

int32_t ssm_workspace_size(const ssm_model* m, int32_t batch, int32_t max_rows, size_t* bytes) {
  int32_t rc = check_model(m);
  if (rc) return rc;
  if (batch < 1 || max_rows < 1 || !bytes) return fail(SSM_E_INVAL, "bad workspace query");
  *bytes = ws_layout(m, batch, max_rows).total;
  return ok();
}

int32_t ssm_denoise_step(const ssm_model* m, const ssm_kv_cache* cache, int32_t cache_mode,
                         int32_t n_cached, int32_t batch, const int32_t* pad, const int32_t* d_pos,
                         int32_t n_rows, const float* d_x, int32_t first_out_row, int32_t k,
                         int32_t* d_argmax, float* d_conf, int32_t* d_topk_ids, float* d_topk_w,
                         float* d_logits_dbg, float* d_hidden_dbg, void* d_ws, size_t ws_bytes,
                         void* stream) {
  int32_t rc = check_model(m);
  if (rc) return rc;
  if (batch < 1 || n_rows < 1) return fail(SSM_E_INVAL, "batch %d / n_rows %d < 1", batch, n_rows);
  if (first_out_row < 0 || first_out_row >= n_rows)
    return fail(SSM_E_INVAL, "first_out_row %d not in [0, n_rows)", first_out_row);
  if (k < 1 || k > 8 || k > m->vocab - 1) return fail(SSM_E_INVAL, "k %d not in [1, 8]", k);
  if (!d_pos || !d_x || !d_argmax || !d_conf || !d_topk_ids || !d_topk_w || !d_ws)
    return fail(SSM_E_INVAL, "null device pointer");
  if (!cache || !cache->k || !cache->v) return fail(SSM_E_INVAL, "null KV cache");
  if (cache_mode == SSM_CACHE_OFF || cache_mode == SSM_CACHE_WRITE) {
    if (n_cached != 0) return fail(SSM_E_INVAL, "n_cached must be 0 unless cache_mode is READ");
  } else if (cache_mode == SSM_CACHE_READ) {
    if (n_cached < 1) return fail(SSM_E_INVAL, "cache_mode READ needs n_cached >= 1");
  } else {
    return fail(SSM_E_INVAL, "unknown cache_mode %d", cache_mode);
  }
  if ((long long)n_cached + n_rows > cache->capacity)
    return fail(SSM_E_CAPACITY, "cache capacity %d < n_cached %d + n_rows %d", cache->capacity, n_cached, n_rows);
  const WsLayout w = ws_layout(m, batch, n_rows);
  if (ws_bytes < w.total) return fail(SSM_E_CAPACITY, "workspace %zu < %zu bytes", ws_bytes, w.total);
  // padding lies in the prefix: the cached slots, or the prefix rows
  Pads pads;
  if ((rc = pads_of(pad, batch, cache_mode == SSM_CACHE_READ ? n_cached : first_out_row, pads)))
    return rc;

  hipStream_t st = (hipStream_t)stream;
  const int dt = m->dtype;
  const int d = m->d_model, H = m->n_heads, Hkv = m->n_kv_heads, dh = m->head_dim;
  const int F = m->ffn_dim, V = m->vocab;
  const int Mt = batch * n_rows, n_out = n_rows - first_out_row, Mo = batch * n_out;
  const int Nk = n_cached + n_rows;
  const size_t es = dt == SSM_DT_BF16 ? 2 : 4;
  char* ws = (char*)d_ws;
  float* resid = (float*)(ws + w.resid);
  // the lo parts of layer l's projection inputs, or null where it rounds once
  struct LoParts { bf16_t *xn, *attn, *act; };
  auto lo_of = [&](int l) {
    const bool p = pair_in_layer(m, l);
    return LoParts{p ? (bf16_t*)(ws + w.xn_lo) : nullptr, p ? (bf16_t*)(ws + w.attn_lo) : nullptr,
                   p ? (bf16_t*)(ws + w.act_lo) : nullptr};
  };
  // every step-local operand has Mt rows; the LM head input has Mo rows
  const int Gt = row_groups(Mt), Go = row_groups(Mo);
  const LoParts head_lo = lo_of(m->n_layers);
  const ActOut head_out{ws + w.xn, head_lo.xn, d, Go};
  const ActIn head_in{ws + w.xn, head_lo.xn, d, Go};
  void* qb = ws + w.q;
  float2* rope = (float2*)(ws + w.rope);
  SplitWs sws{(float*)(ws + w.part), w.part_floats};
  AttnWs aws{(float*)(ws + w.opart), (float*)(ws + w.ml), ATTN_MAX_SPLITS};
  float* logits = d_logits_dbg ? d_logits_dbg : (float*)(ws + w.logits);
  const size_t layer_kv = (size_t)batch * Hkv * cache->capacity * dh * es;

  PROF_TRY("rope_table", launch_rope_table(d_pos, n_rows, dh, m->rope_base, rope, batch, pads, st));
  HIP_TRY(hipMemcpyAsync(resid, d_x, (size_t)Mt * d * 4, hipMemcpyDeviceToDevice, st));
  // the attention norm of layer 0 runs alone; every later norm follows the
  // residual projection before it (fused with its split-K completion)
  if (m->n_layers > 0)
    PROF_TRY("norm", launch_norm(dt, resid, d, m->layers[0].attn_norm, m->rms_eps,
                                 ActOut{ws + w.xn, lo_of(0).xn, d, Gt}, Mt, Mt, 0, 0, st));
  for (int l = 0; l < m->n_layers; ++l) {
    const ssm_layer& y = m->layers[l];
    const LoParts lo = lo_of(l);
    const ActOut xn_out{ws + w.xn, lo.xn, d, Gt}, attn_out{ws + w.attn, lo.attn, H * dh, Gt},
        act_out{ws + w.act, lo.act, F, Gt};
    const ActIn xn_in{ws + w.xn, lo.xn, d, Gt}, attn_in{ws + w.attn, lo.attn, H * dh, Gt},
        act_in{ws + w.act, lo.act, F, Gt};
    // the norm that ends this layer feeds the next layer (or the LM head)
    const ActOut next_out{ws + w.xn, lo_of(l + 1).xn, d, Gt};
    char* kc = (char*)cache->k + l * layer_kv;
    char* vc = (char*)cache->v + l * layer_kv;
    // attention block (its input norm is in xn)
    QKVOut qo{qb, kc, vc, cache->capacity, n_cached, n_rows, rope, pads.any};
    PROF_TRY("gemm_qkv", gemm_qkv(dt, xn_in, Mt, d, y.wq, y.wk, y.wv, H, Hkv, dh, qo, sws, st));
    PROF_TRY("attention", attention(dt == SSM_DT_BF16 ? ATTN_F16 : ATTN_F32, qb, kc, vc, batch, H,
                                    Hkv, dh, n_rows, Nk, cache->capacity, attn_out, aws, pads,
                                    st));
    const NormTo ffn_norm{y.ffn_norm, m->rms_eps, xn_out};
    PROF_TRY("gemm_o", gemm_resid(dt, "o", attn_in, Mt, H * dh, y.wo, d, resid, sws, st, &ffn_norm));
    // feed-forward block
    PROF_TRY("gemm_gate_up", gemm_swiglu(dt, xn_in, Mt, d, y.w_gate, y.w_up, F, act_out, sws, st));
    const bool more = l + 1 < m->n_layers;
    const NormTo next_norm{more ? m->layers[l + 1].attn_norm : nullptr, m->rms_eps, next_out};
    PROF_TRY("gemm_down", gemm_resid(dt, "down", act_in, Mt, F, y.w_down, d, resid, sws, st,
                                     more ? &next_norm : nullptr));
  }
  if (d_hidden_dbg)
    HIP_TRY(hipMemcpyAsync(d_hidden_dbg, resid, (size_t)Mt * d * 4, hipMemcpyDeviceToDevice, st));
  // final norm and LM head over the output rows only: output row o is row
  // first_out_row + o % n_out of sequence o / n_out
  PROF_TRY("norm", launch_norm(dt, resid, d, m->final_norm, m->rms_eps, head_out, Mo, n_out,
                               n_rows, first_out_row, st));
  if (dt == SSM_DT_BF16) {
    PROF_TRY("gemm_lm_head", lm_head_stats(head_in, Mo, d, m->lm_head, V, m->mask_id, k,
                                           ws + w.lmstats, d_logits_dbg, d_argmax, d_conf,
                                           d_topk_ids, d_topk_w, st));
  } else {
    PROF_TRY("gemm_lm_head", gemm_store_f32(head_in, Mo, d, m->lm_head, V, logits, V, sws, st));
    PROF_TRY("rowstats", launch_rowstats(logits, Mo, V, V, m->mask_id, k, d_argmax, d_conf,
                                         d_topk_ids, d_topk_w, st));
  }
  return ok();
}

// Largest split-KV count the attention launcher picks for this grid: it never
// exceeds 512 workgroups over (64-row query tiles x sequences x heads).
static int attn_max_splits(int batch, int n_heads, int n_q) {
  const long tiles = (long)ceil_div(n_q > 0 ? n_q : 1, 64) * batch * n_heads;
  long s = 512 / tiles;
  if (s > ATTN_MAX_SPLITS) s = ATTN_MAX_SPLITS;
  return s < 1 ? 1 : (int)s;
}

int32_t ssm_attention_workspace_size(int32_t batch, int32_t n_heads, int32_t n_q, size_t* bytes) {
  if (!bytes || batch < 1 || n_heads < 1 || n_q < 0) return fail(SSM_E_INVAL, "bad arguments");
  const size_t rows = (size_t)attn_max_splits(batch, n_heads, n_q) * batch * n_heads * n_q;
  *bytes = align256(rows * 128 * 4) + align256(rows * 2 * 4);
  return ok();
}

int32_t ssm_attention(int32_t dtype, int32_t batch, int32_t n_heads, int32_t n_kv_heads,
                      int32_t n_q, int32_t n_keys, int32_t capacity, const void* d_q,
                      const void* d_k, const void* d_v, float* d_out, void* d_ws, size_t ws_bytes,
                      void* stream) {
  if (dtype != SSM_DT_BF16 && dtype != SSM_DT_F16)
    return fail(SSM_E_INVAL, "attention operands must be SSM_DT_BF16 or SSM_DT_F16 (got %d)", dtype);
  if (batch < 1 || n_heads < 1 || n_kv_heads < 1 || n_q < 0 || n_keys < 1 || capacity < 1)
    return fail(SSM_E_INVAL, "bad sizes");
  if (n_heads % n_kv_heads) return fail(SSM_E_SHAPE, "n_heads %d not a multiple of n_kv_heads %d", n_heads, n_kv_heads);
  if (n_keys > capacity) return fail(SSM_E_CAPACITY, "n_keys %d > capacity %d", n_keys, capacity);
  if (!d_q || !d_k || !d_v || !d_out || !d_ws) return fail(SSM_E_INVAL, "null device pointer");
  size_t need = 0;
  ssm_attention_workspace_size(batch, n_heads, n_q, &need);
  if (ws_bytes < need) return fail(SSM_E_CAPACITY, "workspace %zu < %zu bytes", ws_bytes, need);
  const int max_splits = attn_max_splits(batch, n_heads, n_q);
  const size_t rows = (size_t)max_splits * batch * n_heads * n_q;
  AttnWs aws{(float*)d_ws, (float*)((char*)d_ws + align256(rows * 128 * 4)), max_splits};
  const ActOut out{d_out, nullptr, n_heads * 128, 0, 1};
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(attention(dtype == SSM_DT_F16 ? ATTN_F16 : ATTN_BF16, d_q, d_k, d_v, batch, n_heads,
                    n_kv_heads, 128, n_q, n_keys, capacity, out, aws, Pads{}, st));
  return ok();
}

// Bytes of split-KV partial results an attention launch of these sizes uses
// (0 when it does not split the key range).
static size_t attn_partial_bytes(int dtype, int32_t batch, int32_t n_heads, int32_t n_q,
                                 int32_t n_keys, int max_splits) {
  const int S = attention_splits(dtype, batch, n_heads, n_q, n_keys, max_splits, nullptr);
  if (S <= 1) return 0;
  const size_t rows = (size_t)S * batch * n_heads * n_q;
  return align256(rows * 128 * 4) + align256(rows * 2 * 4);
}

int32_t ssm_attention_static(int32_t dtype, int32_t batch, int32_t n_heads, int32_t n_kv_heads,
                             int32_t n_q, int32_t n_keys, int32_t capacity, const void* d_q,
                             const void* d_k, const void* d_v, float* d_out, void* stream) {
  if (dtype != SSM_DT_BF16 && dtype != SSM_DT_F16)
    return fail(SSM_E_INVAL, "attention operands must be SSM_DT_BF16 or SSM_DT_F16 (got %d)", dtype);
  if (batch < 1 || n_heads < 1 || n_kv_heads < 1 || n_q < 0 || n_keys < 1 || capacity < 1)
    return fail(SSM_E_INVAL, "bad sizes");
  if (n_heads % n_kv_heads) return fail(SSM_E_SHAPE, "n_heads %d not a multiple of n_kv_heads %d", n_heads, n_kv_heads);
  if (n_keys > capacity) return fail(SSM_E_CAPACITY, "n_keys %d > capacity %d", n_keys, capacity);
  if (!d_q || !d_k || !d_v || !d_out) return fail(SSM_E_INVAL, "null device pointer");
  // the split count of ssm_attention, so both give identical results
  const int ad = dtype == SSM_DT_F16 ? ATTN_F16 : ATTN_BF16;
  const int max_splits = attn_max_splits(batch, n_heads, n_q);
  const size_t need = attn_partial_bytes(ad, batch, n_heads, n_q, n_keys, max_splits);
  if (need > SSM_ATTENTION_STATIC_SCRATCH_BYTES)
    return fail(SSM_E_CAPACITY, "split-KV partials need %zu bytes, above the %d-byte static scratch "
                "(ssm_attention with a workspace has no such limit)", need,
                SSM_ATTENTION_STATIC_SCRATCH_BYTES);
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= MAX_DEVICES) return fail(SSM_E_UNSUPPORTED, "device %d beyond %d", dev, MAX_DEVICES);
  void* base = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
      void* p = nullptr;
      HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
      g_scratch_ptr[dev] = p;
    }
    base = g_scratch_ptr[dev];
  }
  // partial outputs first, then the (max, sum) pairs, as attn_partial_bytes
  // counts them; every entry is written by its split before the merge reads
  // it, so nothing needs clearing between calls
  const int S = attention_splits(ad, batch, n_heads, n_q, n_keys, max_splits, nullptr);
  const size_t rows = (size_t)S * batch * n_heads * n_q;
  const AttnWs aws{(float*)base, (float*)((char*)base + align256(rows * 128 * 4)), max_splits};
  const ActOut out{d_out, nullptr, n_heads * 128, 0, 1};
  HIP_TRY(attention(ad, d_q, d_k, d_v, batch, n_heads, n_kv_heads, 128, n_q, n_keys, capacity, out,
                    aws, Pads{}, (hipStream_t)stream));
  return ok();
}

int32_t ssm_gather_rows(int32_t batch, int32_t src_rows, int32_t width, const void* d_src,
                        const int32_t* d_pos, int32_t n_rows, void* d_dst, void* stream) {
  if (batch < 1 || src_rows < 0 || width < 8 || width % 8 || n_rows < 0)
    return fail(SSM_E_INVAL, "bad sizes (width must be a positive multiple of 8)");
  if (n_rows > 0 && (!d_src || !d_pos || !d_dst)) return fail(SSM_E_INVAL, "null device pointer");
  HIP_TRY(launch_gather_rows(batch, src_rows, width, (const bf16_t*)d_src, d_pos, n_rows,
                             (bf16_t*)d_dst, (hipStream_t)stream));
  return ok();
}

int32_t ssm_unmask(int32_t* d_tokens, int32_t batch, int32_t seq_len, const int32_t* pad,
                   int32_t block_start, int32_t block_size, int32_t mask_id, int32_t rule,
                   int32_t n_per_step, float threshold, const int32_t* d_argmax, const float* d_conf,
                   const int32_t* d_topk_ids, const float* d_topk_w, int32_t k, int32_t n_out,
                   const int32_t* d_pos_out, int32_t step, int32_t* d_pred_ids, float* d_pred_w,
                   int32_t* d_pred_step, uint8_t* d_selected, int32_t* d_masked_left,
                   void* stream) {
  if (batch < 1 || seq_len < 1) return fail(SSM_E_INVAL, "bad batch / seq_len");
  if (block_size < 1 || block_size > 1024) return fail(SSM_E_INVAL, "block_size %d not in [1, 1024]", block_size);
  if (block_start < 0 || block_start + block_size > seq_len)
    return fail(SSM_E_INVAL, "block [%d, %d) outside the sequence", block_start, block_start + block_size);
  if (n_out < block_size) return fail(SSM_E_INVAL, "n_out %d < block_size %d", n_out, block_size);
  if (k < 1 || k > 8) return fail(SSM_E_INVAL, "k %d not in [1, 8]", k);
  if (rule != SSM_UNMASK_TOPN && rule != SSM_UNMASK_THRESHOLD && rule != SSM_UNMASK_MARGIN)
    return fail(SSM_E_INVAL, "unknown rule %d", rule);
  if (rule == SSM_UNMASK_TOPN && n_per_step < 1) return fail(SSM_E_INVAL, "n_per_step %d < 1", n_per_step);
  if (rule == SSM_UNMASK_MARGIN && k < 2) return fail(SSM_E_INVAL, "the margin rule needs k >= 2");
  if (!d_tokens || !d_argmax || !d_conf || !d_topk_ids || !d_topk_w) return fail(SSM_E_INVAL, "null device pointer");
  if (n_out > block_size && (!d_pos_out || !d_pred_ids || !d_pred_w || !d_pred_step))
    return fail(SSM_E_INVAL, "null prediction-state pointer");
  Pads pads;
  int32_t rc = pads_of(pad, batch, block_start, pads);
  if (rc) return rc;
  hipStream_t st = (hipStream_t)stream;
  PROF_TRY("unmask", launch_unmask(d_tokens, batch, seq_len, block_start, block_size, mask_id,
                                   rule, n_per_step, threshold, d_argmax, d_conf, d_topk_ids,
                                   d_topk_w, k, n_out, d_pos_out, step, d_pred_ids, d_pred_w,
                                   d_pred_step, d_selected, d_masked_left, pads, st));
  return ok();
}

int32_t ssm_early_stop(int32_t* d_tokens, int32_t batch, int32_t seq_len, const int32_t* pad,
                       int32_t block_start, int32_t block_size, int32_t eos_id, int32_t* d_done,
                       void* stream) {
  if (batch < 1 || seq_len < 1) return fail(SSM_E_INVAL, "bad batch / seq_len");
  if (block_size < 1 || block_start < 0 || block_start + block_size > seq_len)
    return fail(SSM_E_INVAL, "block [%d, %d) outside the sequence", block_start, block_start + block_size);
  if (eos_id < 0) return fail(SSM_E_INVAL, "eos_id %d < 0", eos_id);
  if (!d_tokens || !d_done) return fail(SSM_E_INVAL, "null device pointer");
  Pads pads;
  int32_t rc = pads_of(pad, batch, block_start, pads);
  if (rc) return rc;
  hipStream_t st = (hipStream_t)stream;
  PROF_TRY("early_stop", launch_early_stop(d_tokens, batch, seq_len, block_start, block_size,
                                           eos_id, d_done, pads, st));
  return ok();
}

int32_t ssm_profile_enable(int32_t on) {
  g_prof_on = on != 0;
  prof_clear();
  return ok();
}

int32_t ssm_profile_query(const char* tag, int32_t kernel, int32_t* count, double* total_ms) {
  if (!tag || !count || !total_ms) return fail(SSM_E_INVAL, "null argument");
  int n = 0;
  double tot = 0.0;
  for (auto& r : g_prof) {
    if (strcmp(r.tag, tag) != 0 || (kernel >= 0 && r.ordinal != kernel)) continue;
    hipError_t e = hipEventSynchronize(r.b);
    if (e != hipSuccess) return fail(SSM_E_HIP, "hipEventSynchronize: %s", hipGetErrorString(e));
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return fail(SSM_E_HIP, "hipEventElapsedTime: %s", hipGetErrorString(e));
    ++n;
    tot += ms;
  }
  *count = n;
  *total_ms = tot;
  return ok();
}

}  // extern "C"
