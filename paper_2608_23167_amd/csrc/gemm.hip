// Projections of the decoder layer: C = A * W^T with A [M, K] activations
// and W [N, K] row-major weights (nn.Linear layout).
//
// bfloat16 path.  The activation operand arrives as bfloat16 (hi) or as a
// bfloat16 pair (hi, lo) with hi + lo = the float32 value to about 16
// significant bits; with the pair each product is taken twice (hi*W + lo*W),
// the weights being exact in bfloat16.  MFMA v_mfma_f32_16x16x32_bf16, fp32
// accumulation.  A workgroup of 512 threads computes a 128 x BN output tile
// with two kinds of waves (one of each per SIMD):
//   * staging waves (4-7) stream the weight tile from HBM: a ring of four
//     K-steps of 16-byte loads in flight per thread, written into a ring of
//     three or four LDS buffers two or three K-steps ahead of their use;
//   * compute waves (0-3) each own 32 rows x BN columns: they load their
//     activation fragments straight from global memory (small, shared by
//     every workgroup, L2-resident, stored in fragment order so that each
//     16-byte-per-lane load reads 1 KB contiguously) two K-steps ahead, read
//     the weight fragments from LDS and issue the MFMAs.
// Splitting the roles keeps the in-order retirement of vector loads from
// coupling the long HBM latency of the weights to the MFMA issue.  One
// barrier per K-step (64) hands the LDS buffers over.  The output tile is
// staged through LDS so that the epilogue can combine any two columns of the
// tile and store coalesced.
//
// Every output tile of BN columns reads its first BN/2 weight rows from one
// base pointer and its last BN/2 from another.  That is how the fused
// epilogues get the pairs they need without any weight repacking:
//   QKV    : columns (c, c + dh/2) of one head -> rotate-half RoPE, then the
//            query buffer or the KV cache slot of the row;
//   SwiGLU : gate row j and up row j -> silu(g) * u, written as the next
//            projection's activation (pair);
//   resid  : plain rows -> residual stream += value;
//   LM head: per-row softmax statistics of each half tile (merged later).
// Split-K writes float32 partial tiles that a second kernel sums in a fixed
// order before applying the same epilogue.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <type_traits>

#include "internal.h"

namespace ssm {

// ---------------------------------------------------------------------------
// Epilogue policies
// ---------------------------------------------------------------------------
// Eight consecutive row-major elements (16 or 32 bytes, aligned).
__device__ __forceinline__ void store_row8(float* p, const float (&v)[8]) {
  *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
  *(float4*)(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void store_row8(bf16_t* p, const float (&v)[8]) {
  uint16_t h[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = f2bf(v[e]);
  *(u32x4_t*)p = *(const u32x4_t*)h;
}
__device__ __forceinline__ void store_row8(f16_t* p, const float (&v)[8]) {
  f16x8_t h;
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = (f16_t)v[e];
  *(f16x8_t*)p = h;
}

// Column tile t of width BN covers BN / 2 consecutive entries of the
// concatenated first halves of all heads (query heads, then key, then value)
// and the same entries of the second halves, so the pairs (i, i + d_h / 2)
// that RoPE rotates always meet in one tile, at any width whose half is a
// multiple of 8.  T: weight type; TO: type of q and of the KV cache (float16
// for bfloat16 weights: the attention operands keep three more significand
// bits than bfloat16).
template <typename T, typename TO = T>
struct PolQKV {
  static constexpr bool PAIRED = true;
  static constexpr bool ROW_MAP = true;
  const T *wq, *wk, *wv;
  int ldb, H, Hkv, dh;
  TO *q, *kc, *vc;
  int cap, n_cached, n_rows;
  const float2* rope;
  int rope_per_seq;    // 1: RoPE table [B, n_rows, d_h / 2] (padded batch), 0: [n_rows, d_h / 2]

  __device__ __forceinline__ const T* head_rows(int head) const {
    if (head < H) return wq + (size_t)head * dh * ldb;
    if (head < H + Hkv) return wk + (size_t)(head - H) * dh * ldb;
    return wv + (size_t)(head - H - Hkv) * dh * ldb;
  }
  // weight row of tile row r: rows [0, BN/2) from the first halves, the rest
  // from the second
  __device__ __forceinline__ const T* b_row(int t, int BN, int r) const {
    const int half = dh / 2, second = r >= BN / 2;
    const int j = t * (BN / 2) + (second ? r - BN / 2 : r);
    const int head = j / half;
    return head_rows(head) + (size_t)(j - head * half + (second ? half : 0)) * ldb;
  }
  // both halves as row ranges; only for tiles whose half stays in one head
  // ((BN / 2) divides d_h / 2)
  __device__ __forceinline__ void b_ptrs(int t, int BN, const T*& lo, const T*& hi) const {
    lo = b_row(t, BN, 0);
    hi = lo + (size_t)(dh / 2) * ldb;
  }
  __device__ __forceinline__ void store(int m, int t, int c, int BN, float vlo, float vhi) const {
    const int half = dh / 2, j = t * (BN / 2) + c, head = j / half, i = j - head * half;
    const int s = m / n_rows, row = m % n_rows;
    if (head < H + Hkv) {
      const float2 cs = rope[((size_t)(rope_per_seq ? s : 0) * n_rows + row) * half + i];
      const float a = vlo * cs.x - vhi * cs.y;
      const float b = vhi * cs.x + vlo * cs.y;
      vlo = a;
      vhi = b;
    }
    TO* dst;
    if (head < H) dst = q + (((size_t)s * H + head) * n_rows + row) * dh;
    else if (head < H + Hkv) dst = kc + (((size_t)s * Hkv + (head - H)) * cap + n_cached + row) * dh;
    else dst = vc + (((size_t)s * Hkv + (head - H - Hkv)) * cap + n_cached + row) * dh;
    stf(dst + i, vlo);
    stf(dst + i + half, vhi);
  }
  // columns c0 .. c0 + 7 of both halves (c0 a multiple of 8: one head)
  __device__ __forceinline__ void store8(int m, int t, int c0, int BN, const float (&vlo)[8],
                                         const float (&vhi)[8]) const {
    const int half = dh / 2, j = t * (BN / 2) + c0, head = j / half, i0 = j - head * half;
    const int s = m / n_rows, row = m % n_rows;
    float a[8], b[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[e] = vlo[e];
      b[e] = vhi[e];
    }
    if (head < H + Hkv) {
      const float2* cs = rope + ((size_t)(rope_per_seq ? s : 0) * n_rows + row) * half + i0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float2 r = cs[e];
        a[e] = vlo[e] * r.x - vhi[e] * r.y;
        b[e] = vhi[e] * r.x + vlo[e] * r.y;
      }
    }
    TO* dst;
    if (head < H) dst = q + (((size_t)s * H + head) * n_rows + row) * dh;
    else if (head < H + Hkv) dst = kc + (((size_t)s * Hkv + (head - H)) * cap + n_cached + row) * dh;
    else dst = vc + (((size_t)s * Hkv + (head - H - Hkv)) * cap + n_cached + row) * dh;
    store_row8(dst + i0, a);
    store_row8(dst + i0 + half, b);
  }
};

template <typename T>
struct PolSwiGLU {
  static constexpr bool PAIRED = true;
  const T *wg, *wu;
  int ldb, F;
  ActOut act;
  __device__ __forceinline__ void b_ptrs(int t, int BN, const T*& lo, const T*& hi) const {
    lo = wg + (size_t)t * (BN / 2) * ldb;
    hi = wu + (size_t)t * (BN / 2) * ldb;
  }
  __device__ __forceinline__ void store(int m, int t, int c, int BN, float g, float u) const {
    const float silu = g / (1.0f + expf(-g));
    act.store<T>(m, t * (BN / 2) + c, silu * u);
  }
  __device__ __forceinline__ void store8(int m, int t, int c0, int BN, const float (&g)[8],
                                         const float (&u)[8]) const {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = g[e] / (1.0f + expf(-g[e])) * u[e];
    act.store8<T>(m, t * (BN / 2) + c0, v);
  }
};

template <typename T>
struct PolResid {
  static constexpr bool PAIRED = false;
  const T* w;
  int ldb, N;
  float* resid;
  __device__ __forceinline__ void b_ptrs(int t, int BN, const T*& lo, const T*& hi) const {
    lo = w + (size_t)t * BN * ldb;
    hi = lo + (size_t)(BN / 2) * ldb;
  }
  __device__ __forceinline__ void store1(int m, int n, float v) const {
    resid[(size_t)m * N + n] += v;
  }
  __device__ __forceinline__ void store8_1(int m, int n0, const float (&v)[8]) const {
    float4* p = (float4*)(resid + (size_t)m * N + n0);
    float4 a = p[0], b = p[1];
    a.x += v[0]; a.y += v[1]; a.z += v[2]; a.w += v[3];
    b.x += v[4]; b.y += v[5]; b.z += v[6]; b.w += v[7];
    p[0] = a;
    p[1] = b;
  }
};

template <typename T>
struct PolStore {
  static constexpr bool PAIRED = false;
  const T* w;
  int ldb, ldc;
  float* c;
  __device__ __forceinline__ void b_ptrs(int t, int BN, const T*& lo, const T*& hi) const {
    lo = w + (size_t)t * BN * ldb;
    hi = lo + (size_t)(BN / 2) * ldb;
  }
  __device__ __forceinline__ void store1(int m, int n, float v) const {
    c[(size_t)m * ldc + n] = v;
  }
  __device__ __forceinline__ void store8_1(int m, int n0, const float (&v)[8]) const {
    store_row8(c + (size_t)m * ldc + n0, v);
  }
};

// LM head: per-row partial softmax statistics of every half tile (64 vocab
// columns): running max, sum of exp(x - max) and the 8 largest logits with
// their ids, [MASK] excluded; optionally the logits themselves.
struct LMPartial {
  float m, s;
  float v[8];
  int id[8];
};

__device__ __forceinline__ bool stat_better(float v, int i, float w, int j) {
  return v > w || (v == w && i < j);
}

__device__ __forceinline__ void stat_insert(float (&tv)[8], int (&ti)[8], float v, int i) {
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const bool gt = stat_better(v, i, tv[q], ti[q]);
    const float ov = tv[q];
    const int oi = ti[q];
    tv[q] = gt ? v : ov;
    ti[q] = gt ? i : oi;
    v = gt ? ov : v;
    i = gt ? oi : i;
  }
}

template <typename T>
struct PolLMStats {
  static constexpr bool PAIRED = false;
  static constexpr bool TILE = true;
  const T* w;
  int ldb, N, mask_id;
  LMPartial* part;     // [M][2 * ntiles]
  int n_part;          // 2 * ntiles
  float* logits;       // optional [M][ldc]
  int ldc;
  __device__ __forceinline__ void b_ptrs(int t, int BN, const T*& lo, const T*& hi) const {
    lo = w + (size_t)t * BN * ldb;
    hi = lo + (size_t)(BN / 2) * ldb;
  }
  template <int BM, int BN, int CS>
  __device__ __forceinline__ void tile(const float* Cs, int m0, int M, int t) const {
    const int tid = threadIdx.x;
    if (logits) {
      for (int idx = tid; idx < BM * BN; idx += blockDim.x) {
        const int r = idx / BN, c = idx % BN;
        if (m0 + r < M) logits[(size_t)(m0 + r) * ldc + (size_t)t * BN + c] = Cs[r * CS + c];
      }
    }
    // thread -> (row, half): 2 threads per row, each over BN / 2 columns
    for (int idx = tid; idx < BM * 2; idx += blockDim.x) {
      const int r = idx >> 1, h = idx & 1;
      if (m0 + r >= M) continue;
      float tv[8];
      int ti[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) { tv[q] = -INFINITY; ti[q] = 0x7fffffff; }
      float mx = -INFINITY, sm = 0.f;
      const int c0 = h * (BN / 2);
      for (int c = c0; c < c0 + BN / 2; ++c) {
        const int v = t * BN + c;
        if (v == mask_id) continue;
        const float x = Cs[r * CS + c];
        if (x > mx) { sm = sm * expf(mx - x) + 1.0f; mx = x; }
        else sm += expf(x - mx);
        if (stat_better(x, v, tv[7], ti[7])) stat_insert(tv, ti, x, v);
      }
      LMPartial* o = part + (size_t)(m0 + r) * n_part + 2 * t + h;
      o->m = mx;
      o->s = sm;
#pragma unroll
      for (int q = 0; q < 8; ++q) { o->v[q] = tv[q]; o->id[q] = ti[q]; }
    }
  }
};

template <class P, class = void> struct has_tile { static constexpr bool value = false; };
template <class P> struct has_tile<P, std::void_t<decltype(P::TILE)>> {
  static constexpr bool value = P::TILE;
};
template <class P, class = void> struct has_row_map { static constexpr bool value = false; };
template <class P> struct has_row_map<P, std::void_t<decltype(P::ROW_MAP)>> {
  static constexpr bool value = P::ROW_MAP;
};

// Weight row r of column tile t (lo, hi: the tile's two half ranges from
// b_ptrs, for policies whose halves are row ranges).
template <class Pol, class T>
__device__ __forceinline__ const T* weight_row(const Pol& pol, int t, int BN, int r, const T* lo,
                                               const T* hi) {
  if constexpr (has_row_map<Pol>::value) return pol.b_row(t, BN, r);
  else return r < BN / 2 ? lo + (size_t)r * pol.ldb : hi + (size_t)(r - BN / 2) * pol.ldb;
}

// Applies the epilogue to a BM x BN float tile staged in LDS (row stride CS).
template <int BM, int BN, int CS, class Pol>
__device__ __forceinline__ void tile_epilogue(const Pol& pol, const float* Cs, int m0, int M,
                                              int t, float* part, int split, int ldp) {
  const int tid = threadIdx.x;
  if constexpr (has_tile<Pol>::value) {
    pol.template tile<BM, BN, CS>(Cs, m0, M, t);
  } else if (part) {
    // float32 partial tile, 8 columns per thread
    for (int idx = tid; idx < BM * (BN / 8); idx += blockDim.x) {
      const int r = idx / (BN / 8), c0 = (idx % (BN / 8)) * 8, gm = m0 + r;
      if (gm >= M) continue;
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = Cs[r * CS + c0 + e];
      store_row8(part + ((size_t)split * M + gm) * ldp + (size_t)t * BN + c0, v);
    }
  } else if constexpr (Pol::PAIRED) {
    // 8 columns of each half per thread; 16 consecutive threads take the 16
    // rows of one row group, which are adjacent chunks of the fragment order
    constexpr int C8 = BN / 16;
    for (int idx = tid; idx < BM * C8; idx += blockDim.x) {
      const int rest = idx >> 4, r = (rest / C8) * 16 + (idx & 15), c0 = (rest % C8) * 8;
      const int gm = m0 + r;
      if (gm >= M) continue;
      float lo[8], hi[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        lo[e] = Cs[r * CS + c0 + e];
        hi[e] = Cs[r * CS + c0 + BN / 2 + e];
      }
      pol.store8(gm, t, c0, BN, lo, hi);
    }
  } else {
    for (int idx = tid; idx < BM * (BN / 8); idx += blockDim.x) {
      const int r = idx / (BN / 8), c0 = (idx % (BN / 8)) * 8, gm = m0 + r;
      if (gm >= M) continue;
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = Cs[r * CS + c0 + e];
      pol.store8_1(gm, t * BN + c0, v);
    }
  }
}

// ---------------------------------------------------------------------------
// bfloat16 MFMA kernel
// ---------------------------------------------------------------------------
// Tile order: the grid is 1-D over (split, n-tile, m-tile) triples.
// Workgroups are dealt to the 8 XCDs round-robin by linear id, so id w runs
// on XCD w % 8; the order below gives each XCD a contiguous range of the
// triples, split-major, then n-tiles, m-tiles innermost.  The workgroups that
// share a weight tile then run on the same XCD at about the same time and
// read it once into that XCD's L2, and each XCD touches as few K-slices of
// the activations as possible, so that its slice stays resident in its L2.
__device__ __forceinline__ void tile_of(int w, int total, int ntm, int mt, int& split, int& tn,
                                        int& tm) {
  const int per = total / 8;
  const int v = w < per * 8 ? (w % 8) * per + (w / 8) : w;
  split = v / ntm;
  const int t = v % ntm;
  tn = t / mt;
  tm = t % mt;
}

// K-step handover between the two kinds of waves.  The buffer schedule below
// never lets a compute wave read an LDS buffer in the step in which it is
// rewritten, so the compute waves pass the barrier without waiting for their
// own outstanding LDS reads (the fence of __syncthreads would wait for them);
// the staging waves wait for their LDS writes to land first.  The empty asm
// statements keep the compiler from moving memory accesses across.
__device__ __forceinline__ void lds_handover_barrier() {
  asm volatile("s_barrier" ::: "memory");
}
__device__ __forceinline__ void lds_written_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Warp-specialised workgroup of 8 waves, BM rows (64, 128, 192 or 256) x BN
// columns.
//  * Waves 4-7 ("staging") stream the weight tile of each K-step (BN rows x 64
//    k, the HBM-bound stream) through a ring of 4 register stages into a ring
//    of 3 or 4 LDS buffers, 2 or 3 K-steps ahead.  A staging thread holds only BN / 32
//    x 16 bytes per stage, so the ring is deep at little register cost.
//  * Waves 0-3 ("compute") each own BM / 4 rows x all BN columns.  They load
//    their activation fragments (bfloat16 hi and optionally lo, L2-resident)
//    straight from global memory into registers in the MFMA operand layout,
//    two K-steps ahead, read the weight fragments from LDS one half-step
//    ahead of use, and run the MFMAs (v_mfma_f32_16x16x32_bf16) ordered so
//    that updates of one accumulator are FM * FN instructions apart.
// Loads retire in issue order per wave; keeping the two streams in different
// waves lets each wait only for its own data.  LDS carries only the weight
// tile (written once, read once by each compute wave).  Every K-step ends with
// one workgroup barrier on both paths.
template <int BM, int BN, int PW, bool SPLIT, class Pol>
__global__ void __launch_bounds__(512) gemm_bf16_kernel(Pol pol, const bf16_t* __restrict__ Ahi,
                                                        const bf16_t* __restrict__ Alo, int G,
                                                        int M, int k_per_split, int mt,
                                                        int n_split, float* __restrict__ part,
                                                        int ldp, int krot) {
  static_assert(BM == 64 || BM == 128 || BM == 192 || BM == 256, "4 compute waves of BM / 4 rows");
  constexpr int BK = 64, LS = BK + 8;            // LDS row stride (elements), 144 B
  constexpr int FM = BM / 64, FN = BN / 16;      // per compute wave: 16 FM rows x BN columns
  constexpr int RW = 16 * FM;
  constexpr int NA = SPLIT ? 2 : 1;
  constexpr int WR = BN / 32;                    // weight rows per staging thread per stage
  // LDS weight buffers: 4 (three K-steps ahead) for the 96-column tiles, 3
  // (two ahead) for the others, which measured 2-3% slower with 4
  constexpr int NBUF = BN == 96 ? 4 : 3;
  constexpr int AHEAD = NBUF - 1;                // K-steps the staging runs ahead
  static_assert(PW == 4 || PW == 8, "weight register ring of 4 or 8 K-steps");
  static_assert(AHEAD < PW, "the prologue refills the first AHEAD register sets");
  constexpr int BUF_ELEMS = BN * LS;
  constexpr int SMEM_W = NBUF * BUF_ELEMS * 2;
  constexpr int CS = BN + 4;
  constexpr int SMEM_C = BM * CS * 4;
  constexpr int SMEM = SMEM_W > SMEM_C ? SMEM_W : SMEM_C;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  bf16_t* Ws = (bf16_t*)smem;                    // [NBUF][BN][LS]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int t, mtile, split;
  tile_of(blockIdx.x, gridDim.x, gridDim.x / n_split, mt, split, t, mtile);
  const int m0 = mtile * BM;
  const int kbeg = split * k_per_split;
  const int nk = k_per_split / BK;               // a multiple of 4 (host-checked)
  const int last = nk - 1;
  // K-step kt of this tile reads K-step kmap(kt): column tiles start at
  // different K offsets, so the weight rows read at any one time do not all
  // share their low address bits
  const int rot = krot ? (int)(((long long)t * krot) % nk) : 0;
  auto kmap = [rot, nk](int k) {
    const int x = k + rot;
    return x >= nk ? x - nk : x;
  };
  float* Cs = (float*)smem;

  if (wave < 4) {
    // ------------------------------ compute waves ------------------------------
    // activation fragment i, half kk of K-step kt: the 1 KB fragment-order
    // block of row group (m0 + 32 wave + 16 i) / 16, lane l at 8 l (groups past
    // the allocation read the last one; rows past M are computed and discarded)
    const size_t a_kstep = (size_t)G * 1024;
    size_t a_off[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i)
      a_off[i] = (size_t)(kbeg >> 6) * a_kstep +
                 (size_t)min((m0 + RW * wave + 16 * i) >> 4, G - 1) * 1024 + lane * 8;
    // weight fragment j, half kk: LDS row 16 j + lane % 16, column 32 kk + 8 (lane / 16)
    const int wfrag = (lane & 15) * LS + (lane >> 4) * 8;
    f32x4_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    u32x4_t a0[NA][FM][2], a1[NA][FM][2];        // activation stages kt (even / odd)
    bf16x8_t wf0[FN], wf1[FN];                   // weight fragments: two halves of a K-step

#define LOAD_A(RA, KT)                                                                \
  do {                                                                                \
    _Pragma("unroll") for (int i = 0; i < FM; ++i)                                    \
    _Pragma("unroll") for (int kk = 0; kk < 2; ++kk) {                                \
      RA[0][i][kk] = *(const u32x4_t*)(Ahi + a_off[i] + kmap(KT) * a_kstep + kk * 512);  \
      if (SPLIT) RA[NA - 1][i][kk] = *(const u32x4_t*)(Alo + a_off[i] + kmap(KT) * a_kstep + kk * 512); \
    }                                                                                 \
  } while (0)
#define READ_W(F, BUF, KK)                                                            \
  do {                                                                                \
    const bf16_t* base_ = Ws + (BUF) * BUF_ELEMS + wfrag + (KK) * 32;                 \
    _Pragma("unroll") for (int j = 0; j < FN; ++j)                                    \
        F[j] = *(const bf16x8_t*)(base_ + j * 16 * LS);                               \
  } while (0)
#define MFMA_H(RA, F, KK)                                                             \
  do {                                                                                \
    _Pragma("unroll") for (int p = 0; p < NA; ++p)                                    \
    _Pragma("unroll") for (int i = 0; i < FM; ++i)                                    \
    _Pragma("unroll") for (int j = 0; j < FN; ++j)                                    \
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(                          \
            __builtin_bit_cast(bf16x8_t, RA[p][i][KK]), F[j], acc[i][j], 0, 0, 0);     \
  } while (0)
    // step kt: wf0 holds (kt, first half); read (kt, second half) into wf1,
    // use wf0; read (kt + 1, first half) into wf0, use wf1; fetch the
    // activations of kt + 2 into the set just used; barrier
#define CSTEP(KT, RA)                                                                 \
  do {                                                                                \
    const int kt_ = (KT);                                                             \
    READ_W(wf1, kt_ % NBUF, 1);                                                       \
    MFMA_H(RA, wf0, 0);                                                               \
    READ_W(wf0, (kt_ + 1) % NBUF, 0);                                                 \
    MFMA_H(RA, wf1, 1);                                                               \
    LOAD_A(RA, min(kt_ + 2, last));                                                   \
    lds_handover_barrier();                                                           \
  } while (0)

    if (m0 + RW * wave >= M) {
      // every row of this wave is padding (few rows, e.g. the LM head's
      // block rows): no loads or MFMAs, only the barrier schedule
      __syncthreads();
      for (int kt = 0; kt < nk; ++kt) lds_handover_barrier();
    } else {
      LOAD_A(a0, 0);
      LOAD_A(a1, min(1, last));
      __syncthreads();                             // weight stages 0 .. AHEAD - 1 are in LDS
      READ_W(wf0, 0, 0);
      for (int kt = 0; kt < nk; kt += 2) {
        CSTEP(kt, a0);
        CSTEP(kt + 1, a1);
      }
      // accumulators -> LDS tile: acc[i][j][r] = C[RW wave + 16i + 4*(lane/16) + r][16j + lane%16]
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            Cs[(RW * wave + i * 16 + (lane >> 4) * 4 + r) * CS + j * 16 + (lane & 15)] = acc[i][j][r];
    }
#undef LOAD_A
#undef READ_W
#undef MFMA_H
#undef CSTEP
  } else {
    // ------------------------------ staging waves ------------------------------
    const bf16_t *blo, *bhi;
    pol.b_ptrs(t, BN, blo, bhi);
    const int st = tid - 256, r0 = st >> 3, col = (st & 7) * 8;
    const bf16_t* w_src[WR];
#pragma unroll
    for (int i = 0; i < WR; ++i) {
      const int r = r0 + 32 * i;   // tile rows [0, BN/2) come from lo, the rest from hi
      w_src[i] = weight_row(pol, t, BN, r, blo, bhi) + kbeg + col;
    }
    u32x4_t sr[PW][WR];                          // stage x in register set x % PW
#define LOAD_S(S, KT)                                                                 \
  do {                                                                                \
    _Pragma("unroll") for (int i = 0; i < WR; ++i) S[i] = *(const u32x4_t*)(w_src[i] + kmap(KT) * BK); \
  } while (0)
#define STORE_S(S, BUF)                                                               \
  do {                                                                                \
    _Pragma("unroll") for (int i = 0; i < WR; ++i)                                    \
        *(u32x4_t*)(Ws + (BUF) * BUF_ELEMS + (r0 + 32 * i) * LS + col) = S[i];        \
  } while (0)
    // during step kt the compute waves read buffers kt % NBUF and (kt + 1) %
    // NBUF; the staging waves fill buffer (kt + AHEAD) % NBUF with stage
    // kt + AHEAD and fetch stage kt + AHEAD + PW into the register set it
    // came from
#pragma unroll
    for (int u = 0; u < PW; ++u) LOAD_S(sr[u], min(u, last));
#pragma unroll
    for (int u = 0; u < AHEAD; ++u) {
      STORE_S(sr[u], u);
      LOAD_S(sr[u], min(u + PW, last));
    }
    __syncthreads();                               // weight stages 0 .. AHEAD - 1 are in LDS
    for (int kt = 0; kt < nk; kt += PW) {          // nk is a multiple of PW (host-checked)
#pragma unroll
      for (int u = 0; u < PW; ++u) {
        const int x = kt + u + AHEAD;              // the stage stored in this step
        STORE_S(sr[(u + AHEAD) % PW], x % NBUF);
        LOAD_S(sr[(u + AHEAD) % PW], min(x + PW, last));
        lds_written_barrier();
      }
    }
#undef LOAD_S
#undef STORE_S
  }
  __syncthreads();
  tile_epilogue<BM, BN, CS>(pol, Cs, m0, M, t, part, split, ldp);
}

// ---------------------------------------------------------------------------
// bfloat16 MFMA kernel for many rows (block-start steps of long prompts)
// ---------------------------------------------------------------------------
// Waits until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// A BM x BN output tile per workgroup of 8 waves in a WM x WN grid; wave
// (wm, wn) owns rows (BM / WM) wm .. and columns (BN / WN) wn .. (FM x FN MFMA
// blocks).  Shapes: 256 x 128 (4 x 2 waves) and 128 x 256 (2 x 4).
// Both operands go from global memory straight into LDS (global_load_lds,
// 1 KB per instruction) in K-steps of 32, through a ring of two stages:
//  * activations: the fragment-order operand already holds each 16-row x
//    32-column MFMA operand as 1 KB, so a stage is BM / 16 such blocks per
//    part (hi, lo), copied as they are;
//  * weights: BN / 16 blocks of 16 rows x 32 columns, lane l of a block
//    holding row l % 16, columns 8 (l / 16) .. + 7: the B-operand layout.
// Every operand read is then one conflict-free 16-byte LDS load per lane.
// With 64-80 KB of LDS and at most 128 VGPRs, two workgroups share a CU, so
// one workgroup's barrier wait overlaps the other's MFMAs.  The output tile
// goes through LDS in chunks of EB rows into the same epilogues as
// gemm_bf16_kernel.
template <int BM, int BN, int WM, int WN, int NS, bool SPLIT, class Pol>
__global__ void __launch_bounds__(WM * WN * 64, (BM / WM) * (BN / WN) > 4096 ? 2 : 4) gemm_big_kernel(Pol pol, const bf16_t* __restrict__ Ahi,
                                                          const bf16_t* __restrict__ Alo, int G,
                                                          int M, int k_per_split, int mt,
                                                          int n_split, float* __restrict__ part,
                                                          int ldp) {
  constexpr int NW = WM * WN;
  static_assert(NW == 8 || NW == 16, "8 or 16 waves");
  static_assert(NS == 2 || NS == 3, "ring of 2 or 3 stages");
  constexpr int BK = 32;
  constexpr int NA = SPLIT ? 2 : 1;
  constexpr int GB = BM / 16;                                   // row groups per tile
  constexpr int A_BLOCKS = GB * NA, BLOCKS = A_BLOCKS + BN / 16;
  static_assert(BLOCKS % NW == 0, "whole blocks per wave");
  constexpr int CPW = BLOCKS / NW, STAGE = BLOCKS * 1024;
  constexpr int RW = BM / WM, CW = BN / WN, FM = RW / 16, FN = CW / 16;
  constexpr int CS = BN + 4;
  constexpr int EB = BN > 128 ? BM / 2 : 128;                   // epilogue chunk rows
  constexpr int SMEM_W = NS * STAGE, SMEM_C = EB * CS * 4;
  constexpr int SMEM = SMEM_W > SMEM_C ? SMEM_W : SMEM_C;
  static_assert(EB % RW == 0, "a wave's rows in one epilogue chunk");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave % WM, wn = wave / WM;
  int t, mtile, split;
  tile_of(blockIdx.x, gridDim.x, gridDim.x / n_split, mt, split, t, mtile);
  const int m0 = mtile * BM;
  const int kbeg = split * k_per_split, nk = k_per_split / BK, last = nk - 1;

  // this wave's blocks of a stage: block c = wave * CPW + i; c < A_BLOCKS are
  // activation blocks (part c / GB, row group c % GB), the rest weight blocks
  const bf16_t *blo, *bhi;
  pol.b_ptrs(t, BN, blo, bhi);
  const size_t a_kstep = (size_t)G * 1024;
  const bf16_t* src[CPW];
  bool is_a[CPW];
#pragma unroll
  for (int i = 0; i < CPW; ++i) {
    const int c = wave * CPW + i;
    is_a[i] = c < A_BLOCKS;
    if (c < A_BLOCKS) {
      const int grp = min((m0 >> 4) + (c % GB), G - 1);   // groups past the allocation: the last
      src[i] = ((c / GB) ? Alo : Ahi) + (size_t)(kbeg >> 6) * a_kstep + (size_t)grp * 1024 + lane * 8;
    } else {
      const int r = 16 * (c - A_BLOCKS) + (lane & 15);
      src[i] = weight_row(pol, t, BN, r, blo, bhi) + kbeg + 8 * (lane >> 4);
    }
  }
  // K-step ks of the split into the ring slot of K-step kb
  auto issue = [&](int kb, int ks) {
    char* dst = smem + (kb % NS) * STAGE + wave * CPW * 1024;
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const bf16_t* p = is_a[i] ? src[i] + (size_t)(ks >> 1) * a_kstep + (ks & 1) * 512
                                : src[i] + (size_t)ks * BK;
      __builtin_amdgcn_global_load_lds((const void*)p,
                                       (__attribute__((address_space(3))) void*)(dst + i * 1024),
                                       16, 0, 0);
    }
  };
  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // the ring runs NS - 1 K-steps ahead; K-steps past the last one reload the
  // last (never read), which keeps the count of copies in flight uniform
#pragma unroll
  for (int s = 0; s < NS - 1; ++s) issue(s, min(s, last));
  wait_vmcnt<CPW * (NS - 2)>();
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    // slot (kt + NS - 1) % NS was last read in step kt - 1, before the last barrier
    issue(kt + NS - 1, min(kt + NS - 1, last));
    const char* stg = smem + (kt % NS) * STAGE;
    bf16x8_t af[NA][FM], wf[FN];
#pragma unroll
    for (int p = 0; p < NA; ++p)
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[p][i] = *(const bf16x8_t*)(stg + (p * GB + FM * wm + i) * 1024 + lane * 16);
#pragma unroll
    for (int j = 0; j < FN; ++j)
      wf[j] = *(const bf16x8_t*)(stg + (A_BLOCKS + FN * wn + j) * 1024 + lane * 16);
#pragma unroll
    for (int p = 0; p < NA; ++p)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[p][i], wf[j], acc[i][j], 0, 0, 0);
    // this wave's blocks of step kt + 1 (copies retire in issue order; the
    // NS - 2 younger stages stay in flight), then all blocks visible and slot
    // kt free.  A plain barrier: a fenced one would wait for every copy.
    wait_vmcnt<CPW * (NS - 2)>();
    asm volatile("s_barrier" ::: "memory");
  }
  wait_vmcnt<0>();                                 // the ring is reused by the epilogue
  __syncthreads();
  // acc[i][j][r] = C[RW wm + 16 i + 4 (lane / 16) + r][CW wn + 16 j + lane % 16]
  float* Cs = (float*)smem;
#pragma unroll
  for (int h = 0; h < BM / EB; ++h) {
    if ((RW * wm) / EB == h) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            Cs[(RW * wm - h * EB + 16 * i + 4 * (lane >> 4) + r) * CS + CW * wn + 16 * j + (lane & 15)] =
                acc[i][j][r];
    }
    __syncthreads();
    tile_epilogue<EB, BN, CS>(pol, Cs, m0 + h * EB, M, t, part, split, ldp);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// float32 kernel (fp32 mode): 32x32 tiles, BK = 32, 256 threads, 4 outputs each
// ---------------------------------------------------------------------------
template <class Pol>
__global__ void __launch_bounds__(256) gemm_f32_kernel(Pol pol, const float* __restrict__ A, int lda,
                                                       int M, int k_per_split,
                                                       float* __restrict__ part, int ldp) {
  constexpr int BM = 32, BN = 32, BK = 32, CS = BN + 1;
  __shared__ float As[BK][BM + 1];
  __shared__ float Bs[BK][BN + 1];
  __shared__ float Cs[BM * CS];
  const int tid = threadIdx.x;
  const int t = blockIdx.x, m0 = blockIdx.y * BM, split = blockIdx.z;
  const int kbeg = split * k_per_split;
  const float *blo, *bhi;
  pol.b_ptrs(t, BN, blo, bhi);
  const int tr = tid / 8, tc = (tid % 8) * 4;   // output row, first of 4 columns
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = kbeg; k0 < kbeg + k_per_split; k0 += BK) {
    for (int idx = tid; idx < BM * BK; idx += 256) {
      const int r = idx / BK, kk = idx % BK;
      As[kk][r] = A[(size_t)min(m0 + r, M - 1) * lda + k0 + kk];
      const float* rp = r < BN / 2 ? blo + (size_t)r * pol.ldb : bhi + (size_t)(r - BN / 2) * pol.ldb;
      Bs[kk][r] = rp[k0 + kk];
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < BK; ++kk) {
      const float a = As[kk][tr];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = fmaf(a, Bs[kk][tc + j], acc[j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) Cs[tr * CS + tc + j] = acc[j];
  __syncthreads();
  tile_epilogue<BM, BN, CS>(pol, Cs, m0, M, t, part, split, ldp);
}

// ---------------------------------------------------------------------------
// split-K reduction: sums partial tiles in split order, then the epilogue
// ---------------------------------------------------------------------------
// Sum of the split-K partials of 8 consecutive columns, in split order.  SC
// is the split count when known at compile time (all loads in flight before
// the sum), 0 for a runtime count.
template <int SC>
__device__ __forceinline__ void sum_partials8(const float* __restrict__ p, size_t stride, int S,
                                              float (&acc)[8]) {
  if constexpr (SC > 0) {
    float4 v[SC][2];
#pragma unroll
    for (int s = 0; s < SC; ++s) {
      v[s][0] = *(const float4*)(p + s * stride);
      v[s][1] = *(const float4*)(p + s * stride + 4);
    }
#pragma unroll
    for (int s = 0; s < SC; ++s) {
      acc[0] += v[s][0].x; acc[1] += v[s][0].y; acc[2] += v[s][0].z; acc[3] += v[s][0].w;
      acc[4] += v[s][1].x; acc[5] += v[s][1].y; acc[6] += v[s][1].z; acc[7] += v[s][1].w;
    }
  } else {
    for (int s = 0; s < S; ++s) {
      const float4 a = *(const float4*)(p + s * stride), b = *(const float4*)(p + s * stride + 4);
      acc[0] += a.x; acc[1] += a.y; acc[2] += a.z; acc[3] += a.w;
      acc[4] += b.x; acc[5] += b.y; acc[6] += b.z; acc[7] += b.w;
    }
  }
}

template <int BN, class Pol, int SC>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(Pol pol, const float* __restrict__ part,
                                                            int ldp, int M, int S, int ntiles) {
  // one thread per 8 consecutive output columns (of each half, when paired)
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  constexpr int C8 = Pol::PAIRED ? BN / 16 : BN / 8;
  const size_t per_row = (size_t)ntiles * C8;
  if (idx >= (size_t)M * per_row) return;
  const int m = idx / per_row, rem = idx % per_row;
  const int t = rem / C8, c0 = (rem % C8) * 8;
  float lo[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float hi[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const float* p = part + (size_t)m * ldp + (size_t)t * BN + c0;
  sum_partials8<SC>(p, (size_t)M * ldp, S, lo);
  if constexpr (Pol::PAIRED) sum_partials8<SC>(p + BN / 2, (size_t)M * ldp, S, hi);
  if constexpr (Pol::PAIRED) pol.store8(m, t, c0, BN, lo, hi);
  else pol.store8_1(m, t * BN + c0, lo);
}

template <int BN, class Pol>
static void launch_reduce(const Pol& pol, const float* part, int N, int M, int S, int ntiles,
                          hipStream_t st) {
  const size_t total = (size_t)M * N / 8 / (Pol::PAIRED ? 2 : 1);
  const dim3 grid((unsigned)((total + 255) / 256)), block(256);
  if (S == 8) launch((splitk_reduce_kernel<BN, Pol, 8>), grid, block, 0, st, pol, part, N, M, S, ntiles);
  else if (S == 4) launch((splitk_reduce_kernel<BN, Pol, 4>), grid, block, 0, st, pol, part, N, M, S, ntiles);
  else if (S == 2) launch((splitk_reduce_kernel<BN, Pol, 2>), grid, block, 0, st, pol, part, N, M, S, ntiles);
  else launch((splitk_reduce_kernel<BN, Pol, 0>), grid, block, 0, st, pol, part, N, M, S, ntiles);
}

// ---------------------------------------------------------------------------
// host-side dispatch
// ---------------------------------------------------------------------------
// K-step rotation of the column tiles (tile t starts at K-step t * krot mod
// nk); 0 = every tile starts at K-step 0.  Measured on the 120-row steps:
// 1 spreads the concurrently read weight addresses and takes 4% off the step.
// A tuning build (SSM_TUNING defined) lets SSM_GEMM_KROT override it; the
// product build reads no environment variable.
static int gemm_krot() {
#ifdef SSM_TUNING
  static const int krot = [] {
    const char* e = getenv("SSM_GEMM_KROT");
    return e ? atoi(e) : 1;
  }();
  return krot;
#else
  return 1;
#endif
}

// Split-K is only used while S * M stays small, which bounds the workspace.
static constexpr int SPLIT_ROWS_MAX = 1024;
// Row count from which the projections use gemm_big_kernel.
static constexpr int BIG_ROWS_MIN = 512;

size_t gemm_split_ws_floats(int M, int max_n) {
  (void)M;
  return (size_t)SPLIT_ROWS_MAX * max_n;
}

// Per-projection launch choice: tile width BN (64, 96 or 128), split-K S
// (0 = automatic) and the depth PW (4 or 8 K-steps) of the staging waves'
// register ring of weight loads.
struct GemmCfg {
  int bn, s, pw;
  int big = 0;
  int bm = 128;   // row tile of gemm_bf16_kernel (see launch_bf16_bm)    // gemm_big_kernel tile: 1 = 256 x 128, 2 = 128 x 256 (8 waves, 2-stage ring),
                  // 3 = 256 x 256 (16 waves, 3-stage ring), 4 = 128 x 256 (8 waves, 3-stage
                  // ring), 5 = 256 x 256 (8 waves of 64 x 128, 3-stage ring), 6 = 256 x 128
                  // (8 waves, 3-stage ring); 0 = gemm_bf16_kernel; -1 = automatic
};
static int big_rows(int big) { return big == 1 || big == 3 || big == 5 || big == 6 ? 256 : 128; }
static int big_cols(int big) { return big == 1 || big == 6 ? 128 : 256; }

// Tuning override, compiled only into a tuning build (SSM_TUNING defined):
// SSM_GEMM_CFG="kind:bn:s:pw[:big[:bm]],..." with kind one of qkv, o, gate_up,
// down, lm (big and bm as in GemmCfg); read once per process.  The product build
// always takes the measured defaults.
static GemmCfg cfg_override(const char* kind, GemmCfg c) {
#ifdef SSM_TUNING
  static const char* env = getenv("SSM_GEMM_CFG");
  if (!env) return c;
  const size_t kl = strlen(kind);
  for (const char* p = env; p && *p;) {
    if (strncmp(p, kind, kl) == 0 && p[kl] == ':') {
      int bn, s, pw, big = -1, bm = 128;
      const int n = sscanf(p + kl + 1, "%d:%d:%d:%d:%d", &bn, &s, &pw, &big, &bm);
      if (n >= 3) return GemmCfg{bn, s, pw, n >= 4 ? big : c.big, n == 5 ? bm : c.bm};
    }
    p = strchr(p, ',');
    if (p) ++p;
  }
  return c;
#else
  (void)kind;
  return c;
#endif
}

static int auto_split(int tiles, int M, int K, size_t ws_floats, int N) {
  int S = 1;
  while (S < 8 && tiles * S < 192 && K % (256 * S * 2) == 0 && (S * 2) * M <= SPLIT_ROWS_MAX &&
         (size_t)(S * 2) * M * N <= ws_floats)
    S *= 2;
  return S;
}

// Split-K of the big tiles: the S in 1..4 (K a multiple of 256 S, partials
// within the workspace) whose workgroups fill the CUs best over the rounds
// they take; 2% of fill per extra split pays for the partials' traffic.
// The 8-wave tiles with a 2-stage ring fit two workgroups per CU.
static int big_split(int tiles, int big, int M, int K, int N, size_t ws_floats) {
  const int slots = 256 * (big == 1 || big == 2 ? 2 : 1);
  int best = 1;
  double best_score = -1.0;
  for (int S = 1; S <= 4; ++S) {
    if (K % (256 * S) != 0 || (size_t)S * M * N > ws_floats) continue;
    const long wgs = (long)tiles * S;
    const double fill = (double)wgs / ((double)slots * ceil_div((int)wgs, slots));
    const double score = fill - 0.02 * (S - 1);
    if (score > best_score + 1e-9) { best_score = score; best = S; }
  }
  return best;
}

template <int BM, int BN, int PW, bool SPLIT, class Pol>
static hipError_t launch_bf16(const Pol& pol, const ActIn& a, int M, int K, int N, int S,
                              SplitWs ws, hipStream_t st, bool reduce) {
  const int ntiles = N / BN, mt = ceil_div(M, BM);
  const dim3 grid(ntiles * mt * S);
  launch((gemm_bf16_kernel<BM, BN, PW, SPLIT, Pol>), grid, dim3(512), 0, st, pol,
                     (const bf16_t*)a.hi, a.lo, a.G, M, K / S, mt, S,
                     S > 1 ? ws.part : nullptr, N, gemm_krot());
  if constexpr (!has_tile<Pol>::value) {   // whole-tile epilogues never split K
    if (S > 1 && reduce) launch_reduce<BN>(pol, ws.part, N, M, S, ntiles, st);
  }
  return hipGetLastError();
}

template <int BM, int BN, class Pol>
static hipError_t launch_bf16_pw(const Pol& pol, const ActIn& a, int M, int K, int N, int S,
                                 int pw, SplitWs ws, hipStream_t st, bool reduce) {
  const bool split = a.lo != nullptr;
  // the staging loop is unrolled by the ring depth: nk = K / S / 64 must be a
  // multiple of it (of 4 always, host-checked)
  if (pw >= 8 && (K / S / 64) % 8 == 0)
    return split ? launch_bf16<BM, BN, 8, true>(pol, a, M, K, N, S, ws, st, reduce)
                 : launch_bf16<BM, BN, 8, false>(pol, a, M, K, N, S, ws, st, reduce);
  return split ? launch_bf16<BM, BN, 4, true>(pol, a, M, K, N, S, ws, st, reduce)
               : launch_bf16<BM, BN, 4, false>(pol, a, M, K, N, S, ws, st, reduce);
}

// Row tile of gemm_bf16_kernel: 128 (default), 64 (two row tiles share each
// weight tile through L2 on small row counts), 192 or 256 (one-pass layers,
// tiles up to 96 columns: the register budget of a compute wave).
template <int BN, class Pol>
static hipError_t launch_bf16_bm(const Pol& pol, const ActIn& a, int M, int K, int N, int S,
                                 int pw, int bm, SplitWs ws, hipStream_t st, bool reduce) {
  if (bm == 64) return launch_bf16_pw<64, BN>(pol, a, M, K, N, S, pw, ws, st, reduce);
  if constexpr (BN <= 96) {
    if (bm == 192 && a.lo == nullptr) return launch_bf16_pw<192, BN>(pol, a, M, K, N, S, pw, ws, st, reduce);
    if (bm == 256 && a.lo == nullptr) return launch_bf16_pw<256, BN>(pol, a, M, K, N, S, pw, ws, st, reduce);
  }
  return launch_bf16_pw<128, BN>(pol, a, M, K, N, S, pw, ws, st, reduce);
}

// Launch plan of one projection: the configuration with a valid tile width
// and the split-K factor.
template <class Pol>
static GemmCfg plan_bf16(const char* kind, const Pol& pol, int M, int K, int N, GemmCfg c,
                         const SplitWs& ws, int (*bn_ok)(const Pol&, int)) {
  c = cfg_override(kind, c);
  // many rows: the big-tile kernel where its shape constraints hold
  if (c.big < 0) c.big = 0;
  const int big_bn = c.big ? big_cols(c.big) : 128;
  if (c.big && (M < BIG_ROWS_MIN || has_tile<Pol>::value || !bn_ok(pol, big_bn) ||
                N % big_bn != 0 || K % 32 != 0))
    c.big = 0;
  if (c.big) c.bn = big_bn;
  else if (c.bn > 128 || !bn_ok(pol, c.bn) || N % c.bn) c.bn = bn_ok(pol, 128) && N % 128 == 0 ? 128 : 64;
  if (c.big || (c.bm != 64 && c.bm != 192 && c.bm != 256) || ((c.bm == 192 || c.bm == 256) && c.bn > 96))
    c.bm = 128;
  const int tiles = (N / c.bn) * ceil_div(M, c.big ? big_rows(c.big) : c.bm);
  int S = c.s > 0 ? c.s : c.big ? big_split(tiles, c.big, M, K, N, ws.floats)
                                 : auto_split(tiles, M, K, ws.floats, N);
  while (S > 1 && (K % (256 * S) != 0 || (size_t)S * M * N > ws.floats)) S /= 2;
  c.s = S;
  return c;
}

template <int BM, int BN, int WM, int WN, int NS, class Pol>
static hipError_t launch_big(const Pol& pol, const ActIn& a, int M, int K, int N, int S,
                             SplitWs ws, hipStream_t st, bool reduce) {
  if constexpr (has_tile<Pol>::value) {
    return hipErrorInvalidValue;   // whole-tile epilogues run on gemm_bf16_kernel only
  } else {
    const int ntiles = N / BN, mt = ceil_div(M, BM);
    const dim3 grid(ntiles * mt * S), block(64 * WM * WN);
    float* pp = S > 1 ? ws.part : nullptr;
    if (a.lo)
      launch((gemm_big_kernel<BM, BN, WM, WN, NS, true, Pol>), grid, block, 0, st, pol,
             (const bf16_t*)a.hi, a.lo, a.G, M, K / S, mt, S, pp, N);
    else
      launch((gemm_big_kernel<BM, BN, WM, WN, NS, false, Pol>), grid, block, 0, st, pol,
             (const bf16_t*)a.hi, a.lo, a.G, M, K / S, mt, S, pp, N);
    if (S > 1 && reduce) launch_reduce<BN>(pol, ws.part, N, M, S, ntiles, st);
    return hipGetLastError();
  }
}

template <class Pol>
static hipError_t launch_plan(const Pol& pol, const ActIn& a, int M, int K, int N, GemmCfg c,
                              SplitWs ws, hipStream_t st, bool reduce = true) {
  if (c.big == 1) return launch_big<256, 128, 4, 2, 2>(pol, a, M, K, N, c.s, ws, st, reduce);
  if (c.big == 2) return launch_big<128, 256, 2, 4, 2>(pol, a, M, K, N, c.s, ws, st, reduce);
  if (c.big == 3) return launch_big<256, 256, 4, 4, 3>(pol, a, M, K, N, c.s, ws, st, reduce);
  if (c.big == 4) return launch_big<128, 256, 2, 4, 3>(pol, a, M, K, N, c.s, ws, st, reduce);
  if (c.big == 5) return launch_big<256, 256, 4, 2, 3>(pol, a, M, K, N, c.s, ws, st, reduce);
  if (c.big == 6) return launch_big<256, 128, 4, 2, 3>(pol, a, M, K, N, c.s, ws, st, reduce);
  if (c.bn == 96) return launch_bf16_bm<96>(pol, a, M, K, N, c.s, c.pw, c.bm, ws, st, reduce);
  if (c.bn == 64) return launch_bf16_bm<64>(pol, a, M, K, N, c.s, c.pw, c.bm, ws, st, reduce);
  return launch_bf16_bm<128>(pol, a, M, K, N, c.s, c.pw, c.bm, ws, st, reduce);
}

template <class Pol>
static hipError_t run_bf16(const char* kind, Pol pol, const ActIn& a, int M, int K, int N,
                           GemmCfg c, SplitWs ws, hipStream_t st, int (*bn_ok)(const Pol&, int)) {
  c = plan_bf16(kind, pol, M, K, N, c, ws, bn_ok);
  return launch_plan(pol, a, M, K, N, c, ws, st);
}

// Completion of a split-K residual projection fused with the RMSNorm that
// follows it: resid[m] += sum over splits of part[s][m] (split order, as the
// split-K reduction does), then y[m] = resid[m] / rms(resid[m]) * g as the next
// projection's operand.  One workgroup of 512 threads per row; thread t holds
// the 8-column chunks t + 512 q of the row (q < NC).
template <int SC, int NC>
__global__ void __launch_bounds__(512) resid_norm_kernel(const float* __restrict__ part, int S,
                                                         int M, int N, float* __restrict__ resid,
                                                         const bf16_t* __restrict__ g, float eps,
                                                         ActOut y) {
  __shared__ float red[8];
  const int m = blockIdx.x, tid = threadIdx.x, nc8 = N >> 3;
  float v[NC][8];
  float ss = 0.f;
#pragma unroll
  for (int q = 0; q < NC; ++q) {
    const int c8 = tid + 512 * q;
    if (c8 >= nc8) continue;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    sum_partials8<SC>(part + (size_t)m * N + c8 * 8, (size_t)M * N, S, acc);
    float4* r = (float4*)(resid + (size_t)m * N + c8 * 8);
    float4 r0 = r[0], r1 = r[1];
    r0.x += acc[0]; r0.y += acc[1]; r0.z += acc[2]; r0.w += acc[3];
    r1.x += acc[4]; r1.y += acc[5]; r1.z += acc[6]; r1.w += acc[7];
    r[0] = r0;
    r[1] = r1;
    v[q][0] = r0.x; v[q][1] = r0.y; v[q][2] = r0.z; v[q][3] = r0.w;
    v[q][4] = r1.x; v[q][5] = r1.y; v[q][6] = r1.z; v[q][7] = r1.w;
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[q][e] * v[q][e];
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  ss = ((red[0] + red[1]) + (red[2] + red[3])) + ((red[4] + red[5]) + (red[6] + red[7]));
  const float inv = 1.0f / sqrtf(ss / (float)N + eps);
#pragma unroll
  for (int q = 0; q < NC; ++q) {
    const int c8 = tid + 512 * q;
    if (c8 >= nc8) continue;
    const u32x4_t gw = *(const u32x4_t*)(g + c8 * 8);
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t w = gw[e >> 1];
      const float ge = __uint_as_float(e & 1 ? (w & 0xffff0000u) : (w << 16));
      o[e] = v[q][e] * inv * ge;
    }
    y.store8<bf16_t>(m, c8 * 8, o);
  }
}

template <int SC>
static void launch_resid_norm(int nc, int S, int M, int N, const float* part, float* resid,
                              const NormTo* nrm, hipStream_t st) {
  const bf16_t* g = (const bf16_t*)nrm->g;
  if (nc == 1)
    launch(resid_norm_kernel<SC, 1>, dim3(M), dim3(512), 0, st, part, S, M, N, resid, g, nrm->eps, nrm->y);
  else
    launch(resid_norm_kernel<SC, 2>, dim3(M), dim3(512), 0, st, part, S, M, N, resid, g, nrm->eps, nrm->y);
}

template <class Pol>
static hipError_t run_f32(const Pol& pol, const ActIn& a, int M, int K, int N, SplitWs ws,
                          hipStream_t st) {
  constexpr int BN = 32;
  const int ntiles = N / BN, mt = ceil_div(M, 32);
  int S = 1;
  while (S < 8 && ntiles * mt * S < 256 && K % (32 * S * 2) == 0 && (S * 2) * M <= SPLIT_ROWS_MAX &&
         (size_t)(S * 2) * M * N <= ws.floats)
    S *= 2;
  dim3 grid(ntiles, mt, S);
  launch((gemm_f32_kernel<Pol>), grid, dim3(256), 0, st, pol, (const float*)a.hi,
                     a.ld, M, K / S, S > 1 ? ws.part : nullptr, N);
  if (S > 1) launch_reduce<BN>(pol, ws.part, N, M, S, ntiles, st);
  return hipGetLastError();
}

// Default launch choices: the cached-step row counts (M <= 256) are
// HBM-bound and want every CU streaming weights; block-start row counts are
// MFMA-bound and want wide tiles.  `paired`: the activations carry the lo part
// (twice the MFMA work per operand byte, so the wide 3-stage tiles pay more).
// Measured choices:
//  * row tiles of gemm_bf16_kernel: 128 rows, except 256 for the one-pass QKV
//    from 257 to 511 rows (two row tiles instead of three or four) and the
//    one-pass gate/up from 129 to 256 rows (one row tile instead of two); 64-
//    and 192-row tiles and the 256-row tiles elsewhere measured slower;
//  * QKV: 96-column tiles below 512 rows (128 column tiles at d = 4096 with
//    32 + 2 x 32 heads: with the automatic split-K, 2 ways up to 128 rows,
//    256 workgroups where 128-column tiles left 64 CUs idle); 256 x 128 tiles
//    from 512 rows with the pair (2-stage ring) and from 1024 rows in one pass
//    (3-stage ring, 24 KB per stage: two workgroups per CU; below 1024 rows
//    its 256-row tiles leave slots empty).  256-column tiles (two heads) took
//    longer at 1776 rows: 336 tiles leave most of a second round empty;
//  * gate/up: 96-column tiles below 512 rows (one workgroup per CU at
//    2F = 24576; the planner falls back to 128 where 96 does not divide 2F);
//    from 512 rows 128 x 256 with the pair and the 3-stage 256 x 128 tiles
//    in one pass, from 1024 rows 256 x 256 with 16 waves and a 3-stage ring
//    (half the operand bytes per MFMA, two K-steps of copy latency hidden);
//  * O / down (N = d): gemm_bf16_kernel, whose 128-row tiles fill more CUs;
//    from 1024 rows the 256 x 256 tiles with split-K chosen for CU fill
//    (big_split; its partials go through the fused sum + RMSNorm).  Up to
//    128 rows O takes 64-column tiles and split-K 4, which halves the float32
//    partials of the 8-way split.
static GemmCfg default_cfg(const char* kind, int M, bool paired) {
  const bool small = M <= 256;
  if (!strcmp(kind, "qkv")) {
    if (M < 512) {
      GemmCfg c{96, 0, 4, 0};
      if (!paired && M > 256) c.bm = 256;   // two 256-row tiles: 7-17% faster at 376-504 rows
      return c;
    }
    return GemmCfg{128, 1, 3, paired ? 1 : (M >= 1024 ? 6 : 0)};
  }
  if (!strcmp(kind, "gate_up")) {
    if (M < 512) {
      GemmCfg c{96, 1, 4, 0};
      if (!paired && M > 128 && M <= 256) c.bm = 256;   // one row tile: 9% faster at 240 rows
      return c;
    }
    return GemmCfg{128, 1, 3, M >= 1024 ? 3 : (paired ? 2 : 6)};
  }
  if (!strcmp(kind, "lm")) return GemmCfg{128, 1, 4, 0};
  if (!strcmp(kind, "o") && M <= 128) return GemmCfg{64, 4, 4, 0};
  return small ? GemmCfg{128, 0, 4, 0} : GemmCfg{128, 0, 3, M >= 1024 ? 3 : 0};
}

// tile widths: 64, 96 and 128 (gemm_bf16_kernel), 128 and 256 (gemm_big_kernel)
template <class Pol> static int any_bn(const Pol&, int bn) { return bn == 64 || bn == 96 || bn == 128 || bn == 256; }
// any width whose tiles divide the heads' concatenated halves (the epilogue's
// 8-column groups then never straddle a head)
static int qkv_bn(const PolQKV<bf16_t, f16_t>& p, int bn) {
  return (bn == 64 || bn == 96 || bn == 128 || bn == 256) && ((p.H + 2 * p.Hkv) * p.dh) % bn == 0 &&
         (p.dh / 2) % 8 == 0;
}

hipError_t gemm_qkv(int dtype, const ActIn& a, int M, int d, const void* wq, const void* wk,
                    const void* wv, int H, int Hkv, int dh, const QKVOut& o, SplitWs ws,
                    hipStream_t st) {
  const int N = (H + 2 * Hkv) * dh;
  if (dtype == 0) {
    PolQKV<float> p{(const float*)wq, (const float*)wk, (const float*)wv, d, H, Hkv, dh,
                    (float*)o.q, (float*)o.kc, (float*)o.vc, o.cap, o.n_cached, o.n_rows, o.rope,
                    o.rope_per_seq};
    return run_f32(p, a, M, d, N, ws, st);
  }
  PolQKV<bf16_t, f16_t> p{(const bf16_t*)wq, (const bf16_t*)wk, (const bf16_t*)wv, d, H, Hkv, dh,
                          (f16_t*)o.q, (f16_t*)o.kc, (f16_t*)o.vc, o.cap, o.n_cached,
                          o.n_rows, o.rope, o.rope_per_seq};
  return run_bf16("qkv", p, a, M, d, N, default_cfg("qkv", M, a.lo != nullptr), ws, st, qkv_bn);
}

hipError_t gemm_resid(int dtype, const char* kind, const ActIn& a, int M, int K, const void* w,
                      int N, float* resid, SplitWs ws, hipStream_t st, const NormTo* nrm) {
  hipError_t e;
  if (dtype == 0) {
    PolResid<float> p{(const float*)w, K, N, resid};
    e = run_f32(p, a, M, K, N, ws, st);
  } else {
    PolResid<bf16_t> p{(const bf16_t*)w, K, N, resid};
    const GemmCfg c = plan_bf16(kind, p, M, K, N, default_cfg(kind, M, a.lo != nullptr), ws,
                                any_bn<PolResid<bf16_t>>);
    const int nc = ceil_div(N / 8, 512);
    const bool fuse = nrm && c.s > 1 && N % 8 == 0 && nc <= 2 && ((uintptr_t)nrm->g & 15) == 0;
    e = launch_plan(p, a, M, K, N, c, ws, st, !fuse);
    if (e != hipSuccess || !fuse) goto separate;
    if (c.s == 8) launch_resid_norm<8>(nc, c.s, M, N, ws.part, resid, nrm, st);
    else if (c.s == 4) launch_resid_norm<4>(nc, c.s, M, N, ws.part, resid, nrm, st);
    else if (c.s == 2) launch_resid_norm<2>(nc, c.s, M, N, ws.part, resid, nrm, st);
    else launch_resid_norm<0>(nc, c.s, M, N, ws.part, resid, nrm, st);
    return hipGetLastError();
  }
separate:
  if (e != hipSuccess || !nrm) return e;
  return launch_norm(dtype, resid, N, nrm->g, nrm->eps, nrm->y, M, M, 0, 0, st);
}

hipError_t gemm_swiglu(int dtype, const ActIn& a, int M, int d, const void* wg, const void* wu,
                       int F, const ActOut& act, SplitWs ws, hipStream_t st) {
  if (dtype == 0) {
    PolSwiGLU<float> p{(const float*)wg, (const float*)wu, d, F, act};
    return run_f32(p, a, M, d, 2 * F, ws, st);
  }
  PolSwiGLU<bf16_t> p{(const bf16_t*)wg, (const bf16_t*)wu, d, F, act};
  return run_bf16("gate_up", p, a, M, d, 2 * F, default_cfg("gate_up", M, a.lo != nullptr), ws, st,
                  any_bn<PolSwiGLU<bf16_t>>);
}

hipError_t gemm_store_f32(const ActIn& a, int M, int K, const void* w, int N, float* c, int ldc,
                          SplitWs ws, hipStream_t st) {
  PolStore<float> p{(const float*)w, K, ldc, c};
  return run_f32(p, a, M, K, N, ws, st);
}

// Merges the partial statistics of one row (one workgroup per row), in a
// fixed order: deterministic.
__global__ void __launch_bounds__(256) lm_merge_kernel(const LMPartial* __restrict__ part,
                                                       int n_part, int k,
                                                       int32_t* __restrict__ argmax,
                                                       float* __restrict__ conf,
                                                       int32_t* __restrict__ topk_ids,
                                                       float* __restrict__ topk_w) {
  __shared__ float s_m[4];
  __shared__ float s_s[4];
  __shared__ float s_v[4];
  __shared__ int s_i[4];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const LMPartial* P = part + (size_t)row * n_part;
  float tv[8];
  int ti[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) { tv[q] = -INFINITY; ti[q] = 0x7fffffff; }
  float mx = -INFINITY, sm = 0.f;
  // this thread's partials j = tid + 256 i, in that order; CH of them are
  // loaded before any is folded in, so a row costs a few round trips
  constexpr int CH = 4;
  for (int j0 = tid; j0 < n_part; j0 += 256 * CH) {
    LMPartial buf[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c)
      if (j0 + 256 * c < n_part) buf[c] = P[j0 + 256 * c];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if (j0 + 256 * c >= n_part) break;
      const LMPartial& p = buf[c];
      if (p.s > 0.f) {
        if (p.m > mx) { sm = sm * expf(mx - p.m) + p.s; mx = p.m; }
        else sm += p.s * expf(p.m - mx);
      }
      // a partial's values are sorted best first: stop at the first one that
      // does not enter this thread's list
      for (int q = 0; q < 8; ++q) {
        if (!stat_better(p.v[q], p.id[q], tv[7], ti[7])) break;
        stat_insert(tv, ti, p.v[q], p.id[q]);
      }
    }
  }
  // (max, sum) pairs over the workgroup: a butterfly within each wave (both
  // partners compute the same sum, in either order), then the 4 waves in order
  auto combine = [](float& m, float& s, float om, float os) {
    if (!(os > 0.f)) return;
    if (!(s > 0.f)) { m = om; s = os; return; }
    const float M = fmaxf(m, om);
    s = s * expf(m - M) + os * expf(om - M);
    m = M;
  };
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float om = __shfl_xor(mx, o, 64), os = __shfl_xor(sm, o, 64);
    combine(mx, sm, om, os);
  }
  if (lane == 0) { s_m[wave] = mx; s_s[wave] = sm; }
  __syncthreads();
  float M = s_m[0], S = s_s[0];
  for (int w = 1; w < 4; ++w) combine(M, S, s_m[w], s_s[w]);
  float best_v[8];
  int best_i[8];
  for (int q = 0; q < 8; ++q) {
    float v = tv[0];
    int i = ti[0];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(v, o, 64);
      const int oi = __shfl_xor(i, o, 64);
      if (stat_better(ov, oi, v, i)) { v = ov; i = oi; }
    }
    __syncthreads();
    if (lane == 0) { s_v[wave] = v; s_i[wave] = i; }
    __syncthreads();
    v = s_v[0];
    i = s_i[0];
    for (int w = 1; w < 4; ++w)
      if (stat_better(s_v[w], s_i[w], v, i)) { v = s_v[w]; i = s_i[w]; }
    best_v[q] = v;
    best_i[q] = i;
    if (ti[0] == i && tv[0] == v) {   // the owner pops its head (ids are unique)
#pragma unroll
      for (int t = 0; t < 7; ++t) { tv[t] = tv[t + 1]; ti[t] = ti[t + 1]; }
      tv[7] = -INFINITY;
      ti[7] = 0x7fffffff;
    }
  }
  if (tid == 0) {
    argmax[row] = best_i[0];
    conf[row] = 1.0f / S;   // exp(max - max) / sum exp(x - max)
    float z = 0.f;
    for (int q = 0; q < 8; ++q)
      if (q < k) z += expf(best_v[q] - best_v[0]);
    for (int q = 0; q < 8; ++q)
      if (q < k) {
        topk_ids[(size_t)row * k + q] = best_i[q];
        topk_w[(size_t)row * k + q] = expf(best_v[q] - best_v[0]) / z;
      }
  }
}

size_t lm_stats_ws_bytes(int M, int N) { return (size_t)M * (2 * (N / 128)) * sizeof(LMPartial); }

hipError_t lm_head_stats(const ActIn& a, int M, int K, const void* w, int N, int mask_id, int k,
                         void* stats_ws, float* logits, int32_t* argmax, float* conf,
                         int32_t* topk_ids, float* topk_w, hipStream_t st) {
  constexpr int BN = 128;
  const int ntiles = N / BN;
  PolLMStats<bf16_t> p{(const bf16_t*)w, K, N, mask_id, (LMPartial*)stats_ws, 2 * ntiles, logits, N};
  const GemmCfg c = cfg_override("lm", default_cfg("lm", M, a.lo != nullptr));
  SplitWs none{nullptr, 0};
  hipError_t e = launch_bf16_pw<128, BN>(p, a, M, K, N, 1, c.pw, none, st, true);
  if (e != hipSuccess) return e;
  launch(lm_merge_kernel, dim3(M), dim3(256), 0, st, (const LMPartial*)stats_ws,
                     2 * ntiles, k, argmax, conf, topk_ids, topk_w);
  return hipGetLastError();
}

}  // namespace ssm
