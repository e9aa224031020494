// Projections of the decoder layer: C = A * W^T with A [M, K] float32
// activations and W [N, K] row-major weights (nn.Linear layout).
//
// A is read as float32 and optionally scaled on the way in: a per-row scale
// (the RMSNorm factor 1/rms of that row) and a per-column scale (the norm
// weight), so the normalisation of the decoder block is fused into the
// projection that consumes it.  Logical row m of A is physical row
// (m / per) * stride + off + m % per, which lets the LM head read only the
// output rows of every sequence.
//
// bfloat16 path: MFMA v_mfma_f32_16x16x32_bf16, 256 threads (4 waves) per
// workgroup, BK = 64, fp32 accumulation.  Weights stream through a ring of
// register stages PW K-steps ahead (HBM latency), activations PA K-steps
// ahead (L2 latency); both are staged through a double-buffered LDS tile
// with padded rows.  With SPLIT the scaled activation is stored as two
// bfloat16 parts hi = bf16(v), lo = bf16(v - hi) and each product is taken
// twice (hi*W + lo*W): the weights are exact in bfloat16, so the result
// then carries about 16 significant bits of the activation instead of 8.
// The output tile is staged through LDS so that the epilogue can combine any
// two columns of the tile and store coalesced.
//
// Every output tile of BN columns reads its first BN/2 weight rows from one
// base pointer and its last BN/2 from another.  That is how the fused
// epilogues get the pairs they need without any weight repacking:
//   QKV    : columns (c, c + dh/2) of one head -> rotate-half RoPE, then the
//            query buffer or the KV cache slot of the row;
//   SwiGLU : gate row j and up row j -> silu(g) * u;
//   resid  : plain rows -> residual stream += value;
//   store  : plain rows -> float32 output (LM head logits).
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
template <typename T>
struct PolQKV {
  static constexpr bool PAIRED = true;
  const T *wq, *wk, *wv;
  int ldb, H, Hkv, dh, tiles_per_head;
  T *q, *kc, *vc;
  int cap, n_cached, n_rows;
  const float2* rope;

  __device__ __forceinline__ void b_ptrs(int t, int BN, const T*& lo, const T*& hi) const {
    const int head = t / tiles_per_head, sub = t % tiles_per_head;
    const T* base;
    int hh;
    if (head < H) { base = wq; hh = head; }
    else if (head < H + Hkv) { base = wk; hh = head - H; }
    else { base = wv; hh = head - H - Hkv; }
    lo = base + (size_t)(hh * dh + sub * (BN / 2)) * ldb;
    hi = lo + (size_t)(dh / 2) * ldb;
  }
  __device__ __forceinline__ void store(int m, int t, int c, int BN, float vlo, float vhi) const {
    const int head = t / tiles_per_head, sub = t % tiles_per_head;
    const int i = sub * (BN / 2) + c;
    const int s = m / n_rows, row = m % n_rows;
    if (head < H + Hkv) {
      const float2 cs = rope[(size_t)row * (dh / 2) + i];
      const float a = vlo * cs.x - vhi * cs.y;
      const float b = vhi * cs.x + vlo * cs.y;
      vlo = a;
      vhi = b;
    }
    T* dst;
    if (head < H) dst = q + (((size_t)s * H + head) * n_rows + row) * dh;
    else if (head < H + Hkv) dst = kc + (((size_t)s * Hkv + (head - H)) * cap + n_cached + row) * dh;
    else dst = vc + (((size_t)s * Hkv + (head - H - Hkv)) * cap + n_cached + row) * dh;
    stf(dst + i, vlo);
    stf(dst + i + dh / 2, vhi);
  }
};

template <typename T>
struct PolSwiGLU {
  static constexpr bool PAIRED = true;
  const T *wg, *wu;
  int ldb, F;
  float* act;
  __device__ __forceinline__ void b_ptrs(int t, int BN, const T*& lo, const T*& hi) const {
    lo = wg + (size_t)t * (BN / 2) * ldb;
    hi = wu + (size_t)t * (BN / 2) * ldb;
  }
  __device__ __forceinline__ void store(int m, int t, int c, int BN, float g, float u) const {
    const float silu = g / (1.0f + expf(-g));
    act[(size_t)m * F + t * (BN / 2) + c] = silu * u;
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
  __device__ __forceinline__ void store1(int, int, float) const {}
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

// Applies the epilogue to a BM x BN float tile staged in LDS (row stride CS).
template <int BM, int BN, int CS, class Pol>
__device__ __forceinline__ void tile_epilogue(const Pol& pol, const float* Cs, int m0, int M,
                                              int t, float* part, int split, int ldp) {
  const int tid = threadIdx.x;
  if constexpr (has_tile<Pol>::value) {
    pol.template tile<BM, BN, CS>(Cs, m0, M, t);
  } else if (part) {
    for (int idx = tid; idx < BM * BN; idx += blockDim.x) {
      const int r = idx / BN, c = idx % BN, gm = m0 + r;
      if (gm < M) part[((size_t)split * M + gm) * ldp + (size_t)t * BN + c] = Cs[r * CS + c];
    }
  } else if constexpr (Pol::PAIRED) {
    for (int idx = tid; idx < BM * (BN / 2); idx += blockDim.x) {
      const int r = idx / (BN / 2), c = idx % (BN / 2), gm = m0 + r;
      if (gm < M) pol.store(gm, t, c, BN, Cs[r * CS + c], Cs[r * CS + c + BN / 2]);
    }
  } else {
    for (int idx = tid; idx < BM * BN; idx += blockDim.x) {
      const int r = idx / BN, c = idx % BN, gm = m0 + r;
      if (gm < M) pol.store1(gm, t * BN + c, Cs[r * CS + c]);
    }
  }
}

// ---------------------------------------------------------------------------
// bfloat16 MFMA kernel
// ---------------------------------------------------------------------------
// Tile order: the grid is 1-D over (n-tile, m-tile) pairs.  Workgroups are
// dealt to the 8 XCDs round-robin by linear id, so id w runs on XCD w % 8;
// the order below gives each XCD a contiguous range of n-tiles with the
// m-tiles innermost, so the workgroups that share a weight tile run on the
// same XCD at about the same time and read it once into that XCD's L2.
__device__ __forceinline__ void tile_of(int w, int total, int mt, int& tn, int& tm) {
  const int per = total / 8;
  const int t = w < per * 8 ? (w % 8) * per + (w / 8) : w;
  tn = t / mt;
  tm = t % mt;
}

template <int BM, int BN, int WM, int WN, int PA, int PW, bool SPLIT, class Pol>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(Pol pol, GemmA ga, int M, int k_per_split,
                                                        int mt, float* __restrict__ part,
                                                        int ldp) {
  constexpr int BK = 64, LS = BK + 8;            // LDS row stride (elements), 144 B
  constexpr int NWN = BN / WN;
  static_assert((BM / WM) * NWN == 4, "4 waves");
  constexpr int FM = WM / 16, FN = WN / 16;
  constexpr int AR = BM / 32, BCH = BN / 32;     // rows per thread of the A and W tiles
  static_assert(BCH >= 2 && (BCH % 2) == 0, "BN must be a multiple of 64");
  static_assert(PA == 1 || PA == 2, "activation prefetch 1 or 2");
  static_assert(PW == 2 || PW == 4, "weight prefetch 2 or 4");
  constexpr int NA = SPLIT ? 2 : 1;
  constexpr int SMEM_AB = 2 * (NA * BM + BN) * LS * 2;
  constexpr int CS = BN + 4;
  constexpr int SMEM_C = BM * CS * 4;
  constexpr int SMEM = SMEM_AB > SMEM_C ? SMEM_AB : SMEM_C;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  bf16_t* Ah = (bf16_t*)smem;                    // [2][BM][LS]
  bf16_t* Al = Ah + 2 * BM * LS;                 // [2][BM][LS] (SPLIT only)
  bf16_t* Bs = Ah + 2 * NA * BM * LS;            // [2][BN][LS]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / NWN, wn = wave % NWN;
  int t, mtile;
  tile_of(blockIdx.x, gridDim.x, mt, t, mtile);
  const int m0 = mtile * BM, split = blockIdx.y;
  const int kbeg = split * k_per_split;
  const int nk = k_per_split / BK;

  const bf16_t *blo, *bhi;
  pol.b_ptrs(t, BN, blo, bhi);

  // thread -> (row r0 + 32 i, 8 columns at col) of every tile
  const int r0 = tid >> 3, col = (tid & 7) * 8;
  const float* a_row[AR];
  float a_scale[AR];
#pragma unroll
  for (int i = 0; i < AR; ++i) {
    const int m = min(m0 + r0 + 32 * i, M - 1);   // rows past M are computed and discarded
    const int pm = (m / ga.per) * ga.stride + ga.off + m % ga.per;
    a_row[i] = ga.a + (size_t)pm * ga.lda + kbeg + col;
    a_scale[i] = ga.rscale ? ga.rscale[m] : 1.0f;
  }
  const bf16_t* cs_ptr = ga.cscale ? (const bf16_t*)ga.cscale + kbeg + col : nullptr;
  const bf16_t* blo_k = blo + (size_t)r0 * pol.ldb + kbeg + col;
  const bf16_t* bhi_k = bhi + (size_t)r0 * pol.ldb + kbeg + col;
  const size_t bstride = (size_t)32 * pol.ldb;
  const int dst0 = r0 * LS + col;

  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // A stages: 2 x 16 bytes of float32 per row plus the 8 column scales
  u32x4_t ra0[AR][2], ra1[AR][2], rc0, rc1;
  // W stages: ring of PW register sets
  u32x4_t rw0[BCH], rw1[BCH], rw2[BCH], rw3[BCH];

#define LOAD_A(RA, RC, KT)                                                            \
  do {                                                                                \
    _Pragma("unroll") for (int i = 0; i < AR; ++i) {                                  \
      RA[i][0] = *(const u32x4_t*)(a_row[i] + (KT) * BK);                            \
      RA[i][1] = *(const u32x4_t*)(a_row[i] + (KT) * BK + 4);                        \
    }                                                                                 \
    if (cs_ptr) RC = *(const u32x4_t*)(cs_ptr + (KT) * BK);                           \
  } while (0)
#define LOAD_W(RW, KT)                                                                \
  do {                                                                                \
    _Pragma("unroll") for (int i = 0; i < BCH / 2; ++i) {                             \
      RW[i] = *(const u32x4_t*)(blo_k + i * bstride + (KT) * BK);                    \
      RW[i + BCH / 2] = *(const u32x4_t*)(bhi_k + i * bstride + (KT) * BK);          \
    }                                                                                 \
  } while (0)
#define STORE_A(RA, RC, BUF)                                                          \
  do {                                                                                \
    float cs_[8];                                                                     \
    {                                                                                 \
      const bf16x8_t cv_ = __builtin_bit_cast(bf16x8_t, RC);                         \
      _Pragma("unroll") for (int e = 0; e < 8; ++e) cs_[e] = cs_ptr ? (float)cv_[e] : 1.0f; \
    }                                                                                 \
    _Pragma("unroll") for (int i = 0; i < AR; ++i) {                                  \
      const f32x4_t v0_ = __builtin_bit_cast(f32x4_t, RA[i][0]);                     \
      const f32x4_t v1_ = __builtin_bit_cast(f32x4_t, RA[i][1]);                     \
      bf16x8_t hi_, lo_;                                                              \
      _Pragma("unroll") for (int e = 0; e < 8; ++e) {                                 \
        const float v_ = (e < 4 ? v0_[e & 3] : v1_[e & 3]) * a_scale[i] * cs_[e];    \
        hi_[e] = (__bf16)v_;                                                          \
        if (SPLIT) lo_[e] = (__bf16)(v_ - (float)hi_[e]);                             \
      }                                                                               \
      *(bf16x8_t*)(Ah + (BUF) * BM * LS + dst0 + i * 32 * LS) = hi_;                  \
      if (SPLIT) *(bf16x8_t*)(Al + (BUF) * BM * LS + dst0 + i * 32 * LS) = lo_;       \
    }                                                                                 \
  } while (0)
#define STORE_W(RW, BUF)                                                              \
  do {                                                                                \
    _Pragma("unroll") for (int i = 0; i < BCH; ++i)                                   \
        *(u32x4_t*)(Bs + (BUF) * BN * LS + dst0 + i * 32 * LS) = RW[i];               \
  } while (0)
#define COMPUTE(BUF)                                                                  \
  do {                                                                                \
    const int ao_ = (BUF) * BM * LS + (wm * WM + (lane & 15)) * LS + (lane >> 4) * 8; \
    const bf16_t* bs_ = Bs + (BUF) * BN * LS + (wn * WN + (lane & 15)) * LS + (lane >> 4) * 8; \
    _Pragma("unroll") for (int kk = 0; kk < 2; ++kk) {                                \
      bf16x8_t bfr[FN];                                                               \
      _Pragma("unroll") for (int j = 0; j < FN; ++j)                                  \
          bfr[j] = *(const bf16x8_t*)(bs_ + j * 16 * LS + kk * 32);                   \
      _Pragma("unroll") for (int i = 0; i < FM; ++i) {                                \
        const bf16x8_t ah_ = *(const bf16x8_t*)(Ah + ao_ + i * 16 * LS + kk * 32);    \
        _Pragma("unroll") for (int j = 0; j < FN; ++j)                                \
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah_, bfr[j], acc[i][j], 0, 0, 0); \
        if (SPLIT) {                                                                  \
          const bf16x8_t al_ = *(const bf16x8_t*)(Al + ao_ + i * 16 * LS + kk * 32);  \
          _Pragma("unroll") for (int j = 0; j < FN; ++j)                              \
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al_, bfr[j], acc[i][j], 0, 0, 0); \
        }                                                                             \
      }                                                                               \
    }                                                                                 \
  } while (0)
  // One K-step.  Stage kt is in LDS buffer kt & 1; stage kt + 1 arrives in
  // A set (kt + 1) % PA and W set RWN; the loads issued here are for stage
  // kt + 1 + PA (activations) and kt + 1 + PW (weights).
#define STEP(KT, RAN, RCN, RWN)                                                       \
  do {                                                                                \
    const int kt_ = (KT);                                                             \
    if (kt_ < nk) {                                                                   \
      COMPUTE(kt_ & 1);                                                               \
      if (kt_ + 1 < nk) {                                                         \
        STORE_A(RAN, RCN, (kt_ + 1) & 1);                                             \
        STORE_W(RWN, (kt_ + 1) & 1);                                                  \
        if (kt_ + 1 + PA < nk) LOAD_A(RAN, RCN, kt_ + 1 + PA);                        \
        if (kt_ + 1 + PW < nk) LOAD_W(RWN, kt_ + 1 + PW);                             \
      }                                                                               \
      __syncthreads();                                                                \
    }                                                                                 \
  } while (0)

  // prologue: stage 0 -> LDS buffer 0; stages 1.. in flight
  LOAD_A(ra0, rc0, 0);
  LOAD_W(rw0, 0);
  STORE_A(ra0, rc0, 0);
  STORE_W(rw0, 0);
  if (PA == 1) {
    if (1 < nk) LOAD_A(ra1, rc1, 1);
  } else {
    if (1 < nk) LOAD_A(ra1, rc1, 1);
    if (2 < nk) LOAD_A(ra0, rc0, 2);
  }
  if (1 < nk) LOAD_W(rw1, 1);
  if (2 < nk) LOAD_W(rw2, 2);
  if (PW == 4) {
    if (3 < nk) LOAD_W(rw3, 3);
    if (4 < nk) LOAD_W(rw0, 4);
  } else {
    // with PW == 2 stage 2 lives in set 0
    if (2 < nk) LOAD_W(rw0, 2);
  }
  __syncthreads();

  if constexpr (PW == 4) {
    for (int kt = 0; kt < nk; kt += 4) {
      if constexpr (PA == 1) {
        STEP(kt, ra1, rc1, rw1);
        STEP(kt + 1, ra1, rc1, rw2);
        STEP(kt + 2, ra1, rc1, rw3);
        STEP(kt + 3, ra1, rc1, rw0);
      } else {
        STEP(kt, ra1, rc1, rw1);
        STEP(kt + 1, ra0, rc0, rw2);
        STEP(kt + 2, ra1, rc1, rw3);
        STEP(kt + 3, ra0, rc0, rw0);
      }
    }
  } else {
    for (int kt = 0; kt < nk; kt += 2) {
      if constexpr (PA == 1) {
        STEP(kt, ra1, rc1, rw1);
        STEP(kt + 1, ra1, rc1, rw0);
      } else {
        STEP(kt, ra1, rc1, rw1);
        STEP(kt + 1, ra0, rc0, rw0);
      }
    }
  }
#undef LOAD_A
#undef LOAD_W
#undef STORE_A
#undef STORE_W
#undef COMPUTE
#undef STEP

  // accumulators -> LDS tile: acc[i][j][r] = C[16i + 4*(lane/16) + r][16j + lane%16]
  float* Cs = (float*)smem;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        Cs[(wm * WM + i * 16 + (lane >> 4) * 4 + r) * CS + wn * WN + j * 16 + (lane & 15)] =
            acc[i][j][r];
  __syncthreads();
  tile_epilogue<BM, BN, CS>(pol, Cs, m0, M, t, part, split, ldp);
}

// ---------------------------------------------------------------------------
// float32 kernel (fp32 mode): 32x32 tiles, BK = 32, 256 threads, 4 outputs each
// ---------------------------------------------------------------------------
template <class Pol>
__global__ void __launch_bounds__(256) gemm_f32_kernel(Pol pol, GemmA ga, int M, int k_per_split,
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
  const float* cs = (const float*)ga.cscale;
  const int tr = tid / 8, tc = (tid % 8) * 4;   // output row, first of 4 columns
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = kbeg; k0 < kbeg + k_per_split; k0 += BK) {
    for (int idx = tid; idx < BM * BK; idx += 256) {
      const int r = idx / BK, kk = idx % BK;
      const int m = min(m0 + r, M - 1);
      const int pm = (m / ga.per) * ga.stride + ga.off + m % ga.per;
      float v = ga.a[(size_t)pm * ga.lda + k0 + kk];
      if (ga.rscale) v *= ga.rscale[m];
      if (cs) v *= cs[k0 + kk];
      As[kk][r] = v;
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
template <int BN, class Pol>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(Pol pol, const float* __restrict__ part,
                                                            int ldp, int M, int S, int ntiles) {
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if constexpr (Pol::PAIRED) {
    const size_t per_row = (size_t)ntiles * (BN / 2);
    if (idx >= (size_t)M * per_row) return;
    const int m = idx / per_row, rem = idx % per_row;
    const int t = rem / (BN / 2), c = rem % (BN / 2);
    float lo = 0.f, hi = 0.f;
    for (int s = 0; s < S; ++s) {
      const float* p = part + ((size_t)s * M + m) * ldp + (size_t)t * BN + c;
      lo += p[0];
      hi += p[BN / 2];
    }
    pol.store(m, t, c, BN, lo, hi);
  } else {
    const size_t per_row = (size_t)ntiles * BN;
    if (idx >= (size_t)M * per_row) return;
    const int m = idx / per_row, n = idx % per_row;
    float v = 0.f;
    for (int s = 0; s < S; ++s) v += part[((size_t)s * M + m) * ldp + n];
    pol.store1(m, n, v);
  }
}

// ---------------------------------------------------------------------------
// row RMS: inv[o] = 1 / sqrt(mean(x[row(o)]^2) + eps)
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) row_rms_kernel(const float* __restrict__ x, int d, float eps,
                                                      float* __restrict__ inv, int n_rows, int per,
                                                      int stride, int off) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + wave;           // one wave per row
  if (o >= n_rows) return;
  const float* xr = x + ((size_t)(o / per) * stride + off + o % per) * d;
  float ss = 0.f;
  for (int c = lane * 4; c < d; c += 256) {
    const float4 v = *(const float4*)(xr + c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  if (lane == 0) inv[o] = 1.0f / sqrtf(ss / (float)d + eps);
}

hipError_t launch_row_rms(const float* x, int d, float eps, float* inv, int n_rows, int per,
                          int stride, int off, hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  hipLaunchKernelGGL(row_rms_kernel, dim3(ceil_div(n_rows, 4)), dim3(256), 0, st, x, d, eps, inv,
                     n_rows, per, stride, off);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// host-side dispatch
// ---------------------------------------------------------------------------
// Split-K is only used while S * M stays small, which bounds the workspace.
static constexpr int SPLIT_ROWS_MAX = 1024;

size_t gemm_split_ws_floats(int M, int max_n) {
  (void)M;
  return (size_t)SPLIT_ROWS_MAX * max_n;
}

// Per-projection launch choice (tile width BN, split-K S, prefetch depths).
struct GemmCfg {
  int bn, s, pa, pw;
};

// Tuning override: SSM_GEMM_CFG="kind:bn:s:pa:pw,..." with kind one of
// qkv, o, gate_up, down, lm and s = 0 for the automatic split.
static GemmCfg cfg_override(const char* kind, GemmCfg c) {
  static const char* env = getenv("SSM_GEMM_CFG");   // read once per process
  if (!env) return c;
  const size_t kl = strlen(kind);
  for (const char* p = env; p && *p;) {
    if (strncmp(p, kind, kl) == 0 && p[kl] == ':') {
      int bn, s, pa, pw;
      if (sscanf(p + kl + 1, "%d:%d:%d:%d", &bn, &s, &pa, &pw) == 4) return GemmCfg{bn, s, pa, pw};
    }
    p = strchr(p, ',');
    if (p) ++p;
  }
  return c;
}

static int auto_split(int tiles, int M, int K, size_t ws_floats, int N) {
  int S = 1;
  while (S < 8 && tiles * S < 192 && K % (64 * S * 2) == 0 && (S * 2) * M <= SPLIT_ROWS_MAX &&
         (size_t)(S * 2) * M * N <= ws_floats)
    S *= 2;
  return S;
}

template <int BN, int PA, int PW, bool SPLIT, class Pol>
static hipError_t launch_bf16(const Pol& pol, const GemmA& ga, int M, int K, int N, int S,
                              SplitWs ws, hipStream_t st) {
  constexpr int BM = 128, WM = 64, WN = BN / 2;
  const int ntiles = N / BN, mt = ceil_div(M, BM);
  dim3 grid(ntiles * mt, S);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN, PA, PW, SPLIT, Pol>), grid, dim3(256), 0,
                     st, pol, ga, M, K / S, mt, S > 1 ? ws.part : nullptr, N);
  if (S > 1) {
    const size_t total = (size_t)M * N / (Pol::PAIRED ? 2 : 1);
    hipLaunchKernelGGL((splitk_reduce_kernel<BN, Pol>), dim3((unsigned)((total + 255) / 256)),
                       dim3(256), 0, st, pol, ws.part, N, M, S, ntiles);
  }
  return hipGetLastError();
}

template <int BN, bool SPLIT, class Pol>
static hipError_t launch_bf16_pf(const Pol& pol, const GemmA& ga, int M, int K, int N, int S,
                                 int pa, int pw, SplitWs ws, hipStream_t st) {
  if (pa == 2 && pw == 4) return launch_bf16<BN, 2, 4, SPLIT>(pol, ga, M, K, N, S, ws, st);
  if (pa == 1 && pw == 2) return launch_bf16<BN, 1, 2, SPLIT>(pol, ga, M, K, N, S, ws, st);
  if (pa == 2 && pw == 2) return launch_bf16<BN, 2, 2, SPLIT>(pol, ga, M, K, N, S, ws, st);
  return launch_bf16<BN, 1, 4, SPLIT>(pol, ga, M, K, N, S, ws, st);
}

// PolBN<BN> rebinds the tile width of the epilogue policies that depend on it.
template <class Pol>
static hipError_t run_bf16(const char* kind, Pol pol, const GemmA& ga, int M, int K, int N,
                           bool split, GemmCfg c, SplitWs ws, hipStream_t st,
                           void (*rebind)(Pol&, int) = nullptr) {
  c = cfg_override(kind, c);
  if (c.bn != 64 && c.bn != 128) c.bn = 128;
  if (N % c.bn) c.bn = 64;
  if (rebind) rebind(pol, c.bn);
  const int tiles = (N / c.bn) * ceil_div(M, 128);
  int S = c.s > 0 ? c.s : auto_split(tiles, M, K, ws.floats, N);
  while (S > 1 && (K % (64 * S) != 0 || (size_t)S * M * N > ws.floats)) S /= 2;
  if (c.bn == 128)
    return split ? launch_bf16_pf<128, true>(pol, ga, M, K, N, S, c.pa, c.pw, ws, st)
                 : launch_bf16_pf<128, false>(pol, ga, M, K, N, S, c.pa, c.pw, ws, st);
  return split ? launch_bf16_pf<64, true>(pol, ga, M, K, N, S, c.pa, c.pw, ws, st)
               : launch_bf16_pf<64, false>(pol, ga, M, K, N, S, c.pa, c.pw, ws, st);
}

template <class Pol>
static hipError_t run_f32(const Pol& pol, const GemmA& ga, int M, int K, int N, SplitWs ws,
                          hipStream_t st) {
  constexpr int BN = 32;
  const int ntiles = N / BN, mt = ceil_div(M, 32);
  int S = 1;
  while (S < 8 && ntiles * mt * S < 256 && K % (32 * S * 2) == 0 && (S * 2) * M <= SPLIT_ROWS_MAX &&
         (size_t)(S * 2) * M * N <= ws.floats)
    S *= 2;
  dim3 grid(ntiles, mt, S);
  hipLaunchKernelGGL((gemm_f32_kernel<Pol>), grid, dim3(256), 0, st, pol, ga, M, K / S,
                     S > 1 ? ws.part : nullptr, N);
  if (S > 1) {
    const size_t total = (size_t)M * N / (Pol::PAIRED ? 2 : 1);
    hipLaunchKernelGGL((splitk_reduce_kernel<BN, Pol>), dim3((unsigned)((total + 255) / 256)),
                       dim3(256), 0, st, pol, ws.part, N, M, S, ntiles);
  }
  return hipGetLastError();
}

// Default launch choices for the HBM-bound row counts of cached steps (M <=
// 256) and the compute-bound ones of block-start steps.
static GemmCfg default_cfg(const char* kind, int M) {
  const bool small = M <= 256;
  if (!strcmp(kind, "qkv")) return small ? GemmCfg{64, 1, 1, 4} : GemmCfg{128, 1, 1, 2};
  if (!strcmp(kind, "gate_up")) return small ? GemmCfg{128, 1, 1, 4} : GemmCfg{128, 1, 1, 2};
  if (!strcmp(kind, "lm")) return small ? GemmCfg{128, 1, 1, 4} : GemmCfg{128, 1, 1, 2};
  return small ? GemmCfg{128, 0, 1, 4} : GemmCfg{128, 0, 1, 2};   // o, down
}

static void rebind_qkv(PolQKV<bf16_t>& p, int bn) { p.tiles_per_head = p.dh / bn; }

hipError_t gemm_qkv(int dtype, bool split, const GemmA& ga, int M, int d, const void* wq,
                    const void* wk, const void* wv, int H, int Hkv, int dh, const QKVOut& o,
                    SplitWs ws, hipStream_t st) {
  const int N = (H + 2 * Hkv) * dh;
  if (dtype == 0) {
    PolQKV<float> p{(const float*)wq, (const float*)wk, (const float*)wv, d, H, Hkv, dh, dh / 32,
                    (float*)o.q, (float*)o.kc, (float*)o.vc, o.cap, o.n_cached, o.n_rows, o.rope};
    return run_f32(p, ga, M, d, N, ws, st);
  }
  PolQKV<bf16_t> p{(const bf16_t*)wq, (const bf16_t*)wk, (const bf16_t*)wv, d, H, Hkv, dh,
                   dh / 128, (bf16_t*)o.q, (bf16_t*)o.kc, (bf16_t*)o.vc, o.cap, o.n_cached,
                   o.n_rows, o.rope};
  return run_bf16("qkv", p, ga, M, d, N, split, default_cfg("qkv", M), ws, st, rebind_qkv);
}

hipError_t gemm_resid(int dtype, bool split, const char* kind, const GemmA& ga, int M, int K,
                      const void* w, int N, float* resid, SplitWs ws, hipStream_t st) {
  if (dtype == 0) {
    PolResid<float> p{(const float*)w, K, N, resid};
    return run_f32(p, ga, M, K, N, ws, st);
  }
  PolResid<bf16_t> p{(const bf16_t*)w, K, N, resid};
  return run_bf16(kind, p, ga, M, K, N, split, default_cfg(kind, M), ws, st);
}

hipError_t gemm_swiglu(int dtype, bool split, const GemmA& ga, int M, int d, const void* wg,
                       const void* wu, int F, float* act, SplitWs ws, hipStream_t st) {
  if (dtype == 0) {
    PolSwiGLU<float> p{(const float*)wg, (const float*)wu, d, F, act};
    return run_f32(p, ga, M, d, 2 * F, ws, st);
  }
  PolSwiGLU<bf16_t> p{(const bf16_t*)wg, (const bf16_t*)wu, d, F, act};
  return run_bf16("gate_up", p, ga, M, d, 2 * F, split, default_cfg("gate_up", M), ws, st);
}

hipError_t gemm_store(int dtype, bool split, const GemmA& ga, int M, int K, const void* w, int N,
                      float* c, int ldc, SplitWs ws, hipStream_t st) {
  if (dtype == 0) {
    PolStore<float> p{(const float*)w, K, ldc, c};
    return run_f32(p, ga, M, K, N, ws, st);
  }
  PolStore<bf16_t> p{(const bf16_t*)w, K, ldc, c};
  return run_bf16("lm", p, ga, M, K, N, split, default_cfg("lm", M), ws, st);
}

// Merges the partial statistics of one row (one workgroup per row), in a
// fixed order: deterministic.
__global__ void __launch_bounds__(256) lm_merge_kernel(const LMPartial* __restrict__ part,
                                                       int n_part, int k,
                                                       int32_t* __restrict__ argmax,
                                                       float* __restrict__ conf,
                                                       int32_t* __restrict__ topk_ids,
                                                       float* __restrict__ topk_w) {
  __shared__ float s_m[256];
  __shared__ float s_s[256];
  __shared__ float s_v[4];
  __shared__ int s_i[4];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const LMPartial* P = part + (size_t)row * n_part;
  float tv[8];
  int ti[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) { tv[q] = -INFINITY; ti[q] = 0x7fffffff; }
  float mx = -INFINITY, sm = 0.f;
  for (int j = tid; j < n_part; j += 256) {
    const LMPartial& p = P[j];
    if (p.s > 0.f) {
      if (p.m > mx) { sm = sm * expf(mx - p.m) + p.s; mx = p.m; }
      else sm += p.s * expf(p.m - mx);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q)
      if (stat_better(p.v[q], p.id[q], tv[7], ti[7])) stat_insert(tv, ti, p.v[q], p.id[q]);
  }
  s_m[tid] = mx;
  s_s[tid] = sm;
  __syncthreads();
  if (tid == 0) {
    float M = -INFINITY;
    for (int t = 0; t < 256; ++t) M = fmaxf(M, s_m[t]);
    float S = 0.f;
    for (int t = 0; t < 256; ++t)
      if (s_s[t] > 0.f) S += s_s[t] * expf(s_m[t] - M);
    s_s[0] = S;
  }
  __syncthreads();
  const float S = s_s[0];
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

hipError_t lm_head_stats(bool split, const GemmA& ga, int M, int K, const void* w, int N,
                         int mask_id, int k, void* stats_ws, float* logits, int32_t* argmax,
                         float* conf, int32_t* topk_ids, float* topk_w, hipStream_t st) {
  constexpr int BN = 128;
  const int ntiles = N / BN;
  PolLMStats<bf16_t> p{(const bf16_t*)w, K, N, mask_id, (LMPartial*)stats_ws, 2 * ntiles, logits, N};
  GemmCfg c = cfg_override("lm", default_cfg("lm", M));
  const int pa = c.pa, pw = c.pw;
  SplitWs none{nullptr, 0};
  hipError_t e = split ? launch_bf16_pf<BN, true>(p, ga, M, K, N, 1, pa, pw, none, st)
                       : launch_bf16_pf<BN, false>(p, ga, M, K, N, 1, pa, pw, none, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lm_merge_kernel, dim3(M), dim3(256), 0, st, (const LMPartial*)stats_ws,
                     2 * ntiles, k, argmax, conf, topk_ids, topk_w);
  return hipGetLastError();
}

}  // namespace ssm
