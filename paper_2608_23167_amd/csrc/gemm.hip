// Projections of the decoder layer: C = A * W^T with A [M, K] row-major
// activations and W [N, K] row-major weights (nn.Linear layout).
//
// bfloat16 path: MFMA v_mfma_f32_16x16x32_bf16, 256 threads (4 waves) per
// workgroup, BK = 64, double-buffered LDS tiles with padded rows, fp32
// accumulation.  The output tile is staged through LDS so that the epilogue
// can combine any two columns of the tile and store coalesced.
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
  T* act;
  __device__ __forceinline__ void b_ptrs(int t, int BN, const T*& lo, const T*& hi) const {
    lo = wg + (size_t)t * (BN / 2) * ldb;
    hi = wu + (size_t)t * (BN / 2) * ldb;
  }
  __device__ __forceinline__ void store(int m, int t, int c, int BN, float g, float u) const {
    const float silu = g / (1.0f + expf(-g));
    stf(act + (size_t)m * F + t * (BN / 2) + c, silu * u);
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

// Applies the epilogue to a BM x BN float tile staged in LDS (row stride CS).
template <int BM, int BN, int CS, class Pol>
__device__ __forceinline__ void tile_epilogue(const Pol& pol, const float* Cs, int m0, int M,
                                              int t, float* part, int split, int ldp) {
  const int tid = threadIdx.x;
  if (part) {
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
template <int BM, int BN, int WM, int WN, class Pol>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(Pol pol, const bf16_t* __restrict__ A,
                                                        int lda, int M, int k_per_split,
                                                        float* __restrict__ part, int ldp) {
  constexpr int BK = 64, LS = BK + 8;            // LDS row stride (elements), 144 B
  constexpr int NWN = BN / WN;
  static_assert((BM / WM) * NWN == 4, "4 waves");
  constexpr int FM = WM / 16, FN = WN / 16;
  constexpr int ACH = BM * BK / 8 / 256, BCH = BN * BK / 8 / 256;
  static_assert(ACH >= 1 && BCH >= 1, "tile too small for 256 threads");
  constexpr int SMEM_AB = 2 * (BM + BN) * LS * 2;
  constexpr int CS = BN + 4;
  constexpr int SMEM_C = BM * CS * 4;
  constexpr int SMEM = SMEM_AB > SMEM_C ? SMEM_AB : SMEM_C;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];
  bf16_t* As = (bf16_t*)smem;
  bf16_t* Bs = As + 2 * BM * LS;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / NWN, wn = wave % NWN;
  const int t = blockIdx.x, m0 = blockIdx.y * BM, split = blockIdx.z;
  const int kbeg = split * k_per_split;
  const int nk = k_per_split / BK;

  const bf16_t *blo, *bhi;
  pol.b_ptrs(t, BN, blo, bhi);

  // chunk i of a tile covers row (tid / 8) + 32 i, 16 bytes at column 8 * (tid % 8)
  const int r0 = tid >> 3, col = (tid & 7) * 8;
  const bf16_t* a_base = A + kbeg + col;
  const bf16_t* blo_k = blo + (size_t)r0 * pol.ldb + kbeg + col;
  const bf16_t* bhi_k = bhi + (size_t)r0 * pol.ldb + kbeg + col;
  auto a_src = [&](int i, int kt) -> const uint4* {
    const int gm = min(m0 + r0 + 32 * i, M - 1);   // rows past M are computed and discarded
    return (const uint4*)(a_base + (size_t)gm * lda + kt * BK);
  };
  auto b_src = [&](int i, int kt) -> const uint4* {   // first BCH/2 chunks: lo rows
    return i < BCH / 2 ? (const uint4*)(blo_k + (size_t)(32 * i) * pol.ldb + kt * BK)
                       : (const uint4*)(bhi_k + (size_t)(32 * i - BN / 2) * pol.ldb + kt * BK);
  };
  auto dst = [&](int i) { return (r0 + 32 * i) * LS + col; };

  uint4 ra[ACH], rb[BCH];
  f32x4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int i = 0; i < ACH; ++i) ra[i] = *a_src(i, 0);
#pragma unroll
  for (int i = 0; i < BCH; ++i) rb[i] = *b_src(i, 0);
#pragma unroll
  for (int i = 0; i < ACH; ++i) *(uint4*)(As + dst(i)) = ra[i];
#pragma unroll
  for (int i = 0; i < BCH; ++i) *(uint4*)(Bs + dst(i)) = rb[i];
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
#pragma unroll
      for (int i = 0; i < ACH; ++i) ra[i] = *a_src(i, kt + 1);
#pragma unroll
      for (int i = 0; i < BCH; ++i) rb[i] = *b_src(i, kt + 1);
    }
    const bf16_t* as = As + cur * BM * LS + (wm * WM + (lane & 15)) * LS + (lane >> 4) * 8;
    const bf16_t* bs = Bs + cur * BN * LS + (wn * WN + (lane & 15)) * LS + (lane >> 4) * 8;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) af[i] = *(const bf16x8_t*)(as + i * 16 * LS + kk * 32);
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[j] = *(const bf16x8_t*)(bs + j * 16 * LS + kk * 32);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      bf16_t* an = As + (cur ^ 1) * BM * LS;
      bf16_t* bn = Bs + (cur ^ 1) * BN * LS;
#pragma unroll
      for (int i = 0; i < ACH; ++i) *(uint4*)(an + dst(i)) = ra[i];
#pragma unroll
      for (int i = 0; i < BCH; ++i) *(uint4*)(bn + dst(i)) = rb[i];
    }
    __syncthreads();
  }

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
__global__ void __launch_bounds__(256) gemm_f32_kernel(Pol pol, const float* __restrict__ A,
                                                       int lda, int M, int k_per_split,
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
      const int gm = min(m0 + r, M - 1);
      As[kk][r] = A[(size_t)gm * lda + k0 + kk];
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
// host-side dispatch
// ---------------------------------------------------------------------------
// Split-K is only used while S * M stays small, which bounds the workspace.
static constexpr int SPLIT_ROWS_MAX = 1024;

size_t gemm_split_ws_floats(int M, int max_n) {
  (void)M;
  return (size_t)SPLIT_ROWS_MAX * max_n;
}

static int choose_split(int tiles, int M, int K, int BK, size_t ws_floats, int N) {
  int S = 1;
  while (S < 8 && tiles * S < 256 && K % (BK * S * 2) == 0 && (S * 2) * M <= SPLIT_ROWS_MAX &&
         (size_t)(S * 2) * M * N <= ws_floats)
    S *= 2;
  return S;
}

template <int BM, int BN, int WM, int WN, class Pol>
static hipError_t run_bf16(const Pol& pol, const bf16_t* A, int M, int K, int N, SplitWs ws,
                           hipStream_t st) {
  const int ntiles = N / BN, mt = ceil_div(M, BM);
  const int S = choose_split(ntiles * mt, M, K, 64, ws.floats, N);
  dim3 grid(ntiles, mt, S);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN, Pol>), grid, dim3(256), 0, st, pol, A, K,
                     M, K / S, S > 1 ? ws.part : nullptr, N);
  if (S > 1) {
    const size_t total = (size_t)M * N / (Pol::PAIRED ? 2 : 1);
    hipLaunchKernelGGL((splitk_reduce_kernel<BN, Pol>), dim3((unsigned)((total + 255) / 256)),
                       dim3(256), 0, st, pol, ws.part, N, M, S, ntiles);
  }
  return hipGetLastError();
}

template <class Pol>
static hipError_t run_bf16_auto(const Pol& pol, const bf16_t* A, int M, int K, int N, SplitWs ws,
                                hipStream_t st, int max_bn = 128) {
  if (M <= 128 || max_bn < 128) return run_bf16<128, 64, 64, 32>(pol, A, M, K, N, ws, st);
  if (M <= 256) return run_bf16<256, 64, 64, 64>(pol, A, M, K, N, ws, st);
  return run_bf16<128, 128, 64, 64>(pol, A, M, K, N, ws, st);
}

template <class Pol>
static hipError_t run_f32(const Pol& pol, const float* A, int M, int K, int N, SplitWs ws,
                          hipStream_t st) {
  constexpr int BN = 32;
  const int ntiles = N / BN, mt = ceil_div(M, 32);
  const int S = choose_split(ntiles * mt, M, K, 32, ws.floats, N);
  dim3 grid(ntiles, mt, S);
  hipLaunchKernelGGL((gemm_f32_kernel<Pol>), grid, dim3(256), 0, st, pol, A, K, M, K / S,
                     S > 1 ? ws.part : nullptr, N);
  if (S > 1) {
    const size_t total = (size_t)M * N / (Pol::PAIRED ? 2 : 1);
    hipLaunchKernelGGL((splitk_reduce_kernel<BN, Pol>), dim3((unsigned)((total + 255) / 256)),
                       dim3(256), 0, st, pol, ws.part, N, M, S, ntiles);
  }
  return hipGetLastError();
}

hipError_t gemm_qkv(int dtype, const void* xn, int M, int d, const void* wq, const void* wk,
                    const void* wv, int H, int Hkv, int dh, const QKVOut& o, SplitWs ws,
                    hipStream_t st) {
  const int N = (H + 2 * Hkv) * dh;
  if (dtype == 0) {
    PolQKV<float> p{(const float*)wq, (const float*)wk, (const float*)wv, d, H, Hkv, dh, dh / 32,
                    (float*)o.q, (float*)o.kc, (float*)o.vc, o.cap, o.n_cached, o.n_rows, o.rope};
    return run_f32(p, (const float*)xn, M, d, N, ws, st);
  }
  // 64-column tiles: each tile holds (c, c + 64) pairs of one 128-wide head
  PolQKV<bf16_t> p{(const bf16_t*)wq, (const bf16_t*)wk, (const bf16_t*)wv, d, H, Hkv, dh,
                   dh / 64, (bf16_t*)o.q, (bf16_t*)o.kc, (bf16_t*)o.vc, o.cap, o.n_cached,
                   o.n_rows, o.rope};
  if (M <= 256) return run_bf16<128, 64, 64, 32>(p, (const bf16_t*)xn, M, d, N, ws, st);
  p.tiles_per_head = dh / 128;
  return run_bf16<128, 128, 64, 64>(p, (const bf16_t*)xn, M, d, N, ws, st);
}

hipError_t gemm_resid(int dtype, const void* a, int M, int K, const void* w, int N, float* resid,
                      SplitWs ws, hipStream_t st) {
  if (dtype == 0) {
    PolResid<float> p{(const float*)w, K, N, resid};
    return run_f32(p, (const float*)a, M, K, N, ws, st);
  }
  PolResid<bf16_t> p{(const bf16_t*)w, K, N, resid};
  return run_bf16_auto(p, (const bf16_t*)a, M, K, N, ws, st);
}

hipError_t gemm_swiglu(int dtype, const void* xn, int M, int d, const void* wg, const void* wu,
                       int F, void* act, SplitWs ws, hipStream_t st) {
  if (dtype == 0) {
    PolSwiGLU<float> p{(const float*)wg, (const float*)wu, d, F, (float*)act};
    return run_f32(p, (const float*)xn, M, d, 2 * F, ws, st);
  }
  PolSwiGLU<bf16_t> p{(const bf16_t*)wg, (const bf16_t*)wu, d, F, (bf16_t*)act};
  return run_bf16_auto(p, (const bf16_t*)xn, M, d, 2 * F, ws, st);
}

hipError_t gemm_store(int dtype, const void* a, int M, int K, const void* w, int N, float* c,
                      int ldc, SplitWs ws, hipStream_t st) {
  if (dtype == 0) {
    PolStore<float> p{(const float*)w, K, ldc, c};
    return run_f32(p, (const float*)a, M, K, N, ws, st);
  }
  PolStore<bf16_t> p{(const bf16_t*)w, K, ldc, c};
  return run_bf16_auto(p, (const bf16_t*)a, M, K, N, ws, st);
}

}  // namespace ssm
