// Non-causal attention of the compacted rows over every key (cached prefix
// followed by the rows' own keys), with grouped-query heads.
//
// bfloat16 path (head_dim 128): one workgroup = 4 waves of 16 QB query rows
// of one (sequence, head); QB = 2 once there are more than 64 rows, so that
// every K and V fragment read from LDS feeds two MFMAs.  Key tiles of 64 are
// copied from global memory straight into LDS (two buffers per kind).  Each
// wave computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16, so that a lane ends
// up holding 4 keys of one query: the exponentiated scores are then already
// in the B-operand layout of O^T = V^T P^T, whose V^T operand comes from the
// transposing LDS read.  The online softmax (running max, sum of P as an
// extra MFMA output block) runs in base 2 in float32; the scores of the next
// tile are computed while it runs.  Split-KV over the key range fills the GPU
// at small row counts; a merge kernel combines the per-split (max, sum,
// output) triples in split order.  Decode launches (few query rows, a short
// key range) instead give each block of 16 query rows a workgroup of its own,
// whose waves split the key tiles and merge in LDS (attn_dec_kernel).
#include "internal.h"
#include "dcheck.h"

namespace ssm {

constexpr float LOG2E = 1.4426950408889634f;
typedef short v4i16_t __attribute__((ext_vector_type(4)));

// LDS tiles of 64 keys x 128 dimensions, rows of 256 bytes, both copied
// straight from global memory (global_load_lds, 1 KB = 4 rows per
// instruction).
//  * K: the 16-byte chunk j of row r sits at slot j ^ (r % 16); a K fragment
//    (16 rows at one chunk) then reads 16 different slots.
//  * V: the 32-byte block j (dimensions 16j .. 16j + 15) of row r sits at
//    block j ^ (r % 8).  The V^T operand of the P V product is read with the
//    transposing load ds_read_b64_tr_b16: within a group of 16 lanes, lanes
//    4r .. 4r + 3 each supply 4 consecutive dimensions of key row r and lane
//    i receives dimension i of the 4 rows.  A read covers 16 rows x 32 bytes
//    over 8 block positions, 2 rows each: two passes, the minimum for 512 bytes.
__device__ __forceinline__ int k_slot(int row, int chunk) { return row * 256 + ((chunk ^ (row & 15)) << 4); }
__device__ __forceinline__ int v_byte(int row, int block) { return row * 256 + ((block ^ (row & 7)) << 5); }

// Cross-lane maximum over the 4 lanes l, l ^ 16, l ^ 32, l ^ 48 (the lanes
// that hold the scores of one query) with the gfx950 lane-swap instructions.
__device__ __forceinline__ float max_lanes_16_32(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Element type of the MFMA operands q, k, v and P: bfloat16 or float16.  A
// bfloat16 model keeps its attention operands in float16 (see gemm_qkv): the
// same MFMA rate and bytes, three more significand bits.  P is packed with
// round-toward-zero in float16 (one instruction per pair); its relative error
// is then below 2^-10 and the row sum, taken from the same rounded P,
// cancels the bias.
template <typename E> struct AttnOps;
template <> struct AttnOps<bf16_t> {
  typedef bf16x8_t vec;
  static constexpr uint32_t ONE2 = 0x3f803f80u;   // two bfloat16 ones
  __device__ __forceinline__ static f32x4_t mfma(vec a, vec b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ __forceinline__ static uint32_t pack(float a, float b) { return pack_bf16x2(a, b); }
};
template <> struct AttnOps<f16_t> {
  typedef f16x8_t vec;
  static constexpr uint32_t ONE2 = 0x3c003c00u;   // two float16 ones
  __device__ __forceinline__ static f32x4_t mfma(vec a, vec b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
  __device__ __forceinline__ static uint32_t pack(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(a, b));
  }
};

// Workgroup order: a 1-D grid over (query tile, sequence x head, split),
// query tiles innermost, dealt so that each XCD (workgroup id w runs on XCD
// w % 8) gets a contiguous range: the query tiles of one head then read its
// keys and values through one L2 instead of one per XCD.
__device__ __forceinline__ void attn_tile_of(int w, int total, int qtiles, int BH, int& qt,
                                             int& bh, int& split) {
  const int per = total / 8;
  const int v = w < per * 8 ? (w % 8) * per + (w / 8) : w;
  qt = v % qtiles;
  bh = (v / qtiles) % BH;
  split = v / (qtiles * BH);
}

// Four consecutive output columns col .. col + 3 of row `row` (col a multiple
// of 4, so one 8-column chunk of the fragment order holds them): float32
// row-major, or bfloat16 hi (and lo = the rounding remainder) in fragment order.
__device__ __forceinline__ void store_out4(const ActOut& O, int row, int col, const float (&v)[4]) {
  if (O.f32) {
    *(float4*)((float*)O.hi + (size_t)row * O.ld + col) = make_float4(v[0], v[1], v[2], v[3]);
    return;
  }
  const size_t idx = frag_index(row, col, O.G);
  const uint2 hw = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
  *(uint2*)((bf16_t*)O.hi + idx) = hw;
  if (O.lo) {
    float r[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = v[e] - bf2f((bf16_t)((e >> 1 ? hw.y : hw.x) >> (16 * (e & 1))));
    *(uint2*)(O.lo + idx) = uint2{pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3])};
  }
}

// NG key groups per workgroup.  NG = 1: 4 waves walk the workgroup's key
// range.  NG = 2 (small grids of decode steps, one workgroup per CU): two
// groups of 4 waves take the query rows of the tile each, over the first and
// the second half of the key tiles, with buffers of their own; group 1 then
// hands its (output, maximum, sum) to group 0 through LDS, which merges and
// writes.  Both groups pass the same barriers: a group with fewer tiles idles
// through the missing steps.  Two waves per SIMD and half the tile chain per
// wave: a decode launch is bound by the dependent chain of each tile step.
template <int QB, typename E, int NG>
__global__ void __launch_bounds__(256 * NG, NG == 1 ? 2 : 1) attn_bf16_kernel(
    const E* __restrict__ Q, const E* __restrict__ Kc, const E* __restrict__ Vc,
    int H, int Hkv, int Mq, int Nk, int cap, int keys_per_split, float scale_log2,
    ActOut O, float* __restrict__ Opart, float* __restrict__ ML, int qtiles, int BH, Pads pads) {
  typedef AttnOps<E> Ops;
  typedef typename Ops::vec vec;
  constexpr int DH = 128, KT = 64, TBUF = KT * DH;
  static_assert(NG == 1 || (NG == 2 && QB == 1), "two key groups with 16 query rows per wave");
  // two buffers per tile kind and group
  __shared__ __attribute__((aligned(1024))) E Ks_all[NG * 2 * TBUF];
  __shared__ __attribute__((aligned(1024))) E Vs_all[NG * 2 * TBUF];
  const int tid = threadIdx.x, lane = tid & 63;
  const int grp = NG == 1 ? 0 : __builtin_amdgcn_readfirstlane(tid >> 8);
  const int wave = (tid >> 6) & 3;           // wave within its group
  E* const Ks = Ks_all + grp * 2 * TBUF;
  E* const Vs = Vs_all + grp * 2 * TBUF;
  const int g = lane >> 4, c16 = lane & 15;
  int qt, bh, split;
  attn_tile_of(blockIdx.x, gridDim.x, qtiles, BH, qt, bh, split);
  const int s = bh / H, h = bh % H, kvh = h / (H / Hkv);
  // a padded sequence's keys start after its padding slots
  const int kb_wg = pads.of(s) + split * keys_per_split, ke_wg = min(Nk, kb_wg + keys_per_split);
  // query block b of the wave: rows q0 + 16 b .. + 15; this lane's query in it
  const int q0 = (qt * 4 + wave) * 16 * QB;
  if (kb_wg >= ke_wg) {
    // a split past the end of a padded sequence's shorter key range: an empty
    // partial (sum 0), which the merge skips (the host keeps split 0 non-empty)
    if (Opart != nullptr && g == 0 && grp == 0) {
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        const int q = q0 + 16 * b + c16;
        if (q >= Mq) continue;
        const size_t row = ((size_t)split * BH + bh) * Mq + q;
        ML[row * 2] = -INFINITY;
        ML[row * 2 + 1] = 0.f;
      }
    }
    return;
  }
  // this group's part of the range: whole tiles, the first group's part first
  const int steps = (ke_wg - kb_wg + KT * NG - 1) / (KT * NG);          // tiles per group, >= 1
  const int kb = kb_wg + grp * steps * KT, ke = min(ke_wg, kb + steps * KT);
  const int ntile = ke > kb ? (ke - kb + KT - 1) / KT : 0;              // this group's tiles
  SSM_DCHECK(ke_wg <= cap);

  const E* Qh = Q + (size_t)bh * Mq * DH;
  vec qf[QB][4];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    const int q = q0 + 16 * b + c16;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      if (q < Mq) qf[b][kk] = *(const vec*)(Qh + (size_t)q * DH + 32 * kk + 8 * g);
      else qf[b][kk] = __builtin_bit_cast(vec, u32x4_t{0u, 0u, 0u, 0u});
    }
  }
  const E* Kh = Kc + (size_t)(s * Hkv + kvh) * cap * DH;
  const E* Vh = Vc + (size_t)(s * Hkv + kvh) * cap * DH;

  // tile copy: wave w copies rows 16w .. 16w + 15 of a K or V tile, 4 rows
  // per instruction; lane l covers row 16w + 4i + l / 16 and slot l % 16.
  // Keys past the range repeat the last key of the range: their scores are
  // masked, so their probabilities are exactly zero.
  const int crow = 16 * wave + (lane >> 4);
  auto copy_k = [&](int t, int buf) {
    char* dst = (char*)(Ks + buf * TBUF) + wave * 4096;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = crow + 4 * i, key = min(kb + t * KT + r, ke - 1);
      __builtin_amdgcn_global_load_lds((const void*)(Kh + (size_t)key * DH + (c16 ^ (r & 15)) * 8),
                                       (__attribute__((address_space(3))) void*)(dst + i * 1024),
                                       16, 0, 0);
    }
  };
  auto copy_v = [&](int t, int buf) {
    char* dst = (char*)(Vs + buf * TBUF) + wave * 4096;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = crow + 4 * i, key = min(kb + t * KT + r, ke - 1);
      const int vc = (((c16 >> 1) ^ (r & 7)) << 1) | (c16 & 1);
      __builtin_amdgcn_global_load_lds((const void*)(Vh + (size_t)key * DH + vc * 8),
                                       (__attribute__((address_space(3))) void*)(dst + i * 1024),
                                       16, 0, 0);
    }
  };

  // S^T block nb: sc[b][nb][r] = score(key 16nb + 4g + r, query q0 + 16b + c16);
  // each K fragment read from LDS serves the QB query blocks
  auto qk = [&](int buf, f32x4_t (&sc)[QB][4]) {
    const char* kd = (const char*)(Ks + buf * TBUF);
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
#pragma unroll
      for (int b = 0; b < QB; ++b) sc[b][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const vec a = *(const vec*)(kd + k_slot(16 * nb + c16, 4 * kk + g));
#pragma unroll
        for (int b = 0; b < QB; ++b) sc[b][nb] = Ops::mfma(a, qf[b][kk], sc[b][nb]);
      }
    }
  };

  f32x4_t o[QB][8], ol[QB];   // ol: row sums of P, an extra output block of ones
  float m_run[QB];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
#pragma unroll
    for (int i = 0; i < 8; ++i) o[b][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    ol[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    m_run[b] = -INFINITY;
  }
  const vec ones = __builtin_bit_cast(vec, u32x4_t{Ops::ONE2, Ops::ONE2, Ops::ONE2, Ops::ONE2});

  // softmax of tile t in base 2, the scale folded into one fma per score;
  // keys past the range (last tile only) are masked to -inf.  The running
  // maximum is lazy: it moves (and O and the row sums are rescaled) only when
  // some query of the wave sees a score above it by more than RESCALE (log2
  // units), so the probabilities stay below 2^RESCALE; the result is exact
  // after the final division by the row sum either way.
  constexpr float RESCALE = 8.0f;
  auto softmax_max = [&](int t, f32x4_t (&sc)[QB][4]) {
    const int k0 = kb + t * KT;
    if (k0 + KT > ke) {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (k0 + 16 * nb + 4 * g + r >= ke)
#pragma unroll
            for (int b = 0; b < QB; ++b) sc[b][nb][r] = -INFINITY;
    }
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      float mt = sc[b][0][0];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r) mt = fmaxf(mt, sc[b][nb][r]);
      const float m_tile = max_lanes_16_32(mt) * scale_log2;
      if (__builtin_amdgcn_ballot_w64(m_tile > m_run[b] + RESCALE) != 0) {
        const float m_new = fmaxf(m_run[b], m_tile);
        const float alpha = __builtin_amdgcn_exp2f(m_run[b] - m_new);
        ol[b] *= alpha;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[b][i] *= alpha;
        m_run[b] = m_new;
      }
    }
  };
  // P^T operand: slot e of lane group g holds key 32*h2 + 16*(e/4) + 4g + e%4
  auto softmax_exp = [&](const f32x4_t (&sc)[QB][4], vec (&pb)[QB][2]) {
#pragma unroll
    for (int b = 0; b < QB; ++b)
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        float p[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          p[e] = __builtin_amdgcn_exp2f(fmaf(sc[b][2 * h2 + (e >> 2)][e & 3], scale_log2, -m_run[b]));
        const u32x4_t w = {Ops::pack(p[0], p[1]), Ops::pack(p[2], p[3]), Ops::pack(p[4], p[5]),
                           Ops::pack(p[6], p[7])};
        pb[b][h2] = __builtin_bit_cast(vec, w);
      }
  };

  // O^T += V^T P^T.  V^T operand of lane (g, c16) for dimension block db:
  // dimension 16db + c16 of keys 32h2 + 4g .. + 3 (transposing read t = 0)
  // and 32h2 + 16 + 4g .. + 3 (t = 1), the slot order of P^T
  const int tr_r = c16 >> 2, tr_q = c16 & 3;
  auto pv = [&](int buf, const vec (&pb)[QB][2]) {
    const char* vd = (const char*)(Vs + buf * TBUF);
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
#pragma unroll
      for (int b = 0; b < QB; ++b)
        ol[b] = Ops::mfma(ones, pb[b][h2], ol[b]);
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const int r0 = 32 * h2 + 4 * g + tr_r, r1 = r0 + 16;
        const v4i16_t t0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16_t*)(vd + v_byte(r0, db) + tr_q * 8));
        const v4i16_t t1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16_t*)(vd + v_byte(r1, db) + tr_q * 8));
        const vec a = __builtin_bit_cast(
            vec, u32x4_t{__builtin_bit_cast(uint2, t0).x, __builtin_bit_cast(uint2, t0).y,
                         __builtin_bit_cast(uint2, t1).x, __builtin_bit_cast(uint2, t1).y});
#pragma unroll
        for (int b = 0; b < QB; ++b) o[b][db] = Ops::mfma(a, pb[b][h2], o[b][db]);
      }
    }
  };

  {
    // software pipeline: the scores of tile t + 1 are computed (MFMA) while
    // the softmax of tile t runs (VALU).  In step t the waves read K of tile
    // t + 1 and V of tile t while K of tile t + 2 and V of tile t + 1 are
    // copied into the buffers read in step t - 1; one barrier per step.
    if (ntile > 0) {
      copy_k(0, 0);
      copy_v(0, 0);
      if (ntile > 1) copy_k(1, 1);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    f32x4_t sa[QB][4], sb[QB][4];
    if (ntile > 0) qk(0, sa);
    __syncthreads();                                       // K buffer 0 is refilled next
    auto step = [&](int t, f32x4_t (&cur)[QB][4], f32x4_t (&nxt)[QB][4]) {
      if (t < ntile) {
        if (t + 2 < ntile) copy_k(t + 2, t & 1);
        if (t + 1 < ntile) copy_v(t + 1, (t + 1) & 1);
        softmax_max(t, cur);
        // the next tile's score MFMAs between this tile's maximum and its
        // exponentials: the MFMAs of one wave overlap the VALU work of the
        // other wave on the SIMD
        if (t + 1 < ntile) qk((t + 1) & 1, nxt);
        vec pb[QB][2];
        softmax_exp(cur, pb);
        pv(t & 1, pb);
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
    };
    for (int t = 0; t < steps; t += 2) {
      step(t, sa, sb);
      if (t + 1 < steps) step(t + 1, sb, sa);
    }
  }

  if constexpr (NG == 2) {
    // group 1 hands over its state (the loop has drained every copy and
    // read): outputs at Ks_all's second half, (maximum, sum) at Vs_all's
    float* xo = (float*)(Ks_all + 2 * TBUF) + (wave * 64 + lane) * (8 * 4 * QB);
    float* xm = (float*)(Vs_all + 2 * TBUF) + (wave * 64 + lane) * (2 * QB);
    if (grp == 1) {
#pragma unroll
      for (int b = 0; b < QB; ++b) {
#pragma unroll
        for (int i = 0; i < 8; ++i) *(f32x4_t*)(xo + (b * 8 + i) * 4) = o[b][i];
        xm[2 * b] = m_run[b];
        xm[2 * b + 1] = ol[b][0];
      }
    }
    __syncthreads();
    if (grp == 1) return;
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      const float m1 = xm[2 * b], l1 = xm[2 * b + 1];
      const float m = fmaxf(m_run[b], m1);
      // a group without keys has m = -inf and l = 0; its weight is 0
      const float w0 = ol[b][0] > 0.f ? __builtin_amdgcn_exp2f(m_run[b] - m) : 0.f;
      const float w1 = l1 > 0.f ? __builtin_amdgcn_exp2f(m1 - m) : 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[b][i] = o[b][i] * w0 + *(const f32x4_t*)(xo + (b * 8 + i) * 4) * w1;
      ol[b][0] = ol[b][0] * w0 + l1 * w1;
      m_run[b] = m;
    }
  }

#pragma unroll
  for (int b = 0; b < QB; ++b) {
    const float l = ol[b][0];   // every row of the ones block holds the sum
    const int q = q0 + 16 * b + c16;
    if (q >= Mq) continue;
    // o[b][db][r] = O^T[dh 16db + 4g + r][query q]
    if (Opart == nullptr) {
      const float inv = 1.0f / l;
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const float v[4] = {o[b][db][0] * inv, o[b][db][1] * inv, o[b][db][2] * inv, o[b][db][3] * inv};
        store_out4(O, s * Mq + q, h * DH + 16 * db + 4 * g, v);
      }
    } else {
      const size_t row = ((size_t)split * BH + bh) * Mq + q;
      float* op = Opart + row * DH;
#pragma unroll
      for (int db = 0; db < 8; ++db) *(f32x4_t*)(op + 16 * db + 4 * g) = o[b][db];
      if (g == 0) { ML[row * 2] = m_run[b]; ML[row * 2 + 1] = l; }
    }
  }
}

// Decode launches (few query rows, a short key range, no split): one
// workgroup of 8 waves per (sequence, head, block of 16 query rows), so the
// grid holds one workgroup per CU where the 64-row workgroups above would
// leave three CUs in four idle.  All 8 waves take the same 16 query rows;
// wave w takes key tiles w, w + 8, ... of the range.  The K fragments of a
// tile are loaded straight into registers (the A layout of S^T = K Q^T: 16
// bytes of one key row per lane); its V tile goes into the wave's own LDS
// buffer (global_load_lds) and is read back transposed, as above.  No wave
// waits for another until the end, where the (output, maximum, row sum)
// triples meet in LDS and wave w merges them, in wave order, for head
// dimensions 16 w .. 16 w + 15.
template <typename E>
__global__ void __launch_bounds__(512, 1) attn_dec_kernel(
    const E* __restrict__ Q, const E* __restrict__ Kc, const E* __restrict__ Vc,
    int H, int Hkv, int Mq, int Nk, int cap, float scale_log2, ActOut O, int qblocks, int BH,
    Pads pads) {
  typedef AttnOps<E> Ops;
  typedef typename Ops::vec vec;
  constexpr int DH = 128, KT = 64, TBUF = KT * DH, NW = 8;
  __shared__ __attribute__((aligned(1024))) E Vs_all[NW * TBUF];   // 16 KB per wave
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  int qb, bh, split;
  attn_tile_of(blockIdx.x, gridDim.x, qblocks, BH, qb, bh, split);
  const int s = bh / H, h = bh % H, kvh = h / (H / Hkv);
  const int kb = pads.of(s), ke = Nk;
  const int ntile = ke > kb ? (ke - kb + KT - 1) / KT : 0;
  SSM_DCHECK(ke <= cap);
  const int q = qb * 16 + c16;

  const E* Qh = Q + (size_t)bh * Mq * DH;
  vec qf[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    if (q < Mq) qf[kk] = *(const vec*)(Qh + (size_t)q * DH + 32 * kk + 8 * g);
    else qf[kk] = __builtin_bit_cast(vec, u32x4_t{0u, 0u, 0u, 0u});
  }
  const E* Kh = Kc + (size_t)(s * Hkv + kvh) * cap * DH;
  const E* Vh = Vc + (size_t)(s * Hkv + kvh) * cap * DH;
  E* const Vs = Vs_all + wave * TBUF;

  f32x4_t o[8], ol = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;
  const vec ones = __builtin_bit_cast(vec, u32x4_t{Ops::ONE2, Ops::ONE2, Ops::ONE2, Ops::ONE2});
  constexpr float RESCALE = 8.0f;   // lazy maximum, as in attn_bf16_kernel
  const int tr_r = c16 >> 2, tr_q = c16 & 3;

  for (int t = wave; t < ntile; t += NW) {
    const int k0 = kb + t * KT;
    // the previous tile's transposing reads of this buffer have completed
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    // V tile: 16 copies of 4 rows x 256 bytes; row r = 4 i + lane / 16, whose
    // 32-byte block j goes to block position j ^ (r % 8).  Keys past the
    // range repeat the last key; their scores are masked below.
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = 4 * i + g, key = min(k0 + r, ke - 1);
      const int vc = (((c16 >> 1) ^ (r & 7)) << 1) | (c16 & 1);
      __builtin_amdgcn_global_load_lds((const void*)(Vh + (size_t)key * DH + vc * 8),
                                       (__attribute__((address_space(3))) void*)((char*)Vs + i * 1024),
                                       16, 0, 0);
    }
    // K fragments: key 16 nb + c16, dimensions 32 kk + 8 g .. + 7
    vec kf[4][4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const int key = min(k0 + 16 * nb + c16, ke - 1);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) kf[nb][kk] = *(const vec*)(Kh + (size_t)key * DH + 32 * kk + 8 * g);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    // scores S^T: sc[nb][r] = score(key k0 + 16 nb + 4 g + r, query q)
    f32x4_t sc[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      sc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) sc[nb] = Ops::mfma(kf[nb][kk], qf[kk], sc[nb]);
    }
    if (k0 + KT > ke) {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (k0 + 16 * nb + 4 * g + r >= ke) sc[nb][r] = -INFINITY;
    }
    float mt = sc[0][0];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) mt = fmaxf(mt, sc[nb][r]);
    const float m_tile = max_lanes_16_32(mt) * scale_log2;
    if (__builtin_amdgcn_ballot_w64(m_tile > m_run + RESCALE) != 0) {
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      ol *= alpha;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] *= alpha;
      m_run = m_new;
    }
    // P^T operand: slot e of lane group g holds key 32 h2 + 16 (e / 4) + 4 g + e % 4
    vec pb[2];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      float p[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        p[e] = __builtin_amdgcn_exp2f(fmaf(sc[2 * h2 + (e >> 2)][e & 3], scale_log2, -m_run));
      pb[h2] = __builtin_bit_cast(vec, u32x4_t{Ops::pack(p[0], p[1]), Ops::pack(p[2], p[3]),
                                               Ops::pack(p[4], p[5]), Ops::pack(p[6], p[7])});
    }
    // O^T += V^T P^T, the V^T operand read transposed from this wave's buffer
    const char* vd = (const char*)Vs;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      ol = Ops::mfma(ones, pb[h2], ol);
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const int r0 = 32 * h2 + 4 * g + tr_r, r1 = r0 + 16;
        const v4i16_t t0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16_t*)(vd + v_byte(r0, db) + tr_q * 8));
        const v4i16_t t1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) v4i16_t*)(vd + v_byte(r1, db) + tr_q * 8));
        const vec a = __builtin_bit_cast(
            vec, u32x4_t{__builtin_bit_cast(uint2, t0).x, __builtin_bit_cast(uint2, t0).y,
                         __builtin_bit_cast(uint2, t1).x, __builtin_bit_cast(uint2, t1).y});
        o[db] = Ops::mfma(a, pb[h2], o[db]);
      }
    }
  }

  // merge: every wave leaves its triple in LDS (over the V buffers, which all
  // waves have finished reading), outputs as [wave][db][lane] f32x4 and
  // (maximum, sum) as [wave][lane]; wave w then combines dimension block w
  // of the 8 waves in wave order.  A wave without keys has m = -inf and
  // l = 0 and weight 0.
  __syncthreads();
  f32x4_t* xo = (f32x4_t*)Vs_all;
  float2* xm = (float2*)(xo + NW * 8 * 64);
#pragma unroll
  for (int db = 0; db < 8; ++db) xo[(wave * 8 + db) * 64 + lane] = o[db];
  xm[wave * 64 + lane] = make_float2(m_run, ol[0]);   // every row of the ones block holds the sum
  __syncthreads();
  float2 ml[NW];
  f32x4_t ov[NW];
#pragma unroll
  for (int v = 0; v < NW; ++v) {
    ml[v] = xm[v * 64 + lane];
    ov[v] = xo[(v * 8 + wave) * 64 + lane];
  }
  float M = -INFINITY;
#pragma unroll
  for (int v = 0; v < NW; ++v) M = fmaxf(M, ml[v].y > 0.f ? ml[v].x : -INFINITY);
  f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float L = 0.f;
#pragma unroll
  for (int v = 0; v < NW; ++v) {
    const float w = ml[v].y > 0.f ? __builtin_amdgcn_exp2f(ml[v].x - M) : 0.f;
    acc += ov[v] * w;
    L += ml[v].y * w;
  }
  if (q >= Mq) return;
  // acc[r] = O[query q][head dimension 16 wave + 4 g + r] before the division
  const float inv = 1.0f / L;
  const float v[4] = {acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv};
  store_out4(O, s * Mq + q, h * DH + 16 * wave + 4 * g, v);
}

// float32 path: one thread per query row, keys read through the cache.
template <int DH>
__global__ void __launch_bounds__(64) attn_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ Kc, const float* __restrict__ Vc,
    int H, int Hkv, int Mq, int Nk, int cap, int keys_per_split, float scale_log2,
    ActOut O, float* __restrict__ Opart, float* __restrict__ ML, Pads pads) {
  const int bh = blockIdx.y, s = bh / H, h = bh % H, kvh = h / (H / Hkv);
  const int split = blockIdx.z;
  const int kb = pads.of(s) + split * keys_per_split, ke = min(Nk, kb + keys_per_split);
  const int q = blockIdx.x * 64 + threadIdx.x;
  if (q >= Mq) return;
  const float* qp = Q + ((size_t)bh * Mq + q) * DH;
  float qv[DH], ov[DH];
#pragma unroll
  for (int c = 0; c < DH; ++c) { qv[c] = qp[c]; ov[c] = 0.f; }
  const float* Kh = Kc + (size_t)(s * Hkv + kvh) * cap * DH;
  const float* Vh = Vc + (size_t)(s * Hkv + kvh) * cap * DH;
  float m_run = -INFINITY, l_run = 0.f;
  for (int j = kb; j < ke; ++j) {
    const float* kp = Kh + (size_t)j * DH;
    float dot = 0.f;
#pragma unroll
    for (int c = 0; c < DH; ++c) dot = fmaf(qv[c], kp[c], dot);
    const float sv = dot * scale_log2;
    const float m_new = fmaxf(m_run, sv);
    const float alpha = exp2f(m_run - m_new), p = exp2f(sv - m_new);
    l_run = l_run * alpha + p;
    const float* vp = Vh + (size_t)j * DH;
#pragma unroll
    for (int c = 0; c < DH; ++c) ov[c] = ov[c] * alpha + p * vp[c];
    m_run = m_new;
  }
  if (Opart == nullptr) {
    float* out = (float*)O.hi + ((size_t)s * Mq + q) * O.ld + h * DH;
    const float inv = 1.0f / l_run;
#pragma unroll
    for (int c = 0; c < DH; ++c) out[c] = ov[c] * inv;
  } else {
    const size_t row = ((size_t)split * gridDim.y + bh) * Mq + q;
#pragma unroll
    for (int c = 0; c < DH; ++c) Opart[row * DH + c] = ov[c];
    ML[row * 2] = m_run;
    ML[row * 2 + 1] = l_run;
  }
}

// Combines the splits of one (sequence, head, query) row, in split order;
// thread (row, c8) produces head dimensions 8 c8 .. 8 c8 + 7 of the row.
template <typename T>
__global__ void __launch_bounds__(256) attn_merge_kernel(const float* __restrict__ Opart,
                                                         const float* __restrict__ ML, int S,
                                                         int BH, int H, int Mq, int DH, ActOut O) {
  const int c8n = DH / 8;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= BH * Mq * c8n) return;
  const int row = idx / c8n, c0 = (idx % c8n) * 8;   // row over BH * Mq
  const int bh = row / Mq, q = row % Mq, s = bh / H, h = bh % H;
  float M = -INFINITY;
  for (int i = 0; i < S; ++i) M = fmaxf(M, ML[((size_t)i * BH * Mq + row) * 2]);
  float L = 0.f, acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < S; ++i) {
    const size_t r = (size_t)i * BH * Mq + row;
    const float l = ML[r * 2 + 1];
    if (!(l > 0.f)) continue;
    const float w = exp2f(ML[r * 2] - M);
    L += l * w;
    const float4 a = *(const float4*)(Opart + r * DH + c0), b = *(const float4*)(Opart + r * DH + c0 + 4);
    acc[0] += a.x * w; acc[1] += a.y * w; acc[2] += a.z * w; acc[3] += a.w * w;
    acc[4] += b.x * w; acc[5] += b.y * w; acc[6] += b.z * w; acc[7] += b.w * w;
  }
  const float inv = 1.0f / L;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] *= inv;
  O.store8<T>(s * Mq + q, h * DH + c0, acc);
}

// Query rows per wave (16 QB) and split count of a launch (see attention()).
static int attention_qb(int dtype, int BH, int Mq) {
  const bool mfma = dtype == ATTN_BF16 || dtype == ATTN_F16;
  return mfma && Mq > 64 && ceil_div(Mq, 64) * BH >= 512 ? 2 : 1;
}

// Decode launches go to attn_dec_kernel: one workgroup per 16 query rows of a
// head fills at most one round of CUs, and the key range gives each of its 8
// waves at most two tiles.  A tuning build (SSM_TUNING defined) lets
// SSM_ATTN_DEC override the workgroup bound (0: never); the product build
// reads no environment variable.
static bool attention_dec(int BH, int Mq, int Nk) {
  int max_wg = 256;
#ifdef SSM_TUNING
  static const int env = [] {
    const char* e = getenv("SSM_ATTN_DEC");
    return e ? atoi(e) : -1;
  }();
  if (env >= 0) max_wg = env;
#endif
  return ceil_div(Mq, 16) * BH <= max_wg && ceil_div(Nk, 64) <= 16;
}

int attention_splits(int dtype, int B, int H, int Mq, int Nk, int max_splits, int* keys_per_split) {
  const int BH = B * H;
  const int qtiles = ceil_div(Mq, 64 * attention_qb(dtype, BH, Mq));
  // split the key range (whole 64-key tiles) until every split has about two
  // tiles or the grid reaches two workgroups per CU: each workgroup walks its
  // tiles in sequence and hides only the next tile's load, so long ranges
  // spread over many workgroups beat few long walks.  Up to 10 tiles the
  // range is not split: a workgroup's fixed cost (launch, query and first
  // tile loads, output) is about 9 us against 0.4 us per further tile, and
  // the merge kernel would cost more than the shorter walk saves.
  const int key_tiles = ceil_div(Nk, 64);
  int S = key_tiles <= 10 ? 1 : key_tiles / 2;
  if (S > max_splits) S = max_splits;
  if (S > 512 / (qtiles * BH)) S = 512 / (qtiles * BH);
  if (S < 1) S = 1;
  const int kps = ceil_div(key_tiles, S) * 64;
  if (keys_per_split) *keys_per_split = kps;
  return ceil_div(Nk, kps);           // every split holds at least one key
}

hipError_t attention(int dtype, const void* q, const void* kc, const void* vc, int B, int H,
                     int Hkv, int dh, int Mq, int Nk, int cap, const ActOut& out, AttnWs ws,
                     const Pads& pads, hipStream_t st) {
  if (Mq == 0) return hipSuccess;
  const int BH = B * H;
  // bfloat16 / float16: 32 query rows per wave (128 per workgroup), which
  // halves the LDS reads per MFMA, once 64-row tiles alone would give two
  // workgroups per CU; below that 16 per wave, twice the workgroups for a
  // launch that is bound by latency rather than by MFMA or HBM.  float32: 64
  // rows per block.
  const bool mfma = dtype == ATTN_BF16 || dtype == ATTN_F16;
  const int QB = attention_qb(dtype, BH, Mq);
  const int qtiles = ceil_div(Mq, 64 * QB);
  int kps = 0;
  const int S = attention_splits(dtype, B, H, Mq, Nk, ws.max_splits, &kps);
  const float scale_log2 = LOG2E / sqrtf((float)dh);
  float* opart = S > 1 ? ws.opart : nullptr;
  if (mfma && S == 1 && attention_dec(BH, Mq, Nk)) {
    const int qblocks = ceil_div(Mq, 16);
    const dim3 grid(qblocks * BH);
    if (dtype == ATTN_F16)
      launch(attn_dec_kernel<f16_t>, grid, dim3(512), 0, st, (const f16_t*)q, (const f16_t*)kc,
             (const f16_t*)vc, H, Hkv, Mq, Nk, cap, scale_log2, out, qblocks, BH, pads);
    else
      launch(attn_dec_kernel<bf16_t>, grid, dim3(512), 0, st, (const bf16_t*)q, (const bf16_t*)kc,
             (const bf16_t*)vc, H, Hkv, Mq, Nk, cap, scale_log2, out, qblocks, BH, pads);
  } else if (mfma) {
    const dim3 grid(qtiles * BH * S);
    // small grids (at most one workgroup per CU) whose splits hold two tiles or
    // more: two key groups per workgroup
    const bool groups = QB == 1 && qtiles * BH * S <= 256 && kps >= 2 * 64;
    auto go = [&](auto kernel, int threads, auto* qh, auto* kh, auto* vh) {
      launch(kernel, grid, dim3(threads), 0, st, qh, kh, vh, H, Hkv, Mq, Nk, cap, kps, scale_log2,
             out, opart, ws.ml, qtiles, BH, pads);
    };
    if (dtype == ATTN_F16) {
      const f16_t *qh = (const f16_t*)q, *kh = (const f16_t*)kc, *vh = (const f16_t*)vc;
      if (QB == 2) go(attn_bf16_kernel<2, f16_t, 1>, 256, qh, kh, vh);
      else if (groups) go(attn_bf16_kernel<1, f16_t, 2>, 512, qh, kh, vh);
      else go(attn_bf16_kernel<1, f16_t, 1>, 256, qh, kh, vh);
    } else {
      const bf16_t *qh = (const bf16_t*)q, *kh = (const bf16_t*)kc, *vh = (const bf16_t*)vc;
      if (QB == 2) go(attn_bf16_kernel<2, bf16_t, 1>, 256, qh, kh, vh);
      else if (groups) go(attn_bf16_kernel<1, bf16_t, 2>, 512, qh, kh, vh);
      else go(attn_bf16_kernel<1, bf16_t, 1>, 256, qh, kh, vh);
    }
  } else {
    const dim3 grid(qtiles, BH, S);
    const float* qf = (const float*)q;
    const float* kf = (const float*)kc;
    const float* vf = (const float*)vc;
    const ActOut& of = out;
    if (dh == 32)
      launch(attn_f32_kernel<32>, grid, dim3(64), 0, st, qf, kf, vf, H, Hkv, Mq, Nk,
                         cap, kps, scale_log2, of, opart, ws.ml, pads);
    else if (dh == 64)
      launch(attn_f32_kernel<64>, grid, dim3(64), 0, st, qf, kf, vf, H, Hkv, Mq, Nk,
                         cap, kps, scale_log2, of, opart, ws.ml, pads);
    else
      launch(attn_f32_kernel<128>, grid, dim3(64), 0, st, qf, kf, vf, H, Hkv, Mq, Nk,
                         cap, kps, scale_log2, of, opart, ws.ml, pads);
  }
  if (S > 1) {
    const dim3 mgrid(ceil_div(BH * Mq * (dh / 8), 256));
    if (mfma)
      launch(attn_merge_kernel<bf16_t>, mgrid, dim3(256), 0, st, ws.opart, ws.ml, S,
                         BH, H, Mq, dh, out);
    else
      launch(attn_merge_kernel<float>, mgrid, dim3(256), 0, st, ws.opart, ws.ml, S,
                         BH, H, Mq, dh, out);
  }
  return hipGetLastError();
}

}  // namespace ssm
