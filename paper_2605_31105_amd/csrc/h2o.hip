// Token scores of H2O, the token-based eviction method GRKV is paired with
// (Sec. 2: heavy hitters kept by accumulated attention scores; Sec. 4.3,
// compatibility).  A prefix token's score is the attention it receives,
// summed over every prompt position of every query head of its KV head's
// group, each row being the causal softmax of q_i K^T / sqrt(d) over keys
// 0..i:
//   s_j = sum_g sum_{i >= j} 2^(t_{g,i,j} - LSE2_{g,i}),  t = q . k log2(e) / sqrt(d).
// This is the work of a prefill attention without P.V (O(n^2 d) per head),
// done in two MFMA passes with no atomics, each with 8 waves, so that a tile
// staged in LDS feeds many MFMAs per barrier:
//  * h2o_lse_kernel: a block takes 512 / G prompt positions of all G query
//    heads (512 rows, head-major; wave w owns rows 64w .. 64w + 63, four
//    16-row tiles as MFMA B operands in registers) and streams the key tiles
//    (64 keys) up to its last position through LDS, keeping per row and lane
//    an integer reference exponent and an fp64 sum of 2^(t - ref) (as the
//    window's pass A does); the four lanes of a row merge at the end into
//    LSE2 (log2 domain).  Blocks run latest positions first (most keys);
//  * h2o_colsum_kernel: a block takes 128 prefix keys (wave w: keys
//    16w .. 16w + 15 as A operands in registers; more keys per block re-read
//    the queries less but balance the causal triangle worse, measured slower)
//    and streams the query tiles
//    (256 / G positions of all heads) at or after its first key, with their
//    LSE2, through LDS; P = 2^(t - LSE2) under the causal rule is summed per
//    key, in fp32 within a query tile and in fp64 across tiles; a 16-lane
//    reduction at the end gives the key's score.
// Causal masks are applied only on tiles that straddle the diagonal.
// The scores then drive grkv_compress_scored (selection with pool width 1).
#include "grkv_device.h"
#include "grkv_internal.h"

#include <type_traits>

namespace grkv {
namespace {

constexpr int kH2oWaves = 8;
constexpr int kH2oTh = kH2oWaves * 64;
constexpr int kH2oRows = 512;       // rows (positions x heads) of an LSE block
constexpr int kH2oKT = 64;          // keys per streamed key tile (LSE pass)
constexpr int kH2oColKT = 1;       // 16-key tiles per wave (column sums)
constexpr int kH2oColKeys = 16 * kH2oColKT * kH2oWaves;   // keys per column-sum block
constexpr int kH2oQRows = 256;      // rows (positions x heads) of a streamed query tile

// ------------------------------------------------------------ row LSE ----
template <int D, int G>
__global__ __launch_bounds__(kH2oTh) void h2o_lse_kernel(const u16* __restrict__ q_all,
                                                         const u16* __restrict__ K, int n,
                                                         float scale_log2, float* __restrict__ lse2) {
  constexpr int TQ = kH2oRows / G;          // prompt positions per block
  constexpr int KS = D + 8;                 // LDS row stride (bf16)
  constexpr int CH = kH2oKT * D / 8;        // 16-byte chunks of a key tile
  constexpr int PER = (CH + kH2oTh - 1) / kH2oTh;
  constexpr int RT = 4;                     // 16-row tiles per wave
  constexpr int KT = kH2oKT / 16;           // 16-key tiles per key tile
  constexpr float NINF = -__builtin_huge_valf();
  __shared__ __attribute__((aligned(16))) u16 kt_s[2][kH2oKT * KS];
  const int nb = (n + TQ - 1) / TQ;
  const int u = blockIdx.y, p0 = (nb - 1 - (int)blockIdx.x) * TQ, tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, gq = lane >> 4;
  const int head = (64 * wave) / TQ, pw0 = p0 + (64 * wave) % TQ;   // the wave's head, first position
  const u16* ku = K + (size_t)u * n * D;
  const u16* qh = q_all + ((size_t)u * G + head) * n * D;

  // the wave's rows: positions pw0 + 16 rt + l16 (B operand layout)
  bf16x8 qb[RT][D / 32];
  int pos[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    pos[rt] = pw0 + 16 * rt + l16;
    const int pr = min(pos[rt], n - 1);
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
      qb[rt][ks] = *reinterpret_cast<const bf16x8*>(qh + (size_t)pr * D + ks * 32 + 8 * gq);
  }
  // keys 0 .. min(n, p0 + TQ) - 1 in tiles of kH2oKT; a tile needs the
  // causal test only where it reaches past the block's first position
  const int kend = min(n, p0 + TQ);
  const int ntiles = (kend + kH2oKT - 1) / kH2oKT;
  static_assert(CH % kH2oTh == 0, "whole key tiles per block");
  bf16x8 kr[PER];
#define H2O_LOAD_K(T)                                                                     \
  _Pragma("unroll") for (int k = 0; k < PER; ++k) {                                       \
    const int e = tid + k * kH2oTh;                                                       \
    const int key = min((T) * kH2oKT + e / (D / 8), n - 1), ch = e % (D / 8);           \
    kr[k] = *reinterpret_cast<const bf16x8*>(ku + (size_t)key * D + ch * 8);              \
  }
  float mref[RT];
  double srun[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    mref[rt] = NINF;
    srun[rt] = 0.0;
  }
  H2O_LOAD_K(0)
  for (int t = 0; t < ntiles; ++t) {
    u16* cur = kt_s[t & 1];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + k * kH2oTh;
      *reinterpret_cast<bf16x8*>(cur + (e / (D / 8)) * KS + (e % (D / 8)) * 8) = kr[k];
    }
    __syncthreads();
    H2O_LOAD_K(t + 1)   // (past the last tile: clamped rows, never stored)
    const bool edge = (t + 1) * kH2oKT - 1 > pw0 || (t + 1) * kH2oKT > n;   // wave-uniform
    // tv[rt][kt][i]: key 64t + 16kt + 4gq + i, row 16rt + l16
    float tv[RT][KT][4];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      bf16x8 kf[D / 32];
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks)
        kf[ks] = *reinterpret_cast<const bf16x8*>(cur + (16 * kt + l16) * KS + ks * 32 + 8 * gq);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) acc = mfma_bf16(kf[ks], qb[rt][ks], acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) tv[rt][kt][i] = acc[i] * scale_log2;
      }
    }
    if (edge) {
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = t * kH2oKT + 16 * kt + 4 * gq + i;
            if (!(key <= pos[rt] && key < n)) tv[rt][kt][i] = NINF;
          }
    }
    // per row tile: the tile's sum against the running reference (masked keys
    // add nothing and never meet a -inf reference; only edge tiles have any)
    auto accumulate = [&](auto edge_tag) {
      constexpr bool EDGE = decltype(edge_tag)::value;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        auto tile_sum = [&](float ref) {
          float a = 0.f;
#pragma unroll
          for (int kt = 0; kt < KT; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              if constexpr (EDGE)
                a += tv[rt][kt][i] != NINF ? __builtin_amdgcn_exp2f(tv[rt][kt][i] - ref) : 0.f;
              else
                a += __builtin_amdgcn_exp2f(tv[rt][kt][i] - ref);
            }
          return a;
        };
        float a = tile_sum(mref[rt]);
        // a new reference when the tile's sum leaves [0, 2^64] (also taken on
        // the lane's first visible key, while the reference is still -inf)
        if (!(a <= 0x1p64f)) {
          float mx = NINF;
#pragma unroll
          for (int kt = 0; kt < KT; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) mx = fmaxf(mx, tv[rt][kt][i]);
          const float ref = ceilf(mx);   // finite: a was not 0, so a key is visible
          srun[rt] = mref[rt] == NINF ? 0.0 : ldexp(srun[rt], (int)(mref[rt] - ref));
          mref[rt] = ref;
          a = tile_sum(ref);
        }
        srun[rt] += (double)a;
      }
    };
    if (edge)
      accumulate(std::true_type{});
    else
      accumulate(std::false_type{});
    __syncthreads();   // the next store overwrites the other buffer only; this
                       // one is rewritten two tiles later
  }
  // merge the four lanes of each row (exact power-of-two rescales)
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const float M = max_over_groups(mref[rt]);
    const double part = mref[rt] == NINF ? 0.0 : ldexp(srun[rt], (int)(mref[rt] - M));
    const double tot = sum_over_groups(part);
    if (gq == 0 && pos[rt] < n)
      lse2[((size_t)u * G + head) * n + pos[rt]] = (float)((double)M + log2(tot));
  }
#undef H2O_LOAD_K
}

// --------------------------------------------------------- column sums ----
template <int D, int G>
__global__ __launch_bounds__(kH2oTh) void h2o_colsum_kernel(
    const u16* __restrict__ q_all, const u16* __restrict__ K, const float* __restrict__ lse2,
    int n, int P, float scale_log2, float* __restrict__ scores) {
  constexpr int TQ = kH2oQRows / G;         // positions per query tile
  constexpr int QS = D + 8;                 // LDS row stride (bf16) of Q rows
  constexpr int NR = kH2oQRows;             // rows of a query tile (head-major)
  constexpr int CH = NR * D / 8;            // 16-byte chunks of a query tile
  constexpr int PER = (CH + kH2oTh - 1) / kH2oTh;
  __shared__ __attribute__((aligned(16))) u16 q_s[2][NR * QS];
  __shared__ float l_s[2][NR];
  const int u = blockIdx.y, k0 = blockIdx.x * kH2oColKeys, tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, gq = lane >> 4;
  const u16* ku = K + (size_t)u * n * D;
  const u16* qu = q_all + (size_t)u * G * n * D;
  const float* lu = lse2 + (size_t)u * G * n;

  // this wave's keys (kH2oColKT 16-key tiles) as A operands
  constexpr int KT = kH2oColKT;
  const int kb = k0 + 16 * KT * wave;
  bf16x8 kf[KT][D / 32];
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    const int key = min(kb + 16 * kt + l16, n - 1);
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
      kf[kt][ks] = *reinterpret_cast<const bf16x8*>(ku + (size_t)key * D + ks * 32 + 8 * gq);
  }
  // query tiles at or after the block's first key
  const int qt0 = k0 / TQ, qt1 = (n + TQ - 1) / TQ;
  static_assert(CH % kH2oTh == 0 && NR <= kH2oTh, "whole query tiles per block");
  bf16x8 qr[PER];
  float lr = 0.f;
#define H2O_LOAD_Q(QT)                                                                    \
  {                                                                                       \
    const int pl0 = (QT) * TQ;                                                            \
    _Pragma("unroll") for (int k = 0; k < PER; ++k) {                                     \
      const int e = tid + k * kH2oTh;                                                     \
      const int row = e / (D / 8), ch = e % (D / 8);                                      \
      const int hg = row / TQ, pos = min(pl0 + row % TQ, n - 1);                          \
      qr[k] = *reinterpret_cast<const bf16x8*>(qu + ((size_t)hg * n + pos) * D + ch * 8);  \
    }                                                                                     \
    if (tid < NR) {                                                                       \
      const int hg = tid / TQ, pos = pl0 + tid % TQ;                                      \
      lr = pos < n ? lu[(size_t)hg * n + pos] : 0.f;                                      \
    }                                                                                     \
  }
  double col[KT][4];
#pragma unroll
  for (int kt = 0; kt < KT; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) col[kt][i] = 0.0;
  H2O_LOAD_Q(qt0)
  for (int qt = qt0; qt < qt1; ++qt) {
    const int b = (qt - qt0) & 1;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + k * kH2oTh;
      *reinterpret_cast<bf16x8*>(&q_s[b][(e / (D / 8)) * QS + (e % (D / 8)) * 8]) = qr[k];
    }
    if (tid < NR) l_s[b][tid] = lr;
    __syncthreads();
    H2O_LOAD_Q(qt + 1)   // (past the last tile: clamped rows, never stored)
    const int p0 = qt * TQ;
    // the causal test and the end of the prompt matter only on tiles that
    // start before the wave's last key or run past n (wave-uniform)
    const bool edge = p0 < kb + 16 * KT - 1 || p0 + TQ > n;
    float part[KT][4];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) part[kt][i] = 0.f;
#pragma unroll 4
    for (int rt = 0; rt < NR / 16; ++rt) {
      // rows 16 rt .. : head 16 rt / TQ, positions p0 + (16 rt) % TQ + l16
      bf16x8 qf[D / 32];
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks)
        qf[ks] = *reinterpret_cast<const bf16x8*>(&q_s[b][(16 * rt + l16) * QS + ks * 32 + 8 * gq]);
      const int rpos = p0 + (16 * rt) % TQ + l16;
      const float nl = -l_s[b][16 * rt + l16];
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) acc = mfma_bf16(kf[kt][ks], qf[ks], acc);
        // lane: key kb + 16 kt + 4 gq + i, row (head, position rpos)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float x = __builtin_amdgcn_exp2f(fmaf(acc[i], scale_log2, nl));
          if (edge) {
            const int key = kb + 16 * kt + 4 * gq + i;
            part[kt][i] += (rpos < n && key <= rpos) ? x : 0.f;
          } else {
            part[kt][i] += x;
          }
        }
      }
    }
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) col[kt][i] += (double)part[kt][i];
    __syncthreads();   // the tile in buffer b is read before it is rewritten
  }
  // sum over the 16 lanes (rows) sharing each key, in fp64
#pragma unroll
  for (int kt = 0; kt < KT; ++kt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      double v = col[kt][i];
      v += __shfl_xor(v, 1);
      v += __shfl_xor(v, 2);
      v += __shfl_xor(v, 4);
      v += __shfl_xor(v, 8);
      const int key = kb + 16 * kt + 4 * gq + i;
      if (l16 == 0 && key < P) scores[(size_t)u * P + key] = (float)v;
    }
#undef H2O_LOAD_Q
}

template <int D, int G>
hipError_t launch_h2o_t(const u16* q_all, const u16* K, int U, int n, int P, float* lse2,
                        float* scores, hipStream_t s) {
  const float scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  constexpr int TQ = kH2oRows / G;
  hipLaunchKernelGGL((h2o_lse_kernel<D, G>), dim3((n + TQ - 1) / TQ, U), dim3(kH2oTh), 0, s, q_all,
                     K, n, scale_log2, lse2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || P < 1) return e;
  hipLaunchKernelGGL((h2o_colsum_kernel<D, G>), dim3((P + kH2oColKeys - 1) / kH2oColKeys, U),
                     dim3(kH2oTh), 0, s, q_all, K, lse2, n, P, scale_log2, scores);
  return hipGetLastError();
}

}  // namespace

bool h2o_supported(int dtype, int d, int G) {
  return dtype == GRKV_BF16 && (d == 64 || d == 128) && (G == 1 || G == 2 || G == 4 || G == 8);
}

hipError_t launch_h2o(const void* q_all, const void* K, int U, int G, int d, int64_t n, int P,
                      float* lse2, float* scores, hipStream_t s) {
#define GRKV_H2O(DV, GV)                                                                     \
  if (d == DV && G == GV)                                                                    \
    return launch_h2o_t<DV, GV>((const u16*)q_all, (const u16*)K, U, (int)n, P, lse2, scores, s);
  GRKV_H2O(64, 1) GRKV_H2O(64, 2) GRKV_H2O(64, 4) GRKV_H2O(64, 8)
  GRKV_H2O(128, 1) GRKV_H2O(128, 2) GRKV_H2O(128, 4) GRKV_H2O(128, 8)
#undef GRKV_H2O
  return hipErrorInvalidValue;
}

}  // namespace grkv
