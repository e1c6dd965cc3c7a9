// Token scores of H2O, the token-based eviction method GRKV is paired with
// (Sec. 2: heavy hitters kept by accumulated attention scores; Sec. 4.3,
// compatibility).  A prefix token's score is the attention it receives,
// summed over every prompt position of every query head of its KV head's
// group, each row being the causal softmax of q_i K^T / sqrt(d) over keys
// 0..i:
//   s_j = sum_g sum_{i >= j} 2^(t_{g,i,j} - LSE2_{g,i}),  t = q . k log2(e) / sqrt(d).
// This is the work of a prefill attention without P.V (O(n^2 d) per head),
// done in two MFMA passes with no atomics:
//  * h2o_lse_kernel, one block per (unit, 32 prompt positions) with one wave
//    per query head (two 16-row tiles): streams K tiles 0 .. (last position)
//    through LDS and keeps, per row and lane, an integer reference exponent
//    and an fp64 sum of 2^(t - ref) (as the window's pass A does); the four
//    lanes of a row merge at the end into LSE2 (log2 domain);
//  * h2o_colsum_kernel, one block per (unit, 128 prefix keys) with 4 waves of
//    32 keys (K fragments in registers): streams the query tiles at or after
//    its first key (Q rows and their LSE2 through LDS), forms
//    P = 2^(t - LSE2) under the causal rule and accumulates each key's column
//    sum, in fp32 within a query tile and in fp64 across tiles; a 16-lane
//    reduction at the end gives the key's score.
// The scores then drive grkv_compress_scored (selection with pool width 1).
#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

constexpr int kH2oTQ = 32;          // prompt positions per query tile
constexpr int kH2oKT = 32;          // keys per streamed key tile (LSE pass)
constexpr int kH2oColWaves = 4;
constexpr int kH2oColKeys = 32 * kH2oColWaves;   // keys per column-sum block

// ------------------------------------------------------------ row LSE ----
template <int D, int G>
__global__ __launch_bounds__(G * 64) void h2o_lse_kernel(const u16* __restrict__ q_all,
                                                         const u16* __restrict__ K, int n,
                                                         float scale_log2, float* __restrict__ lse2) {
  constexpr int KS = D + 8;                 // LDS row stride (bf16)
  constexpr int NTH = G * 64;
  constexpr int CH = kH2oKT * D / 8;        // 16-byte chunks of a key tile
  constexpr int PER = (CH + NTH - 1) / NTH;
  __shared__ __attribute__((aligned(16))) u16 kt_s[2][kH2oKT * KS];
  const int u = blockIdx.y, p0 = blockIdx.x * kH2oTQ, tid = threadIdx.x;
  const int lane = tid & 63, g = __builtin_amdgcn_readfirstlane(tid >> 6), l16 = lane & 15, gq = lane >> 4;
  const u16* ku = K + (size_t)u * n * D;
  const u16* qh = q_all + ((size_t)u * G + g) * n * D;

  // the wave's rows: positions p0 + 16 rt + l16 of head g (B operand layout)
  uint4 qb[2][D / 32];
  int pos[2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    pos[rt] = p0 + 16 * rt + l16;
    const int pr = min(pos[rt], n - 1);
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
      qb[rt][ks] = *reinterpret_cast<const uint4*>(qh + (size_t)pr * D + ks * 32 + 8 * gq);
  }
  // keys 0 .. min(n, p0 + 32) - 1 in tiles of 32
  const int kend = min(n, p0 + kH2oTQ);
  const int ntiles = (kend + kH2oKT - 1) / kH2oKT;
  uint4 kr[PER];
  auto load = [&](int t) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = min(tid + k * NTH, CH - 1);
      const int key = min(t * kH2oKT + e / (D / 8), n - 1), ch = e % (D / 8);
      kr[k] = *reinterpret_cast<const uint4*>(ku + (size_t)key * D + ch * 8);
    }
  };
  auto store = [&](u16* dst) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + k * NTH;
      if (e < CH) *reinterpret_cast<uint4*>(dst + (e / (D / 8)) * KS + (e % (D / 8)) * 8) = kr[k];
    }
  };
  float mref[2] = {-__builtin_huge_valf(), -__builtin_huge_valf()};
  double srun[2] = {0.0, 0.0};
  load(0);
  for (int t = 0; t < ntiles; ++t) {
    u16* cur = kt_s[t & 1];
    store(cur);
    __syncthreads();
    if (t + 1 < ntiles) load(t + 1);
    float tv[2][2][4];   // [rt][kt][i]: key 32t + 16kt + 4gq + i, row 16rt + l16
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      uint4 kf[D / 32];
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks)
        kf[ks] = *reinterpret_cast<const uint4*>(cur + (16 * kt + l16) * KS + ks * 32 + 8 * gq);
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) acc = mfma_bf16(as_bf16x8(kf[ks]), as_bf16x8(qb[rt][ks]), acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = t * kH2oKT + 16 * kt + 4 * gq + i;
          tv[rt][kt][i] = (key <= pos[rt] && key < n) ? acc[i] * scale_log2 : -__builtin_huge_valf();
        }
      }
    }
    constexpr float NINF = -__builtin_huge_valf();
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      // masked keys add nothing (and never meet a -inf reference)
      float a = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          a += tv[rt][kt][i] != NINF ? __builtin_amdgcn_exp2f(tv[rt][kt][i] - mref[rt]) : 0.f;
      // a new reference when the tile's sum leaves [0, 2^64] (also taken on the
      // lane's first visible key, while the reference is still -inf)
      if (!(a <= 0x1p64f)) {
        float mx = NINF;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) mx = fmaxf(mx, tv[rt][kt][i]);
        const float ref = ceilf(mx);   // finite: a was not 0, so a key is visible
        srun[rt] = mref[rt] == NINF ? 0.0 : ldexp(srun[rt], (int)(mref[rt] - ref));
        mref[rt] = ref;
        a = 0.f;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            a += tv[rt][kt][i] != NINF ? __builtin_amdgcn_exp2f(tv[rt][kt][i] - ref) : 0.f;
      }
      srun[rt] += (double)a;
    }
    __syncthreads();   // the next store overwrites the other buffer only; this
                       // one is rewritten two tiles later
  }
  // merge the four lanes of each row (exact power-of-two rescales)
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const float M = max_over_groups(mref[rt]);
    const double part = mref[rt] == -__builtin_huge_valf() ? 0.0 : ldexp(srun[rt], (int)(mref[rt] - M));
    const double tot = sum_over_groups(part);
    if (gq == 0 && pos[rt] < n)
      lse2[((size_t)u * G + g) * n + pos[rt]] = (float)((double)M + log2(tot));
  }
}

// --------------------------------------------------------- column sums ----
template <int D, int G>
__global__ __launch_bounds__(kH2oColWaves * 64) void h2o_colsum_kernel(
    const u16* __restrict__ q_all, const u16* __restrict__ K, const float* __restrict__ lse2,
    int n, int P, float scale_log2, float* __restrict__ scores) {
  constexpr int QS = D + 8;                  // LDS row stride (bf16) of Q rows
  constexpr int NR = G * kH2oTQ;             // rows of a query tile (head-major)
  constexpr int NTH = kH2oColWaves * 64;
  constexpr int CH = NR * D / 8;             // 16-byte chunks of a query tile
  constexpr int PER = (CH + NTH - 1) / NTH;
  __shared__ __attribute__((aligned(16))) u16 q_s[2][NR * QS];
  __shared__ float l_s[2][NR];
  const int u = blockIdx.y, k0 = blockIdx.x * kH2oColKeys, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, gq = lane >> 4;
  const u16* ku = K + (size_t)u * n * D;
  const u16* qu = q_all + (size_t)u * G * n * D;
  const float* lu = lse2 + (size_t)u * G * n;

  // this wave's 32 keys (two 16-key tiles) as A operands
  const int kb = k0 + 32 * wave;
  uint4 kf[2][D / 32];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt) {
    const int key = min(kb + 16 * kt + l16, n - 1);
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
      kf[kt][ks] = *reinterpret_cast<const uint4*>(ku + (size_t)key * D + ks * 32 + 8 * gq);
  }
  // query tiles at or after the block's first key
  const int qt0 = k0 / kH2oTQ, qt1 = (n + kH2oTQ - 1) / kH2oTQ;
  uint4 qr[PER];
  float lr = 0.f;
  auto load = [&](int qt) {
    const int p0 = qt * kH2oTQ;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = min(tid + k * NTH, CH - 1);
      const int row = e / (D / 8), ch = e % (D / 8);
      const int hg = row / kH2oTQ, pos = min(p0 + row % kH2oTQ, n - 1);
      qr[k] = *reinterpret_cast<const uint4*>(qu + ((size_t)hg * n + pos) * D + ch * 8);
    }
    if (tid < NR) {
      const int hg = tid / kH2oTQ, pos = p0 + tid % kH2oTQ;
      lr = pos < n ? lu[(size_t)hg * n + pos] : 0.f;
    }
  };
  auto store = [&](int b) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + k * NTH;
      if (e < CH) *reinterpret_cast<uint4*>(&q_s[b][(e / (D / 8)) * QS + (e % (D / 8)) * 8]) = qr[k];
    }
    if (tid < NR) l_s[b][tid] = lr;
  };
  double col[2][4] = {{0.0, 0.0, 0.0, 0.0}, {0.0, 0.0, 0.0, 0.0}};
  if (qt0 < qt1) load(qt0);
  for (int qt = qt0; qt < qt1; ++qt) {
    const int b = (qt - qt0) & 1;
    store(b);
    __syncthreads();
    if (qt + 1 < qt1) load(qt + 1);
    const int p0 = qt * kH2oTQ;
    float part[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int rt = 0; rt < 2 * G; ++rt) {
      // rows 16 rt .. : head rt / 2, positions p0 + 16 (rt % 2) + l16
      uint4 qf[D / 32];
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks)
        qf[ks] = *reinterpret_cast<const uint4*>(&q_s[b][(16 * rt + l16) * QS + ks * 32 + 8 * gq]);
      const int rpos = p0 + 16 * (rt & 1) + l16;
      const float nl = -l_s[b][16 * rt + l16];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) acc = mfma_bf16(as_bf16x8(kf[kt][ks]), as_bf16x8(qf[ks]), acc);
        // lane: key kb + 16 kt + 4 gq + i, row (head rt / 2, position rpos)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kb + 16 * kt + 4 * gq + i;
          const float x = __builtin_amdgcn_exp2f(fmaf(acc[i], scale_log2, nl));
          part[kt][i] += (rpos < n && key <= rpos) ? x : 0.f;
        }
      }
    }
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) col[kt][i] += (double)part[kt][i];
    __syncthreads();   // the tile in buffer b is read before it is rewritten
  }
  // sum over the 16 lanes (rows) sharing each key, in fp64
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
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
}

template <int D, int G>
hipError_t launch_h2o_t(const u16* q_all, const u16* K, int U, int n, int P, float* lse2,
                        float* scores, hipStream_t s) {
  const float scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  hipLaunchKernelGGL((h2o_lse_kernel<D, G>), dim3((n + kH2oTQ - 1) / kH2oTQ, U), dim3(G * 64), 0,
                     s, q_all, K, n, scale_log2, lse2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || P < 1) return e;
  hipLaunchKernelGGL((h2o_colsum_kernel<D, G>), dim3((P + kH2oColKeys - 1) / kH2oColKeys, U),
                     dim3(kH2oColWaves * 64), 0, s, q_all, K, lse2, n, P, scale_log2, scores);
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
