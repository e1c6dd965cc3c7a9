// Carrier-concentration diagnostics of a local merge rule (App. B,
// "Quantitative Carrier Concentration"; Sec. 1 on span boundaries): every
// evicted token is assigned to the retained token whose key has the highest
// cosine similarity with its own (the key-similarity matching of D2O/KVMerger),
// and the loads a_i of the retained slots are summarised per unit.
//
// match_kernel: a block takes 256 consecutive cache positions of one unit (one
// wave per 32 of them) and streams the unit's retained keys through LDS in
// tiles of 64, gathered through idx; the inverse norm of each retained key is
// formed while the tile is staged.  S = K_q K_ret^T runs on the bf16 MFMA
// (exact products, fp32 sums); a lane keeps, for each of its 8 rows, the best
// (S / ||k_i||, slot) over the keys it sees, in increasing slot order, and the
// 16 lanes that share a row settle the row at the end (equal values go to the
// lower slot).  Scaling by 1 / ||k_j|| is left out: it does not change the
// argmax.  Retained positions get -1.
// stats_kernel: one block per unit; loads by LDS atomics, then b, b_eff, A_max,
// the Gini coefficient (exact integer sum of |a_i - a_j| over all pairs), and
// the boundary-carrier figures.
#include <math.h>

#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

constexpr int kMatchWaves = 8;
constexpr int kMatchRows = 32 * kMatchWaves;   // cache positions per block
constexpr int kRetTile = 64;                   // retained keys per LDS tile

template <int D>
__global__ __launch_bounds__(kMatchWaves * 64) void match_kernel(
    const u16* __restrict__ K, const int32_t* __restrict__ idx, int64_t n, int c,
    int32_t* __restrict__ assign) {
  constexpr int NTH = kMatchWaves * 64;
  constexpr int KS = D + 8;                      // LDS row stride (bf16)
  constexpr int CH = kRetTile * D / 8;           // 16-byte chunks of a tile
  constexpr int PER = (CH + NTH - 1) / NTH;
  constexpr int CPR = D / 8;                     // chunks per key row
  __shared__ __attribute__((aligned(16))) u16 kt_s[2][kRetTile * KS];
  __shared__ float inv_s[2][kRetTile];
  const int u = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g = lane >> 4;
  const u16* Ku = K + (size_t)u * n * D;
  const int32_t* iu = idx + (size_t)u * c;
  const int64_t r0 = (int64_t)blockIdx.x * kMatchRows + 32 * wave;   // this wave's first row

  // query rows of this wave: rows r0 + 16 rt + l16, k = 32 ks + 8 g ..
  uint4 qa[2][D / 32];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int64_t r = min(r0 + 16 * rt + l16, n - 1);
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
      qa[rt][ks] = *reinterpret_cast<const uint4*>(Ku + (size_t)r * D + ks * 32 + 8 * g);
  }

  // register-staged retained tiles; chunk e of tile t: key t*64 + e / CPR
  uint4 reg[PER];
  auto load = [&](int t) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = min(tid + k * NTH, CH - 1);
      const int slot = min(t * kRetTile + e / CPR, c - 1);
      reg[k] = *reinterpret_cast<const uint4*>(Ku + (size_t)iu[slot] * D + (e % CPR) * 8);
    }
  };
  auto store = [&](int t, int buf) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + k * NTH;
      const int key = e / CPR, ch = e % CPR;
      float ss = 0.f;
      if (e < CH) {
        *reinterpret_cast<uint4*>(&kt_s[buf][key * KS + ch * 8]) = reg[k];
        const uint32_t w4[4] = {reg[k].x, reg[k].y, reg[k].z, reg[k].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float a = __uint_as_float(w4[q] << 16), b = __uint_as_float(w4[q] & 0xffff0000u);
          ss = fmaf(a, a, fmaf(b, b, ss));
        }
      }
      // the CPR chunks of a key sit in CPR consecutive lanes
#pragma unroll
      for (int off = 1; off < CPR; off <<= 1) ss += __shfl_xor(ss, off);
      if (e < CH && ch == 0) {
        const bool live = t * kRetTile + key < c;
        inv_s[buf][key] = (live && ss > 0.f) ? 1.f / sqrtf(ss) : 0.f;
      }
    }
  };

  float best[2][4];
  int bslot[2][4];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      best[rt][i] = -__builtin_huge_valf();
      bslot[rt][i] = 0;
    }

  const int ntiles = (c + kRetTile - 1) / kRetTile;
  load(0);
  store(0, 0);
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) load(t + 1);
    __syncthreads();   // tile t is in LDS; tile t-1's buffer is no longer read
#pragma unroll
    for (int kt = 0; kt < kRetTile / 16; ++kt) {
      const int key = 16 * kt + l16;
      f32x4 acc[2] = {zero4(), zero4()};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        const bf16x8 kb = as_bf16x8(*reinterpret_cast<const uint4*>(&kt_s[buf][key * KS + ks * 32 + 8 * g]));
        acc[0] = mfma_bf16(as_bf16x8(qa[0][ks]), kb, acc[0]);
        acc[1] = mfma_bf16(as_bf16x8(qa[1][ks]), kb, acc[1]);
      }
      const int slot = t * kRetTile + key;
      const float inv = inv_s[buf][key];
      const bool live = slot < c;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = acc[rt][i] * inv;
          if (live && v > best[rt][i]) {   // slots rise within a lane: a tie keeps the lower
            best[rt][i] = v;
            bslot[rt][i] = slot;
          }
        }
    }
    if (t + 1 < ntiles) store(t + 1, buf ^ 1);
  }

  // settle each row over the 16 lanes holding it: larger value, then lower slot
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = best[rt][i];
      int sl = bslot[rt][i];
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float ov = __shfl_xor(v, off);
        const int os = __shfl_xor(sl, off);
        if (ov > v || (ov == v && os < sl)) {
          v = ov;
          sl = os;
        }
      }
      const int64_t r = r0 + 16 * rt + 4 * g + i;
      if (l16 == 0 && r < n) {
        // retained position?  idx is ascending: binary search
        int lo = 0, hi = c;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (iu[mid] < r) lo = mid + 1;
          else hi = mid;
        }
        const bool ret = lo < c && iu[lo] == r;
        assign[(size_t)u * n + r] = ret ? -1 : sl;
      }
    }
}

constexpr int kStatsThreads = 1024;
constexpr int kMaxCarrierSlots = 8192;

// metrics [U][8] = {b, b_eff, A_max, Gini, boundary fraction, boundary share,
// enrichment, boundary / interior mean load}
__global__ __launch_bounds__(kStatsThreads) void stats_kernel(
    const int32_t* __restrict__ assign, const int32_t* __restrict__ idx, int64_t n, int c,
    int32_t* __restrict__ counts, float* __restrict__ metrics) {
  __shared__ int cnt[kMaxCarrierSlots];
  __shared__ unsigned long long red[16][6];
  const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* iu = idx + (size_t)u * c;
  for (int i = tid; i < c; i += kStatsThreads) cnt[i] = 0;
  __syncthreads();
  for (int64_t j = tid; j < n; j += kStatsThreads) {
    const int a = assign[(size_t)u * n + j];
    if (a >= 0 && a < c) atomicAdd(&cnt[a], 1);
  }
  __syncthreads();
  // per thread: sum a, sum a^2, max a, active, boundary slots, boundary load,
  // and the pair sum of |a_i - a_j| over its rows i
  unsigned long long s1 = 0, s2 = 0, amax = 0, act = 0, nb = 0, sb = 0, pair = 0;
  for (int i = tid; i < c; i += kStatsThreads) {
    const unsigned long long a = (unsigned long long)cnt[i];
    s1 += a;
    s2 += a * a;
    amax = a > amax ? a : amax;
    act += a > 0;
    const bool first = i == 0 || iu[i - 1] + 1 != iu[i];
    const bool last = i == c - 1 || iu[i] + 1 != iu[i + 1];
    if (first || last) {
      ++nb;
      sb += a;
    }
    if (counts) counts[(size_t)u * c + i] = (int32_t)a;
    for (int j = 0; j < c; ++j) {
      const int dlt = cnt[i] - cnt[j];
      pair += (unsigned long long)(dlt < 0 ? -dlt : dlt);
    }
  }
  unsigned long long v[6] = {s1, s2, act, nb, sb, pair};
  for (int off = 32; off > 0; off >>= 1) {
#pragma unroll
    for (int k = 0; k < 6; ++k) v[k] += __shfl_xor(v[k], off);
    const unsigned long long om = __shfl_xor(amax, off);
    amax = om > amax ? om : amax;
  }
  __shared__ unsigned long long redmax[16];
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < 6; ++k) red[wave][k] = v[k];
    redmax[wave] = amax;
  }
  __syncthreads();
  if (tid == 0) {
    unsigned long long t[6] = {0, 0, 0, 0, 0, 0}, mx = 0;
    for (int w = 0; w < kStatsThreads / 64; ++w) {
      for (int k = 0; k < 6; ++k) t[k] += red[w][k];
      mx = redmax[w] > mx ? redmax[w] : mx;
    }
    const double tot = (double)t[0], cc = (double)c;
    const float nanf_ = __builtin_nanf("");
    float m[8];
    m[0] = (float)t[2];
    m[4] = (float)((double)t[3] / cc);
    if (t[0] > 0) {
      m[1] = (float)(tot * tot / (double)t[1]);
      m[2] = (float)((double)mx / (tot / cc));
      m[3] = (float)((double)t[5] / (2.0 * cc * tot));
      const double share = (double)t[4] / tot;
      m[5] = (float)share;
      m[6] = (float)(share / ((double)t[3] / cc));
      const double ni = cc - (double)t[3];
      if (t[3] > 0 && ni > 0) {
        const double mi = (tot - (double)t[4]) / ni;
        m[7] = mi > 0 ? (float)(((double)t[4] / (double)t[3]) / mi) : __builtin_huge_valf();
      } else {
        m[7] = nanf_;
      }
    } else {
      m[1] = m[2] = m[3] = m[5] = m[6] = m[7] = nanf_;
    }
    for (int k = 0; k < 8; ++k) metrics[(size_t)u * 8 + k] = m[k];
  }
}

// L_common = sum_u D_after_u ||Y_u||^2 / sum_u ||Y_u||^2 from the stats of a
// grkv_compress call (one block, fixed summation order).
__global__ __launch_bounds__(256) void lcommon_kernel(const float* __restrict__ stats, int U,
                                                      float* __restrict__ out) {
  __shared__ double rn[4], rd[4];
  const int tid = threadIdx.x;
  double num = 0, den = 0;
  for (int u = tid; u < U; u += 256) {
    num += (double)stats[u * 4 + 2] * stats[u * 4 + 0];
    den += (double)stats[u * 4 + 0];
  }
  for (int off = 32; off > 0; off >>= 1) {
    num += __shfl_xor(num, off);
    den += __shfl_xor(den, off);
  }
  if ((tid & 63) == 0) {
    rn[tid >> 6] = num;
    rd[tid >> 6] = den;
  }
  __syncthreads();
  if (tid == 0) {
    double a = 0, b = 0;
    for (int k = 0; k < 4; ++k) { a += rn[k]; b += rd[k]; }
    out[0] = b > 0 ? (float)(a / b) : 0.f;
  }
}

}  // namespace

bool carrier_supported(int dtype, int d, int c) {
  return dtype == GRKV_BF16 && (d == 64 || d == 128) && c >= 1 && c <= kMaxCarrierSlots;
}

hipError_t launch_carrier(const void* K, const int32_t* idx, int U, int64_t n, int c, int d,
                          const float* stats, int32_t* assign, int32_t* counts, float* metrics,
                          float* l_common, hipStream_t s) {
  const dim3 grid((unsigned)((n + kMatchRows - 1) / kMatchRows), U);
  if (d == 128)
    hipLaunchKernelGGL(match_kernel<128>, grid, dim3(kMatchWaves * 64), 0, s, (const u16*)K, idx,
                       n, c, assign);
  else
    hipLaunchKernelGGL(match_kernel<64>, grid, dim3(kMatchWaves * 64), 0, s, (const u16*)K, idx,
                       n, c, assign);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(stats_kernel, dim3(U), dim3(kStatsThreads), 0, s, assign, idx, n, c, counts,
                     metrics);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (stats && l_common) {
    hipLaunchKernelGGL(lcommon_kernel, dim3(1), dim3(256), 0, s, stats, U, l_common);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace grkv
