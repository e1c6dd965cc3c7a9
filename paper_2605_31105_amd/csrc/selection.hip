// SnapKV-style span retention for each unit, one 1024-thread block per unit:
//   1. pooling: p_j = sum_{t=j-h}^{j+h} s_t over the prefix (zero outside),
//      summed left to right;
//   2. radix select (4 passes of 8 bits on the fp32 bit patterns, which order
//      like the values since p >= 0) of the (c-w)-th and of the
//      floor(beta*c)-th largest pooled score;
//   3. compaction in ascending position order: every prefix position above
//      the threshold, plus the lowest-position ones equal to it until the
//      count is met (ties go to the lower position), then the w window
//      positions; the fixed flag marks sinks, window tokens and the top
//      floor(beta*c) selections.
// Then the gather of the retained K rows (bit-exact copy), of V0 in the input
// type for the retained-cache passes, and of V0 in fp32 into v_out.
#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

struct SelK {
  const float* colsum;
  float* pooled;
  int32_t* idx;
  uint8_t* fixed;
  int prefix, c, w, h, s_sel, n_top, n_sink, fix_window;
  int64_t n;
  const RagUnit* rag;   // ragged budgets, or null (every unit keeps c)
};

// Budget, selection count, fixed-subset count and first output slot of unit u.
struct UnitSel {
  int c, s_sel, n_top;
  size_t base;
};
__device__ __forceinline__ UnitSel unit_sel(const SelK& a, int u) {
  UnitSel r;
  if (a.rag) {
    const RagUnit ru = a.rag[u];
    r.c = ru.c; r.s_sel = ru.c - a.w; r.n_top = ru.ntop; r.base = (size_t)ru.off;
  } else {
    r.c = a.c; r.s_sel = a.s_sel; r.n_top = a.n_top; r.base = (size_t)u * a.c;
  }
  return r;
}

constexpr uint32_t kBandUlps = 16;
constexpr uint32_t kBandCap = 1024;

// ---------------------------------------------------------------------------
// Selection for prefixes too long for registers (or pools too wide for the
// register kernel), one 1024-thread block per unit, the pooled scores held in
// global memory (a unit's 512 KB at n = 128k stays in the L2 cache).  Every
// sweep over them is block-strided (position j = j0 + q * 1024, coalesced)
// with 16 loads in flight per thread; nothing depends on a thread owning a
// contiguous run of positions:
//  1. pooling, through LDS in rounds of positions;
//  2. both thresholds at once (the (c-w)-th largest pooled score T0 and the
//     floor(beta*c)-th largest T1): each round splits each bracket at 15
//     pivots and counts every key against them in one sweep (no histogram
//     atomics: the scores crowd into a few exponent bins), until at most
//     kLargeCand keys remain inside; those go to LDS and 8-bit radix rounds
//     on their offsets finish;
//  3. the boundary band of each threshold (keys within kBandUlps units in the
//     last place of it) is collected in any order and ranked by the pooled
//     sum recomputed in fp64 from the fp32 column sums, then by position (as
//     the register kernel's refine_boundary does); a band of more than
//     kBandCap keys keeps the fp32 order with ties to the lower positions;
//  4. per segment of 131072 positions: the taken positions are marked in an
//     LDS bitmap (keys above the band, band entries taken, ties taken), and
//     one block scan over the bitmap words writes them in ascending order.
constexpr uint32_t kLargeCand = 4096;
constexpr int kWays = 16;
constexpr int kLoadBatch = 16;
constexpr int kSegBits = 131072;                   // positions per bitmap segment
constexpr int kSegWords = kSegBits / 32;
constexpr int kWordsPerThread = kSegWords / kSelectThreads;

// keys of positions j0 + q * kSelectThreads (a block-strided sweep); keys past
// the end read as 0
__device__ __forceinline__ void load_strided(const float* p, int j0, int P, uint32_t (&k)[kLoadBatch]) {
#pragma unroll
  for (int q = 0; q < kLoadBatch; ++q) {
    const int j = j0 + q * kSelectThreads;
    k[q] = j < P ? __float_as_uint(p[j]) : 0u;
  }
}

// Two k-th largest searches sharing their sweeps.
struct KthWork {
  uint32_t part[kSelectThreads / 64][2 * kWays];
  uint32_t tot[2 * kWays];
  uint32_t hist[256];
  uint32_t sh[4];
  uint32_t ncand[2];
  uint32_t cand[2][kLargeCand];
};

struct Search {
  uint32_t k, lo, hi, clo, chi;   // lo <= T < hi, clo = count(>= lo) >= k > count(>= hi) = chi
  bool on;
  __device__ __forceinline__ bool wide() const { return on && hi - lo > 1 && clo - chi > kLargeCand; }
};

__device__ __forceinline__ uint32_t wave_sum_u(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += (uint32_t)__shfl_xor((int)v, off);
  return v;
}

// Radix rounds over the candidates of one search (8-bit offsets in the bracket).
__device__ void radix_finish(Search& b, const uint32_t* cand, uint32_t L, KthWork& wk) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
#pragma unroll 1
  for (int it = 0; it < 5 && b.hi - b.lo > 1; ++it) {
    const uint32_t width = b.hi - b.lo;
    const int bits = 32 - __builtin_clz(width - 1);   // width - 1 < 2^bits
    const int shift = bits > 8 ? bits - 8 : 0;
    if (tid < 256) wk.hist[tid] = 0u;
    __syncthreads();
    for (uint32_t e = tid; e < L; e += kSelectThreads) {
      const uint32_t x = cand[e];
      if (x >= b.lo && x < b.hi) atomicAdd(&wk.hist[(x - b.lo) >> shift], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      // lane l holds bins 4l .. 4l+3; counts of keys at or above each bin
      uint32_t h4[4], suf = 0;
#pragma unroll
      for (int i = 3; i >= 0; --i) {
        h4[i] = wk.hist[4 * lane + i];
        suf += h4[i];
      }
      uint32_t incl = suf;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t t = (uint32_t)__shfl_down((int)incl, off);
        if (lane + off < 64) incl += t;
      }
      uint32_t above = b.chi + incl - suf;
      int best = -1;
      uint32_t bc = 0, bh = 0;
#pragma unroll
      for (int i = 3; i >= 0; --i) {
        const uint32_t c = above + h4[i];
        if (best < 0 && c >= b.k) { best = 4 * lane + i; bc = c; bh = above; }
        above = c;
      }
      const uint64_t hit = __ballot(best >= 0);
      const int owner = 63 - __builtin_clzll(hit);
      if (lane == owner) {
        const uint32_t nl = b.lo + ((uint32_t)best << shift);
        const uint64_t nh = (uint64_t)b.lo + ((uint64_t)(best + 1) << shift);
        wk.sh[0] = nl;
        wk.sh[1] = nh < b.hi ? (uint32_t)nh : b.hi;
        wk.sh[2] = bc;
        wk.sh[3] = bh;
      }
    }
    __syncthreads();
    b.lo = __builtin_amdgcn_readfirstlane(wk.sh[0]);
    b.hi = __builtin_amdgcn_readfirstlane(wk.sh[1]);
    b.clo = __builtin_amdgcn_readfirstlane(wk.sh[2]);
    b.chi = __builtin_amdgcn_readfirstlane(wk.sh[3]);
    __syncthreads();
  }
}

// A first bracket for each search from a sample of the keys: every stride-th
// key (kSample of them at most, the rest key 0), eight per thread in
// registers; the samples about 4 sqrt(r) + 16 ranks either side of rank
// r = k / stride bound T, found by one joint bisection of the four order
// statistics (counts of two of them packed per word, one barrier per step).
// One sweep then counts the keys at or above both bounds of both searches
// exactly; a bracket is taken only when it provably holds T
// (count(>= lo) >= k > count(>= hi)), so a poor sample costs that sweep and
// the searches start from the full range as before.
constexpr int kSample = 2 * kLargeCand;
constexpr int kSamplePer = kSample / kSelectThreads;

__device__ void sampled_bracket(const float* p, int P, Search (&b)[2], KthWork& wk) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int NW = kSelectThreads / 64;
  static_assert(kSample % kSelectThreads == 0 && kSample < 65536, "packed 16-bit counts");
  const int stride = (P + kSample - 1) / kSample;   // >= 1
  const int ns = (P + stride - 1) / stride;         // real samples
  uint32_t sv[kSamplePer];
#pragma unroll
  for (int m = 0; m < kSamplePer; ++m) {
    const int i = tid + m * kSelectThreads;
    const int64_t j = min((int64_t)i * stride, (int64_t)P - 1);
    const uint32_t x = __float_as_uint(p[j]);
    sv[m] = i < ns ? x : 0u;
  }
  // targets 2t (rank jh: the bound above T) and 2t + 1 (rank jl: below T)
  int J[4];
  bool act[4];
  uint32_t lo[2], hi[2];
  bool try_[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    lo[t] = b[t].lo;
    hi[t] = b[t].hi;
    const bool w = b[t].wide();
    const int r = w ? (int)(b[t].k / (uint32_t)stride) : 0;
    const int delta = 4 * (int)sqrtf((float)r) + 16;
    J[2 * t] = r - delta;
    J[2 * t + 1] = r + delta;
    act[2 * t] = w && r - delta >= 0;
    act[2 * t + 1] = w && r + delta < ns;
    try_[t] = act[2 * t] || act[2 * t + 1];
  }
  // the J-th largest sample (0-based) is the largest x with count(>= x) > J:
  // L keeps count(>= L) > J, H count(>= H) <= J (key 0 counts every sample)
  uint32_t L[4], H[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { L[i] = 0u; H[i] = 0x7F800001u; }
  int parity = 0;
#pragma unroll 1
  for (int it = 0; it < 32; ++it) {
    bool more = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) more |= act[i] && H[i] - L[i] > 1;
    if (!more) break;   // uniform
    uint32_t mid[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) mid[i] = L[i] + (H[i] - L[i]) / 2;
    uint32_t c01 = 0, c23 = 0;
#pragma unroll
    for (int m = 0; m < kSamplePer; ++m) {
      c01 += (uint32_t)(sv[m] >= mid[0]) + ((uint32_t)(sv[m] >= mid[1]) << 16);
      c23 += (uint32_t)(sv[m] >= mid[2]) + ((uint32_t)(sv[m] >= mid[3]) << 16);
    }
    c01 = wave_sum_u(c01);
    c23 = wave_sum_u(c23);
    if (lane == 0) { wk.part[wave][2 * parity] = c01; wk.part[wave][2 * parity + 1] = c23; }
    __syncthreads();
    uint32_t t01 = 0, t23 = 0;
#pragma unroll
    for (int q = 0; q < NW; ++q) { t01 += wk.part[q][2 * parity]; t23 += wk.part[q][2 * parity + 1]; }
    parity ^= 1;   // (the other pair of words next step: one barrier per step)
    const uint32_t cnt[4] = {t01 & 0xFFFFu, t01 >> 16, t23 & 0xFFFFu, t23 >> 16};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (!(act[i] && H[i] - L[i] > 1)) continue;
      if (cnt[i] > (uint32_t)J[i]) L[i] = mid[i];
      else H[i] = mid[i];
    }
  }
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    if (act[2 * t]) hi[t] = __builtin_amdgcn_readfirstlane(L[2 * t]);
    if (act[2 * t + 1]) lo[t] = __builtin_amdgcn_readfirstlane(L[2 * t + 1]);
    if (!(lo[t] < hi[t])) try_[t] = false;
  }
  __syncthreads();   // the last step's words are read before part is reused
  if (!try_[0] && !try_[1]) return;
  uint32_t cl[2] = {0u, 0u}, ch[2] = {0u, 0u};
  for (int j0 = tid; j0 < P; j0 += kLoadBatch * kSelectThreads) {
    uint32_t kk[kLoadBatch];
    load_strided(p, j0, P, kk);
#pragma unroll
    for (int q = 0; q < kLoadBatch; ++q) {
      const bool in = j0 + q * kSelectThreads < P;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        cl[t] += in && kk[q] >= lo[t];
        ch[t] += in && kk[q] >= hi[t];
      }
    }
  }
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const uint32_t x = wave_sum_u(cl[t]), y = wave_sum_u(ch[t]);
    if (lane == 0) { wk.part[wave][2 * t] = x; wk.part[wave][2 * t + 1] = y; }
  }
  __syncthreads();
  if (tid < 4) {
    uint32_t v = 0;
    for (int q = 0; q < NW; ++q) v += wk.part[q][tid];
    wk.tot[tid] = v;
  }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const uint32_t clo = wk.tot[2 * t], chi = wk.tot[2 * t + 1];
    if (try_[t] && clo >= b[t].k && chi < b[t].k) {
      b[t].lo = __builtin_amdgcn_readfirstlane(lo[t]);
      b[t].hi = __builtin_amdgcn_readfirstlane(hi[t]);
      b[t].clo = __builtin_amdgcn_readfirstlane(clo);
      b[t].chi = __builtin_amdgcn_readfirstlane(chi);
    }
  }
  __syncthreads();   // part and tot are reused
}

// The k-th largest keys of both searches (each found exactly: T = lo).
__device__ void kth_pair(const float* p, int P, Search (&b)[2], KthWork& wk) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int NW = kSelectThreads / 64;
  if (b[0].wide() || b[1].wide()) sampled_bracket(p, P, b, wk);
#pragma unroll 1
  while (b[0].wide() || b[1].wide()) {
    uint32_t piv[2][kWays - 1], cnt[2][kWays - 1];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const uint32_t width = b[t].hi - b[t].lo;
      const uint32_t step = width / kWays + (width % kWays ? 1u : 0u);   // >= 1
#pragma unroll
      for (int w = 0; w < kWays - 1; ++w) {
        const uint64_t pv = (uint64_t)b[t].lo + (uint64_t)(w + 1) * step;
        piv[t][w] = pv < b[t].hi ? (uint32_t)pv : b[t].hi;
        cnt[t][w] = 0u;
      }
    }
    for (int j0 = tid; j0 < P; j0 += kLoadBatch * kSelectThreads) {
      uint32_t kk[kLoadBatch];
      load_strided(p, j0, P, kk);
#pragma unroll
      for (int q = 0; q < kLoadBatch; ++q) {
        const bool in = j0 + q * kSelectThreads < P;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int w = 0; w < kWays - 1; ++w) cnt[t][w] += in && kk[q] >= piv[t][w];
      }
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int w = 0; w < kWays - 1; ++w) {
        const uint32_t v = wave_sum_u(cnt[t][w]);
        if (lane == 0) wk.part[wave][t * kWays + w] = v;
      }
    __syncthreads();
    if (tid < 2 * kWays) {
      uint32_t t = 0;
      for (int q = 0; q < NW; ++q) t += wk.part[q][tid];
      wk.tot[tid] = t;
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (!b[t].wide()) continue;
      // the largest pivot whose count still reaches k bounds T from below
      // (pivot counts do not increase with w); no pivot reaching k means
      // T < piv[0]
      uint32_t nlo = b[t].lo, nclo = b[t].clo, nhi = piv[t][0], nchi = wk.tot[t * kWays];
#pragma unroll
      for (int w = 0; w < kWays - 1; ++w) {
        const uint32_t cw = wk.tot[t * kWays + w];
        if (cw >= b[t].k) {
          nlo = piv[t][w];
          nclo = cw;
          if (w + 1 < kWays - 1) {
            nhi = piv[t][w + 1];
            nchi = wk.tot[t * kWays + w + 1];
          } else {
            nhi = b[t].hi;
            nchi = b[t].chi;
          }
        }
      }
      b[t].lo = __builtin_amdgcn_readfirstlane(nlo);
      b[t].clo = __builtin_amdgcn_readfirstlane(nclo);
      b[t].hi = __builtin_amdgcn_readfirstlane(nhi);
      b[t].chi = __builtin_amdgcn_readfirstlane(nchi);
    }
    __syncthreads();   // part and tot are rewritten next round
  }
  // candidates of both brackets into LDS (in any order: only values matter)
  if (tid < 2) wk.ncand[tid] = 0u;
  __syncthreads();
  const bool need0 = b[0].on && b[0].hi - b[0].lo > 1, need1 = b[1].on && b[1].hi - b[1].lo > 1;
  if (need0 || need1) {
    for (int j0 = tid; j0 < P; j0 += kLoadBatch * kSelectThreads) {
      uint32_t kk[kLoadBatch];
      load_strided(p, j0, P, kk);
#pragma unroll
      for (int q = 0; q < kLoadBatch; ++q) {
        if (j0 + q * kSelectThreads >= P) continue;
        if (need0 && kk[q] >= b[0].lo && kk[q] < b[0].hi) {
          const uint32_t o = atomicAdd(&wk.ncand[0], 1u);
          if (o < kLargeCand) wk.cand[0][o] = kk[q];
        }
        if (need1 && kk[q] >= b[1].lo && kk[q] < b[1].hi) {
          const uint32_t o = atomicAdd(&wk.ncand[1], 1u);
          if (o < kLargeCand) wk.cand[1][o] = kk[q];
        }
      }
    }
  }
  __syncthreads();
  if (need0) radix_finish(b[0], wk.cand[0], min(wk.ncand[0], kLargeCand), wk);
  if (need1) radix_finish(b[1], wk.cand[1], min(wk.ncand[1], kLargeCand), wk);
}

// Boundary band of one threshold: its entries (unordered), their fp64 pooled
// sums and take flags.
struct BandSet {
  uint32_t n;                 // keys inside [lo, hi] (may exceed kBandCap: "big")
  uint32_t nabove, ngt;       // count(> hi), count(> T)
  int32_t pos[kBandCap];
  double v64[kBandCap];
  uint32_t take[kBandCap];
};

__device__ __forceinline__ uint32_t band_lo(uint32_t T) { return T > kBandUlps ? T - kBandUlps : 0u; }
__device__ __forceinline__ uint32_t band_hi(uint32_t T) {
  return T < 0x7F800000u - kBandUlps ? T + kBandUlps : 0x7F800000u;
}

__global__ __launch_bounds__(kSelectThreads) void select_kernel(SelK a) {
  __shared__ BandSet band[2];
  __shared__ KthWork wk;
  __shared__ uint32_t bits[3][kSegWords];   // taken (T0), taken (T1), ties at T (big band)
  __shared__ uint32_t scan_scratch[16];
  __shared__ uint32_t mm[2][kSelectThreads / 64];
  __shared__ uint32_t cnt_sh[4];
  float* stage = reinterpret_cast<float*>(&bits[0][0]);   // pooling staging (48 KB)
  constexpr int kStageFloats = 3 * kSegWords;

  const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int P = a.prefix;
  const float* s = a.colsum + (size_t)u * P;
  float* p = a.pooled + (size_t)u * P;
  const UnitSel us = unit_sel(a, u);
  int32_t* idx = a.idx + us.base;
  uint8_t* fixed = a.fixed + us.base;

  // 1. pooling, summed left to right; through LDS in rounds of CH outputs when
  // the window fits beside them, straight from global memory otherwise
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  const int h = a.h;
  const int CH = kStageFloats - 2 * h >= 2048 ? min(16384, kStageFloats - 2 * h) : 0;
  if (CH > 0) {
    // a round's CH + 2h scores fit one batch of kLoadBatch per thread; the
    // next round's are loaded (clamped into the prefix, masked) while this
    // round pools
    static_assert(kStageFloats <= kLoadBatch * kSelectThreads, "one load batch per round");
    float nv[kLoadBatch];
    auto fetch = [&](int base) {
#pragma unroll
      for (int q = 0; q < kLoadBatch; ++q) {
        const int t = tid + q * kSelectThreads, j = base - h + t;
        const uint32_t x = __float_as_uint(s[min(max(j, 0), P - 1)]);
        // masked with an AND, not a select: a select of a load is turned
        // into a branch around the load, which then waits alone
        const uint32_t keep = (t < CH + 2 * h && j >= 0 && j < P) ? 0xFFFFFFFFu : 0u;
        nv[q] = __uint_as_float(x & keep);
      }
    };
    fetch(0);
    for (int base = 0; base < P; base += CH) {
      __syncthreads();
#pragma unroll
      for (int q = 0; q < kLoadBatch; ++q) {
        const int t = tid + q * kSelectThreads;
        if (t < CH + 2 * h) stage[t] = nv[q];
      }
      __syncthreads();
      if (base + CH < P) fetch(base + CH);
      for (int q = tid; q < CH && base + q < P; q += kSelectThreads) {
        float acc = 0.f;
        for (int t = 0; t <= 2 * h; ++t) acc += stage[q + t];
        const uint32_t key = __float_as_uint(acc);
        p[base + q] = acc;
        kmin = min(kmin, key);
        kmax = max(kmax, key);
      }
    }
  } else {
    for (int j = tid; j < P; j += kSelectThreads) {
      const int lo = j - h < 0 ? 0 : j - h;
      const int hi = j + h > P - 1 ? P - 1 : j + h;
      float acc = 0.f;
      for (int t0 = lo; t0 <= hi; t0 += 8) {   // eight loads in flight, summed left to right
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = s[min(t0 + i, hi)];
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (t0 + i <= hi) acc += v[i];
      }
      p[j] = acc;
      kmin = min(kmin, __float_as_uint(acc));
      kmax = max(kmax, __float_as_uint(acc));
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, off));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, off));
  }
  if (lane == 0) { mm[0][wave] = kmin; mm[1][wave] = kmax; }
  __syncthreads();   // also: every pooled score is written before the sweeps read them
  kmin = 0xFFFFFFFFu;
  kmax = 0u;
#pragma unroll
  for (int q = 0; q < kSelectThreads / 64; ++q) {
    kmin = min(kmin, mm[0][q]);
    kmax = max(kmax, mm[1][q]);
  }
  kmax = min(kmax, 0x7F800000u);   // +inf at most (no NaN scores)

  // 2. T0 = the (c-w)-th largest, T1 = the floor(beta*c)-th largest
  const bool any[2] = {us.s_sel > 0, us.n_top > 0};
  Search b[2];
  b[0] = {(uint32_t)us.s_sel, kmin, kmax + 1, (uint32_t)P, 0u, any[0]};
  b[1] = {(uint32_t)us.n_top, kmin, kmax + 1, (uint32_t)P, 0u, any[1]};
  kth_pair(p, P, b, wk);
  const uint32_t T[2] = {b[0].lo, b[1].lo};
  const uint32_t lo[2] = {band_lo(T[0]), band_lo(T[1])}, hi[2] = {band_hi(T[0]), band_hi(T[1])};
  const uint32_t kk_[2] = {(uint32_t)us.s_sel, (uint32_t)us.n_top};

  // 3. the boundary bands: entries (unordered), counts above the band and above T
  if (tid < 2) { band[tid].n = 0u; cnt_sh[2 * tid] = 0u; cnt_sh[2 * tid + 1] = 0u; }
  __syncthreads();
  {
    uint32_t nab[2] = {0u, 0u}, ngt[2] = {0u, 0u};
    for (int j0 = tid; j0 < P; j0 += kLoadBatch * kSelectThreads) {
      uint32_t kk[kLoadBatch];
      load_strided(p, j0, P, kk);
#pragma unroll
      for (int q = 0; q < kLoadBatch; ++q) {
        const int j = j0 + q * kSelectThreads;
        if (j >= P) continue;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          if (!any[t]) continue;
          nab[t] += kk[q] > hi[t];
          ngt[t] += kk[q] > T[t];
          if (kk[q] >= lo[t] && kk[q] <= hi[t]) {
            const uint32_t o = atomicAdd(&band[t].n, 1u);
            if (o < kBandCap) band[t].pos[o] = j;
          }
        }
      }
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const uint32_t x = wave_sum_u(nab[t]), y = wave_sum_u(ngt[t]);
      if (lane == 0) { atomicAdd(&cnt_sh[2 * t], x); atomicAdd(&cnt_sh[2 * t + 1], y); }
    }
  }
  __syncthreads();
  bool big[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    band[t].nabove = cnt_sh[2 * t];   // (same value from every thread)
    band[t].ngt = cnt_sh[2 * t + 1];
    big[t] = band[t].n > kBandCap;
  }
  __syncthreads();
  // fp64 pooled sums of the band entries (left to right), then their ranks by
  // (sum descending, position ascending): the first k - nabove are taken
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    if (!any[t] || big[t]) continue;
    for (uint32_t e = tid; e < band[t].n; e += kSelectThreads) {
      const int j = band[t].pos[e];
      const int t0 = j - h < 0 ? 0 : j - h, t1 = j + h > P - 1 ? P - 1 : j + h;
      double acc = 0.0;
      for (int x0 = t0; x0 <= t1; x0 += 8) {   // eight loads in flight, summed left to right
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = s[min(x0 + i, t1)];
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if (x0 + i <= t1) acc += (double)v[i];
      }
      band[t].v64[e] = acc;
    }
  }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    if (!any[t] || big[t]) continue;
    const uint32_t nb = band[t].n, need = kk_[t] - band[t].nabove;
    for (uint32_t e = tid; e < nb; e += kSelectThreads) {
      const double v = band[t].v64[e];
      const int j = band[t].pos[e];
      uint32_t rank = 0;
      for (uint32_t f = 0; f < nb; ++f) {
        const double w = band[t].v64[f];
        rank += w > v || (w == v && band[t].pos[f] < j);
      }
      band[t].take[e] = rank < need;
    }
  }
  __syncthreads();

  // 4. per segment: mark the taken positions, then write them in order
  uint32_t out_before = 0, eq_before[2] = {0u, 0u};
  for (int seg0 = 0; seg0 < P; seg0 += kSegBits) {
    const int seg1 = min(P, seg0 + kSegBits);
    __syncthreads();
    for (int wd = tid; wd < 3 * kSegWords; wd += kSelectThreads) (&bits[0][0])[wd] = 0u;
    __syncthreads();
    for (int t = 0; t < 2; ++t) {
      if (!any[t]) continue;
      // keys above the band (or, for a big band, above T; ties marked apart)
      for (int j0 = seg0 + tid; j0 < seg1; j0 += kLoadBatch * kSelectThreads) {
        uint32_t kk[kLoadBatch];
        load_strided(p, j0, seg1, kk);
#pragma unroll
        for (int q = 0; q < kLoadBatch; ++q) {
          const int j = j0 + q * kSelectThreads;
          if (j >= seg1) continue;
          const int bi = j - seg0;
          if (big[t] ? kk[q] > T[t] : kk[q] > hi[t]) atomicOr(&bits[t][bi >> 5], 1u << (bi & 31));
          if (big[t] && kk[q] == T[t]) atomicOr(&bits[2][bi >> 5], 1u << (bi & 31));
        }
      }
      if (!big[t]) {
        for (uint32_t e = tid; e < band[t].n; e += kSelectThreads) {
          const int j = band[t].pos[e];
          if (band[t].take[e] && j >= seg0 && j < seg1)
            atomicOr(&bits[t][(j - seg0) >> 5], 1u << ((j - seg0) & 31));
        }
        continue;
      }
      // big band: ties at T go to the lowest positions, k - count(> T) of them
      __syncthreads();
      const uint32_t krem = kk_[t] - band[t].ngt;
      uint32_t wv[kWordsPerThread], c = 0;
#pragma unroll
      for (int i = 0; i < kWordsPerThread; ++i) {
        wv[i] = bits[2][tid * kWordsPerThread + i];
        c += __builtin_popcount(wv[i]);
      }
      uint32_t tot;
      uint32_t r = eq_before[t] + block_exclusive_scan(c, scan_scratch, &tot);
#pragma unroll
      for (int i = 0; i < kWordsPerThread; ++i) {
        uint32_t wbits = wv[i], take = 0u;
        while (wbits) {
          const int bpos = __builtin_ctz(wbits);
          if (r < krem) take |= 1u << bpos;
          ++r;
          wbits &= wbits - 1;
        }
        if (take) atomicOr(&bits[t][tid * kWordsPerThread + i], take);
      }
      eq_before[t] += tot;
      __syncthreads();
      for (int wd = tid; wd < kSegWords; wd += kSelectThreads) bits[2][wd] = 0u;
      __syncthreads();   // cleared before the next threshold marks its ties
    }
    __syncthreads();
    // the taken positions of this segment, ascending, with their fixed flags
    uint32_t wv[kWordsPerThread], c = 0;
#pragma unroll
    for (int i = 0; i < kWordsPerThread; ++i) {
      wv[i] = bits[0][tid * kWordsPerThread + i];
      c += __builtin_popcount(wv[i]);
    }
    uint32_t tot;
    uint32_t off = out_before + block_exclusive_scan(c, scan_scratch, &tot);
#pragma unroll
    for (int i = 0; i < kWordsPerThread; ++i) {
      const uint32_t topw = bits[1][tid * kWordsPerThread + i];
      uint32_t wbits = wv[i];
      while (wbits) {
        const int bpos = __builtin_ctz(wbits);
        const int j = seg0 + (tid * kWordsPerThread + i) * 32 + bpos;
        idx[off] = j;
        fixed[off] = (j < a.n_sink || ((topw >> bpos) & 1u)) ? 1 : 0;
        ++off;
        wbits &= wbits - 1;
      }
    }
    out_before += tot;
  }
  for (int i = tid; i < a.w; i += blockDim.x) {
    int64_t pos = a.n - a.w + i;
    idx[us.s_sel + i] = (int32_t)pos;
    fixed[us.s_sel + i] = (a.fix_window || pos < a.n_sink) ? 1 : 0;
  }
}

constexpr int kSmallThreads = 1024;
constexpr int kSmallPer = 32;          // pooled scores per thread: prefixes up to 32768
constexpr uint32_t kCandCap = 4096;    // candidates finished by one wave (64 per lane)

// A value known to be the same in every lane, kept in a scalar register.
__device__ __forceinline__ uint32_t uniform_u(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}

// Sum over the 64 lanes of a wave, in every lane (DPP within 16-lane rows,
// then the four row totals).
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
  int x = (int)v;
  x += __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x140, 0xF, 0xF, false);
  return (uint32_t)(__builtin_amdgcn_readlane(x, 0) + __builtin_amdgcn_readlane(x, 16) +
                    __builtin_amdgcn_readlane(x, 32) + __builtin_amdgcn_readlane(x, 48));
}

// Block-wide sum of one value per thread; `part` holds 2 x 16 words and
// alternates by `parity`, so consecutive calls need one barrier each.
__device__ __forceinline__ uint32_t block_sum_small(uint32_t v, uint32_t (*part)[16], int parity) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) part[parity][threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t tot = 0;
#pragma unroll
  for (int k = 0; k < kSmallThreads / 64; ++k) tot += part[parity][k];
  return uniform_u(tot);
}

// Inclusive prefix sum over the 64 lanes of a wave: DPP shifts within each
// 16-lane row, then the totals of the rows below, read from lanes 15, 31, 47.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  int x = (int)v;
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);   // row_shr:8
  const int row = (threadIdx.x & 63) >> 4;
  const int r0 = __builtin_amdgcn_readlane(x, 15), r1 = __builtin_amdgcn_readlane(x, 31),
            r2 = __builtin_amdgcn_readlane(x, 47);
  x += (row >= 1 ? r0 : 0) + (row >= 2 ? r1 : 0) + (row >= 3 ? r2 : 0);
  return (uint32_t)x;
}

// Exclusive prefix sums over the block of two values per thread, and their
// block totals, with one barrier: `scr` holds 2 x 32 words and alternates by
// `parity` (shared with block_sum_small's), so consecutive calls need no
// second barrier.
__device__ __forceinline__ void block_scan2_small(uint32_t v0, uint32_t v1,
                                                  uint32_t (*scr)[32], int parity,
                                                  uint32_t& e0, uint32_t& e1, uint32_t& t0,
                                                  uint32_t& t1) {
  const uint32_t i0 = wave_incl_scan(v0), i1 = wave_incl_scan(v1);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 63) {
    scr[parity][wave] = i0;
    scr[parity][16 + wave] = i1;
  }
  __syncthreads();
  uint32_t b0 = 0, b1 = 0, a0 = 0, a1 = 0;
#pragma unroll
  for (int k = 0; k < kSmallThreads / 64; ++k) {
    const uint32_t s0 = scr[parity][k], s1 = scr[parity][16 + k];
    b0 += k < wave ? s0 : 0u;
    b1 += k < wave ? s1 : 0u;
    a0 += s0;
    a1 += s1;
  }
  e0 = b0 + i0 - v0;
  e1 = b1 + i1 - v1;
  t0 = uniform_u(a0);
  t1 = uniform_u(a1);
}

// State of one k-th-largest search over the keys (fp32 bit patterns of
// non-negative scores, which order like the values): lo <= T < hi with
// clo = count(>= lo) >= k > count(>= hi) = chi.
struct Bracket {
  uint32_t lo, hi, clo, chi;
};

// Boundary band of one threshold in the small kernel: positions, fp64 sums
// and take flags of its keys (unordered), kBandCap * 16 bytes of LDS.
struct SmallBand {
  double* v64;
  int32_t* pos;
  uint32_t* take;
  __device__ __forceinline__ explicit SmallBand(float* base)
      : v64(reinterpret_cast<double*>(base)),
        pos(reinterpret_cast<int32_t*>(v64 + kBandCap)),
        take(reinterpret_cast<uint32_t*>(pos + kBandCap)) {}
};

// Selection for prefixes of at most 32768 tokens, each thread keeping 32
// consecutive pooled scores in registers.  Both thresholds (the (c-w)-th
// largest score T0 and the floor(beta*c)-th largest T1) are searched
// together, so every block-wide step serves both:
//  * bisection on the bit patterns from the [min, max] bracket, the two
//    counts "score >= mid" packed in one word per reduction, until at most
//    kCandCap keys remain inside each bracket;
//  * those candidates go to LDS, and radix rounds (256 bins of the bit
//    pattern's offset in the bracket, one histogram per search) finish;
//  * the fp32 pooled sums round away differences that decide the order (two
//    overlapping windows share all but their edge terms), so the keys within
//    kBandUlps units in the last place of each threshold are ranked again by
//    their sums recomputed in fp64 from the fp32 column sums, then by
//    position; the keys above the band are taken and the band fills the
//    remaining places.  A band of more than kBandCap keys (scores equal over
//    long runs) keeps the fp32 order with ties to the lower position.
// Per-key work is written without branches (bounds by clamped addresses and
// selects, compaction through per-lane spare slots), since a branch per key
// costs far more than the key's arithmetic.  H = (pool width - 1) / 2 is a
// template argument, so the pooling and the band sums unroll.
constexpr int kSmallWords = kSmallThreads * kSmallPer + kSmallThreads * kSmallPer / 64;
constexpr int kSpare = 2 * kCandCap;          // 64 per-lane spare slots after the candidates
constexpr int kMaskWords = kSpare + 64;       // 2 x 1024 per-thread take masks of the bands

template <int H>
__global__ __launch_bounds__(kSmallThreads) void select_small_kernel(SelK a) {
  __shared__ __attribute__((aligned(16))) float sl[kSmallWords];
  __shared__ uint32_t part[2][16];
  __shared__ uint32_t scr[2][32];
  __shared__ uint32_t sh[2][4];
  __shared__ uint32_t hist[2][256];
  static_assert(kMaskWords + 2 * kSmallThreads <= kSmallWords, "LDS areas");
  static_assert(2 * kBandCap * 4 <= kSpare, "band areas inside the candidate area");
  constexpr int PER = kSmallPer;
  const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int P = a.prefix;
  const float* s = a.colsum + (size_t)u * P;
  float* pg = a.pooled + (size_t)u * P;
  const UnitSel us = unit_sel(a, u);
  int32_t* idx = a.idx + us.base;
  uint8_t* fixed = a.fixed + us.base;
  const int j0 = tid * PER;
  uint32_t* slu = reinterpret_cast<uint32_t*>(sl);
  uint32_t* mw = slu + kMaskWords;   // [2][kSmallThreads]

  if (P > 0) {
  // Scores of the whole prefix into LDS (coalesced), one pad word per 64
  // entries so that the lanes of a wave, each reading its own contiguous
  // run, fall on distinct banks.  Each thread then pools its 32 positions
  // (plus H on either side) in registers, summing s[j-H..j+H] left to right.
  // Positions past the prefix get key 0: they rank after every real position
  // with an equal score and are never taken while real positions are left.
  {
    float ld[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int t = tid + k * kSmallThreads;
      ld[k] = s[min(t, P - 1)];
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int t = tid + k * kSmallThreads;
      sl[t + (t >> 6)] = t < P ? ld[k] : 0.f;
    }
  }
  __syncthreads();
  uint32_t key[PER];
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  {
    float v[PER + 2 * H];
#pragma unroll
    for (int q = 0; q < PER + 2 * H; ++q) {
      const int t = j0 - H + q;
      const int tc = min(max(t, 0), kSmallThreads * PER - 1);
      const float x = sl[tc + (tc >> 6)];
      v[q] = t >= 0 ? x : 0.f;   // past the prefix, sl holds zeros
    }
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int j = j0 + q;
      float acc = 0.f;
#pragma unroll
      for (int t = 0; t <= 2 * H; ++t)   // offsets -H..H in increasing order
        acc += v[q + t];
      key[q] = j < P ? __float_as_uint(acc) : 0u;
      kmin = min(kmin, j < P ? key[q] : 0xFFFFFFFFu);
      kmax = max(kmax, key[q]);
    }
  }

  // key range of the real positions (block min and max); the barrier also
  // ends the pooling reads of sl, which is reused from here on
  {
    uint32_t mn = kmin, mx = kmax;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      mn = min(mn, (uint32_t)__shfl_xor((int)mn, off));
      mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
    }
    if (lane == 0) {
      part[0][wave] = mn;
      part[1][wave] = mx;
    }
    __syncthreads();
    kmin = 0xFFFFFFFFu;
    kmax = 0u;
#pragma unroll
    for (int k = 0; k < kSmallThreads / 64; ++k) {
      kmin = min(kmin, part[0][k]);
      kmax = max(kmax, part[1][k]);
    }
    mw[tid] = 0u;
    mw[kSmallThreads + tid] = 0u;
    __syncthreads();   // part is reused below
  }
  kmin = uniform_u(kmin);
  kmax = uniform_u(min(kmax, 0x7F800000u));   // +inf at most (no NaN scores)
  int parity = 0;

  const uint32_t kk[2] = {(uint32_t)us.s_sel, (uint32_t)us.n_top};
  const bool on[2] = {kk[0] > 0, kk[1] > 0};
  // count(>= kmin) = P (the padding keys, 0, count only when kmin is 0)
  const uint32_t all = kmin > 0 ? (uint32_t)P : (uint32_t)(kSmallThreads * PER);
  Bracket b[2];
  b[0] = b[1] = Bracket{kmin, kmax + 1, all, 0u};
  auto wide = [&](int i) {
    return on[i] && b[i].hi - b[i].lo > 1 && b[i].clo - b[i].chi > kCandCap;
  };
  auto open = [&](int i) { return on[i] && b[i].hi - b[i].lo > 1; };

  // 1. bisection, both searches per reduction (each count <= 32768 < 2^16)
#pragma unroll 1
  for (int it = 0; it < 33 && (wide(0) || wide(1)); ++it) {
    const uint32_t m0 = b[0].lo + (b[0].hi - b[0].lo) / 2;
    const uint32_t m1 = b[1].lo + (b[1].hi - b[1].lo) / 2;
    uint32_t n = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) n += (uint32_t)(key[q] >= m0) + ((uint32_t)(key[q] >= m1) << 16);
    const uint32_t c = block_sum_small(n, part, parity);
    parity ^= 1;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (!wide(i)) continue;
      const uint32_t ci = i ? c >> 16 : c & 0xFFFFu;
      const uint32_t mid = i ? m1 : m0;
      if (ci >= kk[i]) { b[i].lo = mid; b[i].clo = ci; }
      else { b[i].hi = mid; b[i].chi = ci; }
    }
  }

  // 2. the candidates of each open bracket into LDS (at most kCandCap each):
  // a key is inside [lo, hi) when key - lo < hi - lo (unsigned); keys
  // outside go to the lane's spare slot, so the stores need no branch
  uint32_t* cand[2] = {slu, slu + kCandCap};
  uint32_t L[2] = {0u, 0u};
  if (open(0) || open(1)) {
    const uint32_t w0 = open(0) ? b[0].hi - b[0].lo : 0u, w1 = open(1) ? b[1].hi - b[1].lo : 0u;
    uint32_t in0 = 0, in1 = 0;   // bit q: key q inside bracket 0 / 1
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      in0 |= (uint32_t)(key[q] - b[0].lo < w0) << q;
      in1 |= (uint32_t)(key[q] - b[1].lo < w1) << q;
    }
    uint32_t e0, e1, t0, t1;
    block_scan2_small(__builtin_popcount(in0), __builtin_popcount(in1), scr, parity, e0, e1, t0, t1);
    parity ^= 1;
    const uint32_t spare = kSpare + lane;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const uint32_t f0 = (in0 >> q) & 1u, f1 = (in1 >> q) & 1u;
      slu[f0 && e0 < kCandCap ? e0 : spare] = key[q];
      slu[f1 && e1 < kCandCap ? kCandCap + e1 : spare] = key[q];
      e0 += f0;
      e1 += f1;
    }
    L[0] = min(t0, kCandCap);
    L[1] = min(t1, kCandCap);
    __syncthreads();
  }

  // 3. radix rounds on the candidates: 256 bins of (x - lo) >> shift cover
  // [lo, hi); the bin holding the k-th largest becomes the new bracket.  A
  // 32-bit range takes at most four rounds.  Wave i scans histogram i.
#pragma unroll 1
  for (int it = 0; it < 5 && (open(0) || open(1)); ++it) {
    int shift[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t width = b[i].hi - b[i].lo;
      const int bits = width > 1 ? 32 - __builtin_clz(width - 1) : 1;   // width - 1 < 2^bits
      shift[i] = bits > 8 ? bits - 8 : 0;
    }
    if (tid < 512) hist[tid >> 8][tid & 255] = 0u;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (!open(i)) continue;
      const uint32_t wi = b[i].hi - b[i].lo;
      for (uint32_t e = tid; e < L[i]; e += kSmallThreads) {
        const uint32_t x = cand[i][e];
        if (x - b[i].lo < wi) atomicAdd(&hist[i][(x - b[i].lo) >> shift[i]], 1u);
      }
    }
    __syncthreads();
    if (wave < 2 && (wave == 0 ? open(0) : open(1))) {
      const int i = wave;
      const Bracket bi = i ? b[1] : b[0];
      const uint32_t ki = i ? kk[1] : kk[0];
      const int si = i ? shift[1] : shift[0];
      // lane l holds bins 4(63 - l) .. 4(63 - l) + 3, so a prefix sum over
      // the lanes counts the keys at or above each lane's bins
      const int base = 4 * (63 - lane);
      uint32_t h4[4], suf = 0;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        h4[r] = hist[i][base + r];
        suf += h4[r];
      }
      const uint32_t incl = wave_incl_scan(suf);
      uint32_t above = bi.chi + incl - suf;   // keys in higher bins, plus those >= hi
      int best = -1;
      uint32_t bc = 0, bh = 0;
#pragma unroll
      for (int r = 3; r >= 0; --r) {
        const uint32_t c = above + h4[r];
        const bool hit = best < 0 && c >= ki;
        best = hit ? base + r : best;
        bc = hit ? c : bc;
        bh = hit ? above : bh;
        above = c;
      }
      // the lowest lane with a hit (the highest bins) owns the answer
      const uint64_t hit = __ballot(best >= 0);
      const int owner = __builtin_ctzll(hit);
      if (lane == owner) {
        const uint32_t nlo = bi.lo + ((uint32_t)best << si);
        const uint64_t nhi = (uint64_t)bi.lo + ((uint64_t)(best + 1) << si);
        sh[i][0] = nlo;
        sh[i][1] = nhi < bi.hi ? (uint32_t)nhi : bi.hi;
        sh[i][2] = bc;
        sh[i][3] = bh;
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i)
      if (open(i))
        b[i] = Bracket{uniform_u(sh[i][0]), uniform_u(sh[i][1]), uniform_u(sh[i][2]), uniform_u(sh[i][3])};
    // (hist and sh are rewritten after the next round's first barrier)
  }
  const uint32_t T[2] = {b[0].lo, b[1].lo};

  // 4. the boundary bands [blo, bhi] around each threshold: masks of the keys
  // above and inside them, and their counts in one scan
  uint32_t m[2] = {0u, 0u}, inb[2] = {0u, 0u};
  uint32_t eb[2] = {0u, 0u}, tb[2] = {0u, 0u}, need[2] = {0u, 0u};
  {
    uint32_t na[2] = {0u, 0u}, nb[2] = {0u, 0u};
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (!on[i]) continue;
      const uint32_t blo = band_lo(T[i]), bw = band_hi(T[i]) - blo;
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        m[i] |= (uint32_t)(key[q] > blo + bw) << q;
        inb[i] |= (uint32_t)(key[q] - blo <= bw) << q;
      }
      na[i] = __builtin_popcount(m[i]);
      nb[i] = __builtin_popcount(inb[i]);
    }
    uint32_t e0, e1, t0, t1;
    block_scan2_small(na[0] | (na[1] << 16), nb[0] | (nb[1] << 16), scr, parity, e0, e1, t0, t1);
    parity ^= 1;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int sft = 16 * i;
      eb[i] = (e1 >> sft) & 0xFFFFu;
      tb[i] = on[i] ? (t1 >> sft) & 0xFFFFu : 0u;
      need[i] = on[i] ? kk[i] - ((t0 >> sft) & 0xFFFFu) : 0u;   // 1 <= need <= tb
    }
  }
  // bands too wide to rank: fp32 order, ties (key == T) to the lower position
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    if (!on[i] || tb[i] <= kBandCap) continue;
    uint32_t gt = 0, eq = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      gt += key[q] > T[i];
      eq += key[q] == T[i];
    }
    uint32_t e, dummy, tg, teq;
    block_scan2_small(eq, gt, scr, parity, e, dummy, teq, tg);
    parity ^= 1;
    const uint32_t krem = kk[i] - tg;
    uint32_t mm = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const bool take = key[q] > T[i] || (key[q] == T[i] && e < krem);
      e += key[q] == T[i];
      mm |= (uint32_t)take << q;
    }
    m[i] = mm;
  }
  const bool rank0 = on[0] && tb[0] <= kBandCap, rank1 = on[1] && tb[1] <= kBandCap;
  if (rank0 || rank1) {
    const SmallBand band[2] = {SmallBand(sl), SmallBand(sl + kBandCap * 4)};
    const bool rk[2] = {rank0, rank1};
    // band positions (few keys: a loop over the set bits of the band mask)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if (!rk[i]) continue;
      uint32_t o = eb[i], bits = inb[i];
      while (bits) {
        band[i].pos[o++] = j0 + __builtin_ctz(bits);
        bits &= bits - 1;
      }
    }
    __syncthreads();
    // fp64 sums of the band entries, left to right (terms outside the prefix
    // are zero), with all loads of an entry in flight
    const uint32_t n0 = rank0 ? tb[0] : 0u, n1 = rank1 ? tb[1] : 0u;
    for (uint32_t e = tid; e < n0 + n1; e += kSmallThreads) {
      const bool second = e >= n0;
      const uint32_t r = second ? e - n0 : e;
      const SmallBand& bd = second ? band[1] : band[0];
      const int j = bd.pos[r];
      float st[2 * H + 1];
#pragma unroll
      for (int t = -H; t <= H; ++t) st[t + H] = s[min(max(j + t, 0), P - 1)];
      double acc = 0.0;
#pragma unroll
      for (int t = -H; t <= H; ++t)
        acc += (j + t >= 0 && j + t < P) ? (double)st[t + H] : 0.0;
      bd.v64[r] = acc;
    }
    __syncthreads();
    // rank inside the band; the taken entries set their bit in the owning
    // thread's mask word (position j belongs to thread j / 32, bit j % 32)
    for (uint32_t e = tid; e < n0 + n1; e += kSmallThreads) {
      const bool second = e >= n0;
      const uint32_t r = second ? e - n0 : e, nb = second ? n1 : n0;
      const SmallBand& bd = second ? band[1] : band[0];
      const double v = bd.v64[r];
      const int j = bd.pos[r];
      uint32_t rank = 0;
      for (uint32_t f = 0; f < nb; ++f) {
        const double w = bd.v64[f];
        rank += w > v || (w == v && bd.pos[f] < j);
      }
      if (rank < (second ? need[1] : need[0]))
        atomicOr(&mw[(second ? kSmallThreads : 0) + (j >> 5)], 1u << (j & 31));
    }
    __syncthreads();
    if (rank0) m[0] |= mw[tid];
    if (rank1) m[1] |= mw[kSmallThreads + tid];
  }

  // 5. the selected positions in increasing order, through LDS (position,
  // and the fixed-subset flag in bit 31), then stored coalesced
  {
    uint32_t selm = m[0];
    const uint32_t topm = m[1];
    uint32_t off, dummy, tot, tdummy;
    block_scan2_small(__builtin_popcount(selm), 0u, scr, parity, off, dummy, tot, tdummy);
    parity ^= 1;
    while (selm) {
      const int q = __builtin_ctz(selm);
      slu[off++] = (uint32_t)(j0 + q) | (((topm >> q) & 1u) << 31);
      selm &= selm - 1;
    }
    __syncthreads();
    for (uint32_t r = tid; r < (uint32_t)us.s_sel; r += kSmallThreads) {
      const uint32_t v = slu[r];
      const int j = (int)(v & 0x7FFFFFFFu);
      idx[r] = j;
      fixed[r] = (j < a.n_sink || (v >> 31)) ? 1 : 0;
    }
  }

  // 6. the pooled scores (an intermediate the caller may inspect), through
  // LDS so that the stores are coalesced
  __syncthreads();   // the staged positions are no longer read
#pragma unroll
  for (int q = 0; q < PER; ++q) sl[j0 + q + ((j0 + q) >> 6)] = __uint_as_float(key[q]);
  __syncthreads();
  for (int t = tid; t < P; t += kSmallThreads) pg[t] = sl[t + (t >> 6)];
  }   // P > 0

  for (int i = tid; i < a.w; i += kSmallThreads) {
    const int64_t pos = a.n - a.w + i;
    idx[us.s_sel + i] = (int32_t)pos;
    fixed[us.s_sel + i] = (a.fix_window || pos < a.n_sink) ? 1 : 0;
  }
}

template <typename T>
__global__ void gather_kernel(const T* K, const T* V, const int32_t* idx, T* k_out, T* v0c,
                              float* v_out, int c, int64_t n, int D) {
  // one 16-byte chunk of one retained row per thread
  const int u = blockIdx.y;
  const int epc = 16 / (int)sizeof(T);
  const int cpr = D / epc;
  const int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (chunk >= (int64_t)c * cpr) return;
  const int row = (int)(chunk / cpr), cc = (int)(chunk % cpr);
  const int64_t src = idx[(size_t)u * c + row];
  const size_t so = ((size_t)u * n + src) * D + (size_t)cc * epc;
  const size_t dof = ((size_t)u * c + row) * D + (size_t)cc * epc;
  uint4 kv = make_uint4(0, 0, 0, 0), vv = kv;
  if (src >= 0 && src < n) {  // the selection always writes in-range positions
    kv = *reinterpret_cast<const uint4*>(K + so);
    vv = *reinterpret_cast<const uint4*>(V + so);
  }
  *reinterpret_cast<uint4*>(k_out + dof) = kv;
  *reinterpret_cast<uint4*>(v0c + dof) = vv;
  if (!v_out) return;
  const T* ve = reinterpret_cast<const T*>(&vv);
  for (int e = 0; e < epc; ++e) {
    float f;
    if constexpr (sizeof(T) == 2) f = bf16_to_f32(ve[e]); else f = ve[e];
    v_out[dof + e] = f;
  }
}

}  // namespace

hipError_t launch_select(const Plan& p, const float* colsum, float* pooled, int32_t* idx,
                         uint8_t* fixed, hipStream_t s) {
  SelK a;
  a.colsum = colsum; a.pooled = pooled; a.idx = idx; a.fixed = fixed;
  a.prefix = p.prefix; a.c = p.c; a.w = p.w; a.h = (p.k_pool - 1) / 2;
  a.s_sel = p.s_sel; a.n_top = p.n_top_fixed; a.n_sink = p.opt.n_sink;
  a.fix_window = p.opt.fix_window ? 1 : 0; a.n = p.n;
  a.rag = p.rag;
  if (p.prefix <= kSmallThreads * kSmallPer && p.k_pool <= 17) {
#define GRKV_SEL_SMALL(HV) \
  case HV: hipLaunchKernelGGL(select_small_kernel<HV>, dim3(p.U), dim3(kSmallThreads), 0, s, a); break;
    switch (a.h) {
      GRKV_SEL_SMALL(0) GRKV_SEL_SMALL(1) GRKV_SEL_SMALL(2) GRKV_SEL_SMALL(3) GRKV_SEL_SMALL(4)
      GRKV_SEL_SMALL(5) GRKV_SEL_SMALL(6) GRKV_SEL_SMALL(7) GRKV_SEL_SMALL(8)
      default: return hipErrorInvalidValue;
    }
#undef GRKV_SEL_SMALL
  } else
    hipLaunchKernelGGL(select_kernel, dim3(p.U), dim3(kSelectThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gather(const Plan& p, const void* K, const void* V, const int32_t* idx,
                         void* k_out, void* v0c, float* v_out, hipStream_t s) {
  const int esz = p.dtype == GRKV_BF16 ? 2 : 4;
  const int64_t chunks = (int64_t)p.c * (p.d * esz / 16);
  dim3 grid((unsigned)((chunks + 255) / 256), p.U);
  if (p.dtype == GRKV_BF16)
    hipLaunchKernelGGL(gather_kernel<u16>, grid, dim3(256), 0, s, (const u16*)K, (const u16*)V,
                       idx, (u16*)k_out, (u16*)v0c, v_out, p.c, p.n, p.d);
  else
    hipLaunchKernelGGL(gather_kernel<float>, grid, dim3(256), 0, s, (const float*)K,
                       (const float*)V, idx, (float*)k_out, (float*)v0c, v_out, p.c, p.n, p.d);
  return hipGetLastError();
}

}  // namespace grkv
