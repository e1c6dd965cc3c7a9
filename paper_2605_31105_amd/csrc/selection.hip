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

// Band of candidates around a threshold, as refine_boundary below describes
// (that is the form for keys held in registers); here each thread scans the
// contiguous positions [j0, j1) of the pooled scores in memory.  With
// big == false the band's positions (ascending) and take flags are in `bt`
// and `boff` is where this thread's band entries start.
constexpr uint32_t kBandUlps = 16;
constexpr uint32_t kBandCap = 1024;

struct BandRule {
  uint32_t T, lo, hi, krem;   // krem: ties at T taken when the band is too big
  bool big;
  uint32_t boff;
  const uint32_t* take;
};

__device__ BandRule band_rule(const float* p, uint32_t T, uint32_t k, const float* s, int j0,
                              int j1, int P, int h, char* work, uint32_t* scan_scratch) {
  BandRule r;
  r.T = T;
  r.lo = T > kBandUlps ? T - kBandUlps : 0u;
  r.hi = T < 0x7F800000u - kBandUlps ? T + kBandUlps : 0x7F800000u;
  uint32_t nabove = 0, nband = 0, ngt = 0, neq = 0;
  for (int j = j0; j < j1; ++j) {
    const uint32_t key = __float_as_uint(p[j]);
    nabove += key > r.hi;
    nband += key >= r.lo && key <= r.hi;
    ngt += key > T;
    neq += key == T;
  }
  uint32_t tot_above, tot_band, tot_gt, tot_eq;
  block_exclusive_scan(nabove, scan_scratch, &tot_above);
  r.boff = block_exclusive_scan(nband, scan_scratch, &tot_band);
  block_exclusive_scan(ngt, scan_scratch, &tot_gt);
  r.krem = block_exclusive_scan(neq, scan_scratch, &tot_eq);   // this thread's first tie index
  r.krem = (k - tot_gt) > r.krem ? (k - tot_gt) - r.krem : 0u;  // ties this thread may take
  r.big = tot_band > kBandCap;
  double* v64 = reinterpret_cast<double*>(work);
  int32_t* bpos = reinterpret_cast<int32_t*>(v64 + kBandCap);
  uint32_t* btake = reinterpret_cast<uint32_t*>(bpos + kBandCap);
  r.take = btake;
  if (r.big) return r;
  const uint32_t need = k - tot_above;
  {
    uint32_t o = r.boff;
    for (int j = j0; j < j1; ++j) {
      const uint32_t key = __float_as_uint(p[j]);
      if (key >= r.lo && key <= r.hi) bpos[o++] = j;
    }
  }
  __syncthreads();
  for (uint32_t e = threadIdx.x; e < tot_band; e += blockDim.x) {
    const int j = bpos[e];
    const int t0 = j - h < 0 ? 0 : j - h, t1 = j + h > P - 1 ? P - 1 : j + h;
    double acc = 0.0;
    for (int t = t0; t <= t1; ++t) acc += (double)s[t];   // left to right
    v64[e] = acc;
  }
  __syncthreads();
  for (uint32_t e = threadIdx.x; e < tot_band; e += blockDim.x) {
    const double v = v64[e];
    const int j = bpos[e];
    uint32_t rank = 0;
    for (uint32_t f = 0; f < tot_band; ++f) {
      const double w = v64[f];
      rank += w > v || (w == v && bpos[f] < j);
    }
    btake[e] = rank < need;
  }
  __syncthreads();
  return r;
}

// Whether position key is taken under rule r; `e` counts this thread's band
// entries (or, for a big band, its ties at T) seen so far.
__device__ __forceinline__ bool band_take(const BandRule& r, uint32_t key, uint32_t& e) {
  if (r.big) {
    const bool t = key > r.T || (key == r.T && e < r.krem);
    e += key == r.T;
    return t;
  }
  if (key > r.hi) return true;
  if (key >= r.lo) return r.take[r.boff + e++] != 0;
  return false;
}

__global__ __launch_bounds__(kSelectThreads) void select_kernel(SelK a) {
  __shared__ __attribute__((aligned(16))) char band_work[2][kBandCap * 16];
  __shared__ uint32_t hist[2][256];
  __shared__ uint32_t sh_state[4];
  __shared__ uint32_t scan_scratch[16];

  const int u = blockIdx.x, tid = threadIdx.x;
  const int P = a.prefix;
  const float* s = a.colsum + (size_t)u * P;
  float* p = a.pooled + (size_t)u * P;
  const UnitSel us = unit_sel(a, u);
  int32_t* idx = a.idx + us.base;
  uint8_t* fixed = a.fixed + us.base;

  for (int j = tid; j < P; j += blockDim.x) {
    int lo = j - a.h < 0 ? 0 : j - a.h;
    int hi = j + a.h > P - 1 ? P - 1 : j + a.h;
    float acc = 0.f;
    for (int t = lo; t <= hi; ++t) acc += s[t];
    p[j] = acc;
  }
  __syncthreads();

  // radix select of the k-th largest for k = s_sel (target 0) and n_top (1)
  uint32_t prefix[2] = {0u, 0u}, krem[2] = {(uint32_t)us.s_sel, (uint32_t)us.n_top};
  uint32_t mask = 0u;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < 512; b += blockDim.x) (&hist[0][0])[b] = 0u;
    __syncthreads();
    for (int j = tid; j < P; j += blockDim.x) {
      uint32_t key = __float_as_uint(p[j]);
#pragma unroll
      for (int t = 0; t < 2; ++t)
        if (krem[t] > 0 && (key & mask) == prefix[t]) atomicAdd(&hist[t][(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 2 && krem[tid] > 0) {
      uint32_t cum = 0;
      int digit = 0;
      for (int b = 255; b >= 0; --b) {
        uint32_t hcount = hist[tid][b];
        if (cum + hcount >= krem[tid]) { digit = b; break; }
        cum += hcount;
      }
      sh_state[2 * tid] = prefix[tid] | ((uint32_t)digit << shift);
      sh_state[2 * tid + 1] = krem[tid] - cum;
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < 2; ++t)
      if (krem[t] > 0) { prefix[t] = sh_state[2 * t]; krem[t] = sh_state[2 * t + 1]; }
    mask |= 255u << shift;
    __syncthreads();
  }
  // prefix[t] = bits of the k-th largest score; krem[t] = how many scores
  // equal to it are taken (lowest positions first); all larger ones are taken.
  const uint32_t T0 = prefix[0], T1 = prefix[1];
  const bool any0 = us.s_sel > 0, any1 = us.n_top > 0;

  const int per = (P + blockDim.x - 1) / blockDim.x;
  const int j0 = min(P, tid * per), j1 = min(P, j0 + per);
  BandRule r0 = {}, r1 = {};
  if (any0) r0 = band_rule(p, T0, (uint32_t)us.s_sel, s, j0, j1, P, a.h, band_work[0], scan_scratch);
  if (any1) r1 = band_rule(p, T1, (uint32_t)us.n_top, s, j0, j1, P, a.h, band_work[1], scan_scratch);
  uint32_t nsel = 0;
  {
    uint32_t e0 = 0;
    for (int j = j0; j < j1; ++j) {
      const uint32_t key = __float_as_uint(p[j]);
      nsel += any0 && band_take(r0, key, e0);
    }
  }
  uint32_t tot;
  uint32_t off = block_exclusive_scan(nsel, scan_scratch, &tot);
  {
    uint32_t e0 = 0, e1 = 0;
    for (int j = j0; j < j1; ++j) {
      const uint32_t key = __float_as_uint(p[j]);
      const bool sel = any0 && band_take(r0, key, e0);
      const bool top = any1 && band_take(r1, key, e1);
      if (sel) {
        idx[off] = j;
        fixed[off] = (j < a.n_sink || top) ? 1 : 0;
        ++off;
      }
    }
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
  return tot;
}

// State of one k-th-largest search over the keys (fp32 bit patterns of
// non-negative scores, which order like the values): lo <= T < hi with
// clo = count(>= lo) >= k > count(>= hi) = chi.
struct Bracket {
  uint32_t lo, hi, clo, chi;
};

// The positions taken at a threshold T, the k-th largest fp32 pooled score,
// as a mask over the PER keys of this thread (key q <-> position j0 + q).
//
// The fp32 pooled sums round away differences that decide the order: two
// overlapping windows share all but their edge terms, and when a large score
// sits in both, their fp32 sums are equal while the edge terms differ.  So
// the candidates whose fp32 sum lies within kBandUlps units in the last place
// of T are ranked again by their sum recomputed in fp64 from the fp32 column
// sums (in which the shared terms cancel exactly), then by position; the
// keys above the band are taken, and the band fills the remaining places.
// A band of more than kBandCap keys (scores equal over long runs) keeps the
// fp32 order with ties to the lower position.  `work` is LDS of at least
// kBandCap * (8 + 4 + 4) bytes.
template <int PER>
__device__ uint32_t refine_boundary(const uint32_t (&key)[PER], uint32_t T, uint32_t k,
                                    const float* s, int j0, int P, int h, float* work,
                                    uint32_t (*part)[16], uint32_t* scan_scratch, uint32_t* sh) {
  const uint32_t lo = T > kBandUlps ? T - kBandUlps : 0u;
  const uint32_t hi = T < 0x7F800000u - kBandUlps ? T + kBandUlps : 0x7F800000u;
  uint32_t nabove = 0, nband = 0;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    nabove += key[q] > hi;
    nband += key[q] >= lo && key[q] <= hi;
  }
  // both counts in one scan (each total is at most PER * blockDim <= 32768)
  uint32_t tot;
  const uint32_t boff = block_exclusive_scan(nabove | (nband << 16), scan_scratch, &tot) >> 16;
  const uint32_t tot_above = tot & 0xFFFFu, tot_band = tot >> 16;
  const uint32_t need = k - tot_above;   // 1 <= need <= tot_band
  uint32_t m = 0;
  if (tot_band > kBandCap) {
    // fp32 order, ties (key == T) to the lower position
    uint32_t gt = 0, eq = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      gt += key[q] > T;
      eq += key[q] == T;
    }
    uint32_t t2;
    uint32_t e = block_exclusive_scan(gt | (eq << 16), scan_scratch, &t2) >> 16;
    const uint32_t krem = k - (t2 & 0xFFFFu);
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const bool take = key[q] > T || (key[q] == T && e < krem);
      e += key[q] == T;
      m |= (uint32_t)take << q;
    }
    return m;
  }
  double* v64 = reinterpret_cast<double*>(work);                       // [kBandCap]
  int32_t* bpos = reinterpret_cast<int32_t*>(v64 + kBandCap);          // [kBandCap]
  uint32_t* btake = reinterpret_cast<uint32_t*>(bpos + kBandCap);      // [kBandCap]
  {
    uint32_t o = boff;
#pragma unroll
    for (int q = 0; q < PER; ++q)
      if (key[q] >= lo && key[q] <= hi) bpos[o++] = j0 + q;
  }
  __syncthreads();
  for (uint32_t e = threadIdx.x; e < tot_band; e += blockDim.x) {
    const int j = bpos[e];
    const int t0 = j - h < 0 ? 0 : j - h, t1 = j + h > P - 1 ? P - 1 : j + h;
    double acc = 0.0;
    for (int t = t0; t <= t1; ++t) acc += (double)s[t];   // left to right
    v64[e] = acc;
  }
  __syncthreads();
  for (uint32_t e = threadIdx.x; e < tot_band; e += blockDim.x) {
    const double v = v64[e];
    const int j = bpos[e];
    uint32_t rank = 0;
    for (uint32_t f = 0; f < tot_band; ++f) {
      const double w = v64[f];
      rank += w > v || (w == v && bpos[f] < j);
    }
    btake[e] = rank < need;
  }
  __syncthreads();
  {
    uint32_t o = boff;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      bool take = key[q] > hi;
      if (key[q] >= lo && key[q] <= hi) take = btake[o++] != 0;
      m |= (uint32_t)take << q;
    }
  }
  __syncthreads();   // work is reused by the next call
  return m;
}

// Same selection for prefixes of at most 32768 tokens, with each thread
// keeping 32 consecutive pooled scores in registers.  The (c-w)-th largest
// score T0 is found by bisection on the bit patterns: block-wide counts of
// "score >= mid" from the [min, max] bracket until at most kCandCap keys
// remain inside it; those candidates go to LDS and radix rounds (256 bins of
// the bit pattern's offset in the bracket) finish.  The floor(beta*c)-th
// largest T1 lies among the keys >= T0 (about c-w of them), so it starts
// from the candidates directly.
__global__ __launch_bounds__(kSmallThreads) void select_small_kernel(SelK a) {
  __shared__ float sl[kSmallThreads * kSmallPer + kSmallThreads * kSmallPer / 64];
  __shared__ uint32_t part[2][16];
  __shared__ uint32_t scan_scratch[16];
  __shared__ uint32_t sh[8];
  __shared__ uint32_t hist[256];
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

  // Scores of the whole prefix into LDS (coalesced), one pad word per 64
  // entries so that the lanes of a wave, each reading its own contiguous
  // run, fall on distinct banks.  Each thread then pools its 32 positions
  // (plus 8 on either side) in registers, summing s[j-h..j+h] left to right.
  // Positions past the prefix get key 0: they rank after every real position
  // with an equal score and are never taken while real positions are left.
  {
    // all PER loads of a thread in flight at once
    float ld[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int t = tid + k * kSmallThreads;
      ld[k] = t < P ? s[t] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int t = tid + k * kSmallThreads;
      sl[t + (t >> 6)] = ld[k];
    }
  }
  __syncthreads();
  uint32_t key[PER];
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  {
    float v[PER + 16];
#pragma unroll
    for (int q = 0; q < PER + 16; ++q) {
      const int t = j0 - 8 + q;
      v[q] = (t >= 0 && t < P) ? sl[t + (t >> 6)] : 0.f;
    }
    const int h = a.h;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int j = j0 + q;
      float acc = 0.f;
#pragma unroll
      for (int t = -8; t <= 8; ++t)   // offsets -h..h in increasing order
        if (t >= -h && t <= h) acc += v[q + 8 + t];
      key[q] = j < P ? __float_as_uint(acc) : 0u;
      if (j < P) {
        kmin = min(kmin, key[q]);
        kmax = max(kmax, key[q]);
      }
    }
  }
  // the pooled scores (an intermediate the caller may inspect), coalesced
  __syncthreads();
#pragma unroll
  for (int q = 0; q < PER; ++q) sl[j0 + q + ((j0 + q) >> 6)] = __uint_as_float(key[q]);
  __syncthreads();
  for (int t = tid; t < P; t += kSmallThreads) pg[t] = sl[t + (t >> 6)];

  // key range of the real positions (block min and max)
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
    __syncthreads();   // part is reused below
  }
  kmax = min(kmax, 0x7F800000u);   // +inf at most (no NaN scores)
  uint32_t* cand = reinterpret_cast<uint32_t*>(sl);   // [kCandCap], reuses the staging area
  int parity = 0;

  // k-th largest key from bracket b: block rounds while more than kCandCap
  // keys lie in [lo, hi), then the candidates into LDS and radix rounds.
  // Returns T with b.lo = T, b.hi = T + 1 (so b.chi = count(> T) and
  // b.clo = count(>= T)).
  auto kth = [&](uint32_t k, Bracket b) -> Bracket {
#pragma unroll 1
    for (int it = 0; it < 33 && b.hi - b.lo > 1 && b.clo - b.chi > kCandCap; ++it) {
      const uint32_t mid = b.lo + (b.hi - b.lo) / 2;
      uint32_t n = 0;
#pragma unroll
      for (int q = 0; q < PER; ++q) n += key[q] >= mid;
      const uint32_t c = block_sum_small(n, part, parity);
      parity ^= 1;
      if (c >= k) { b.lo = mid; b.clo = c; }
      else { b.hi = mid; b.chi = c; }
    }
    if (b.hi - b.lo <= 1) return b;
    uint32_t n = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) n += key[q] >= b.lo && key[q] < b.hi;
    uint32_t tot;
    uint32_t o = block_exclusive_scan(n, scan_scratch, &tot);
#pragma unroll
    for (int q = 0; q < PER; ++q)
      if (key[q] >= b.lo && key[q] < b.hi) {
        if (o < kCandCap) cand[o] = key[q];
        ++o;
      }
    __syncthreads();
    // Radix rounds on the candidates: 256 bins of (x - lo) >> shift cover
    // [lo, hi); the bin holding the k-th largest becomes the new bracket.  A
    // 32-bit range takes at most four rounds.
    const uint32_t L = min(b.clo - b.chi, kCandCap);
#pragma unroll 1
    for (int it = 0; it < 5 && b.hi - b.lo > 1; ++it) {
      const uint32_t width = b.hi - b.lo;
      const int bits = 32 - __builtin_clz(width - 1);   // width - 1 < 2^bits
      const int shift = bits > 8 ? bits - 8 : 0;
      if (tid < 256) hist[tid] = 0u;
      __syncthreads();
      for (uint32_t e = tid; e < L; e += kSmallThreads) {
        const uint32_t x = cand[e];
        if (x >= b.lo && x < b.hi) atomicAdd(&hist[(x - b.lo) >> shift], 1u);
      }
      __syncthreads();
      if (wave == 0) {
        // suffix sums over the bins: lane l holds bins 4l .. 4l+3
        uint32_t h4[4], suf = 0;
#pragma unroll
        for (int i = 3; i >= 0; --i) {
          h4[i] = hist[4 * lane + i];
          suf += h4[i];
        }
        // inclusive suffix scan across lanes (lanes above l)
        uint32_t incl = suf;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const uint32_t o = (uint32_t)__shfl_down((int)incl, off);
          if (lane + off < 64) incl += o;
        }
        // count(>= start of bin 4l + i) = chi + (bins above) ; the largest bin
        // whose count reaches k holds the k-th largest
        uint32_t above = b.chi + incl - suf;   // keys in bins > 4l+3, plus those >= hi
        int best = -1;
        uint32_t bc = 0, bh = 0;
#pragma unroll
        for (int i = 3; i >= 0; --i) {
          const uint32_t c = above + h4[i];
          if (best < 0 && c >= k) { best = 4 * lane + i; bc = c; bh = above; }
          above = c;
        }
        // the highest lane with a hit owns the answer
        const uint64_t hit = __ballot(best >= 0);
        const int owner = 63 - __builtin_clzll(hit);
        if (lane == owner) {
          const uint32_t nlo = b.lo + ((uint32_t)best << shift);
          const uint64_t nhi = (uint64_t)b.lo + ((uint64_t)(best + 1) << shift);
          sh[0] = nlo;
          sh[1] = nhi < b.hi ? (uint32_t)nhi : b.hi;
          sh[2] = bc;
          sh[3] = bh;
        }
      }
      __syncthreads();
      b.lo = sh[0]; b.hi = sh[1]; b.clo = sh[2]; b.chi = sh[3];
      __syncthreads();   // hist and sh are rewritten by the next round
    }
    return b;
  };

  const uint32_t k0 = (uint32_t)us.s_sel, k1 = (uint32_t)us.n_top;
  const bool any0 = k0 > 0, any1 = k1 > 0;
  // count(>= kmin) = P (the padding keys, 0, count only when kmin is 0)
  const uint32_t all = kmin > 0 ? (uint32_t)P : (uint32_t)(kSmallThreads * PER);
  Bracket b0 = {kmin, kmax + 1, all, 0u};
  if (any0) b0 = kth(k0, b0);
  // the n_top-th largest is at least T0 (n_top <= s_sel)
  Bracket b1 = any0 ? Bracket{b0.lo, kmax + 1, b0.clo, 0u} : Bracket{kmin, kmax + 1, all, 0u};
  if (any1) b1 = kth(k1, b1);
  const uint32_t T0 = b0.lo, T1 = b1.lo;
  uint32_t selm = any0 ? refine_boundary(key, T0, k0, s, j0, P, a.h, sl, part, scan_scratch, sh) : 0u;
  uint32_t topm = any1 ? refine_boundary(key, T1, k1, s, j0, P, a.h, sl, part, scan_scratch, sh) : 0u;
  uint32_t tot;
  uint32_t off = block_exclusive_scan(__builtin_popcount(selm), scan_scratch, &tot);
  // the selected positions in increasing order
  while (selm) {
    const int q = __builtin_ctz(selm);
    const int j = j0 + q;
    idx[off] = j;
    fixed[off] = (j < a.n_sink || ((topm >> q) & 1)) ? 1 : 0;
    ++off;
    selm &= selm - 1;
  }
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
  if (p.prefix <= kSmallThreads * kSmallPer && p.k_pool <= 17)
    hipLaunchKernelGGL(select_small_kernel, dim3(p.U), dim3(kSmallThreads), 0, s, a);
  else
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
