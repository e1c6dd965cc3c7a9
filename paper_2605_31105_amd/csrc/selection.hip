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
};

__global__ __launch_bounds__(kSelectThreads) void select_kernel(SelK a) {
  __shared__ uint32_t hist[2][256];
  __shared__ uint32_t sh_state[4];
  __shared__ uint32_t scan_scratch[16];

  const int u = blockIdx.x, tid = threadIdx.x;
  const int P = a.prefix;
  const float* s = a.colsum + (size_t)u * P;
  float* p = a.pooled + (size_t)u * P;
  int32_t* idx = a.idx + (size_t)u * a.c;
  uint8_t* fixed = a.fixed + (size_t)u * a.c;

  for (int j = tid; j < P; j += blockDim.x) {
    int lo = j - a.h < 0 ? 0 : j - a.h;
    int hi = j + a.h > P - 1 ? P - 1 : j + a.h;
    float acc = 0.f;
    for (int t = lo; t <= hi; ++t) acc += s[t];
    p[j] = acc;
  }
  __syncthreads();

  // radix select of the k-th largest for k = s_sel (target 0) and n_top (1)
  uint32_t prefix[2] = {0u, 0u}, krem[2] = {(uint32_t)a.s_sel, (uint32_t)a.n_top};
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
  const bool any0 = a.s_sel > 0, any1 = a.n_top > 0;

  const int per = (P + blockDim.x - 1) / blockDim.x;
  const int j0 = min(P, tid * per), j1 = min(P, j0 + per);
  uint32_t eq0 = 0, eq1 = 0;
  for (int j = j0; j < j1; ++j) {
    uint32_t key = __float_as_uint(p[j]);
    eq0 += (any0 && key == T0);
    eq1 += (any1 && key == T1);
  }
  uint32_t tot;
  uint32_t eqb0 = block_exclusive_scan(eq0, scan_scratch, &tot);
  uint32_t eqb1 = block_exclusive_scan(eq1, scan_scratch, &tot);
  uint32_t nsel = 0;
  {
    uint32_t e0 = eqb0;
    for (int j = j0; j < j1; ++j) {
      uint32_t key = __float_as_uint(p[j]);
      bool sel = any0 && (key > T0 || (key == T0 && e0 < krem[0]));
      e0 += (any0 && key == T0);
      nsel += sel;
    }
  }
  uint32_t off = block_exclusive_scan(nsel, scan_scratch, &tot);
  {
    uint32_t e0 = eqb0, e1 = eqb1;
    for (int j = j0; j < j1; ++j) {
      uint32_t key = __float_as_uint(p[j]);
      bool sel = any0 && (key > T0 || (key == T0 && e0 < krem[0]));
      bool top = any1 && (key > T1 || (key == T1 && e1 < krem[1]));
      e0 += (any0 && key == T0);
      e1 += (any1 && key == T1);
      if (sel) {
        idx[off] = j;
        fixed[off] = (j < a.n_sink || top) ? 1 : 0;
        ++off;
      }
    }
  }
  for (int i = tid; i < a.w; i += blockDim.x) {
    int64_t pos = a.n - a.w + i;
    idx[a.s_sel + i] = (int32_t)pos;
    fixed[a.s_sel + i] = (a.fix_window || pos < a.n_sink) ? 1 : 0;
  }
}

constexpr int kSmallThreads = 512;
constexpr int kSmallPer = 64;   // pooled scores per thread: prefixes up to 32768

// Block-wide sum of one value per thread (kSmallThreads threads); `part` holds
// 2 x 8 words and alternates by `parity` so consecutive calls need one barrier.
// Within a wave: DPP sums over 16-lane rows, then the four row totals.
__device__ __forceinline__ uint32_t block_sum_small(uint32_t v, uint32_t (*part)[8], int parity) {
  int x = (int)v;
  x += __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x140, 0xF, 0xF, false);
  v = (uint32_t)(__builtin_amdgcn_readlane(x, 0) + __builtin_amdgcn_readlane(x, 16) +
                 __builtin_amdgcn_readlane(x, 32) + __builtin_amdgcn_readlane(x, 48));
  if ((threadIdx.x & 63) == 0) part[parity][threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t tot = 0;
#pragma unroll
  for (int k = 0; k < kSmallThreads / 64; ++k) tot += part[parity][k];
  return tot;
}

// Same selection for prefixes of at most 32768 tokens, with each thread
// keeping 64 consecutive pooled scores in registers.  The k-th largest score
// is found by bisection on the fp32 bit pattern (scores are >= 0, so bit
// patterns order like values): 31 block-wide counts of "score >= mid", no
// histograms and no atomics.
__global__ __launch_bounds__(kSmallThreads) void select_small_kernel(SelK a) {
  __shared__ float sl[kSmallThreads * kSmallPer + kSmallThreads * kSmallPer / 64];
  __shared__ uint32_t part[2][8];
  __shared__ uint32_t scan_scratch[16];
  constexpr int PER = kSmallPer;
  const int u = blockIdx.x, tid = threadIdx.x;
  const int P = a.prefix;
  const float* s = a.colsum + (size_t)u * P;
  float* pg = a.pooled + (size_t)u * P;
  int32_t* idx = a.idx + (size_t)u * a.c;
  uint8_t* fixed = a.fixed + (size_t)u * a.c;
  const int j0 = tid * PER;

  // Positions past the prefix get key 0 (score 0.0): they rank after every
  // real position with an equal score, so they are never taken while real
  // positions are left.
  // Scores of the whole prefix into LDS (coalesced), stored with one pad word
  // per 64 entries so that the 64 lanes of a wave, each reading its own
  // contiguous run, fall on distinct banks.  Each thread then takes its 64
  // positions plus 8 on either side into registers and pools them, summing
  // s[j-h..j+h] left to right.
  for (int t = tid; t < P; t += kSmallThreads) sl[t + (t >> 6)] = s[t];
  __syncthreads();
  uint32_t key[PER];
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
    }
  }
  // the pooled scores (an intermediate the caller may inspect), coalesced
  __syncthreads();
#pragma unroll
  for (int q = 0; q < PER; ++q) sl[j0 + q + ((j0 + q) >> 6)] = __uint_as_float(key[q]);
  __syncthreads();
  for (int t = tid; t < P; t += kSmallThreads) pg[t] = sl[t + (t >> 6)];

  // count of keys >= x over the block
  int parity = 0;
  auto count_ge = [&](uint32_t x0, uint32_t x1, uint32_t* c0, uint32_t* c1) {
    uint32_t n0 = 0, n1 = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      n0 += key[q] >= x0;
      n1 += key[q] >= x1;
    }
    *c0 = block_sum_small(n0 | (n1 << 16), part, parity);
    parity ^= 1;
    *c1 = *c0 >> 16;
    *c0 &= 0xFFFF;
  };
  // largest T with count(>= T) >= k, for k = s_sel (0) and n_top (1)
  uint32_t lo0 = 0, hi0 = 0x7F800001u, lo1 = 0, hi1 = 0x7F800001u;
  const uint32_t k0 = (uint32_t)a.s_sel, k1 = (uint32_t)a.n_top;
#pragma unroll 1
  for (int it = 0; it < 32; ++it) {
    const bool go0 = k0 > 0 && hi0 - lo0 > 1, go1 = k1 > 0 && hi1 - lo1 > 1;
    if (!go0 && !go1) break;   // uniform: every thread holds the same bounds
    const uint32_t m0 = lo0 + (hi0 - lo0) / 2, m1 = lo1 + (hi1 - lo1) / 2;
    uint32_t c0, c1;
    count_ge(m0, m1, &c0, &c1);
    if (go0) { if (c0 >= k0) lo0 = m0; else hi0 = m0; }
    if (go1) { if (c1 >= k1) lo1 = m1; else hi1 = m1; }
  }
  const uint32_t T0 = lo0, T1 = lo1;
  uint32_t gt0, gt1;
  count_ge(T0 + 1, T1 + 1, &gt0, &gt1);
  const bool any0 = k0 > 0, any1 = k1 > 0;
  const uint32_t krem0 = k0 - gt0, krem1 = k1 - gt1;   // ties taken, lowest positions first

  uint32_t eq0 = 0, eq1 = 0;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    eq0 += key[q] == T0;
    eq1 += key[q] == T1;
  }
  if (!any0) eq0 = 0;
  if (!any1) eq1 = 0;
  uint32_t tot;
  const uint32_t eqb0 = block_exclusive_scan(eq0, scan_scratch, &tot);
  const uint32_t eqb1 = block_exclusive_scan(eq1, scan_scratch, &tot);
  uint32_t nsel = 0;
  {
    uint32_t e0 = eqb0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const bool sel = key[q] > T0 || (key[q] == T0 && e0 < krem0);
      e0 += key[q] == T0;
      nsel += sel;
    }
    if (!any0) nsel = 0;
  }
  uint32_t off = block_exclusive_scan(nsel, scan_scratch, &tot);
  // selection and top-beta membership as bit masks over this thread's positions,
  // then the selected positions in increasing order
  uint64_t selm = 0, topm = 0;
  {
    uint32_t e0 = eqb0, e1 = eqb1;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const bool sel = key[q] > T0 || (key[q] == T0 && e0 < krem0);
      const bool top = key[q] > T1 || (key[q] == T1 && e1 < krem1);
      e0 += key[q] == T0;
      e1 += key[q] == T1;
      selm |= (uint64_t)sel << q;
      topm |= (uint64_t)top << q;
    }
  }
  if (!any0) selm = 0;
  if (!any1) topm = 0;
  while (selm) {
    const int q = __builtin_ctzll(selm);
    const int j = j0 + q;
    idx[off] = j;
    fixed[off] = (j < a.n_sink || ((topm >> q) & 1)) ? 1 : 0;
    ++off;
    selm &= selm - 1;
  }
  for (int i = tid; i < a.w; i += blockDim.x) {
    const int64_t pos = a.n - a.w + i;
    idx[a.s_sel + i] = (int32_t)pos;
    fixed[a.s_sel + i] = (a.fix_window || pos < a.n_sink) ? 1 : 0;
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
