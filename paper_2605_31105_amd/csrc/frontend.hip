// Adaptive per-head budgets (the head-wise allocation of Ada-KV, with which
// the paper pairs GRKV in Sec. 4): inside each layer the H heads share
// H (c - w) selected tokens, taken as the highest pooled SnapKV scores over
// all heads of the layer (ties to the lower head, then the lower position),
// and head h keeps w plus the number of its tokens taken.
//
// One block per layer.  Pooled scores are non-negative, so their fp32 bit
// patterns order like the values: a radix select over the 31-bit keys (three
// digits of 11, 11 and 9 bits, one LDS histogram pass over the layer's scores
// per digit) finds the k-th largest key T; a last pass counts every head's
// keys above T and equal to T, and the keys equal to T are shared out in
// head order.
#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

constexpr int kAdaThreads = 1024;
constexpr int kAdaMaxHeads = 128;
constexpr int kAdaUnroll = 32;    // independent loads in flight per thread
constexpr int kAdaBins = 2048;    // widest digit (11 bits)
// Each bin is kept in kAdaCopies copies (chosen by lane), so that lanes of a
// wave landing in one crowded bin (scores share few exponents) add to
// different words; the scan sums the copies.
constexpr int kAdaCopies = 16;

// The scores of one layer, kAdaUnroll coalesced loads per thread at a time;
// past the end the key is 0xFFFFFFFF, which no radix prefix of a finite
// non-negative score matches.
template <typename F>
__device__ __forceinline__ void for_keys(const uint32_t* __restrict__ key, int64_t N, F f) {
  for (int64_t e0 = 0; e0 < N; e0 += (int64_t)kAdaThreads * kAdaUnroll) {
    uint32_t x[kAdaUnroll];
#pragma unroll
    for (int k = 0; k < kAdaUnroll; ++k) {
      const int64_t e = e0 + (int64_t)k * kAdaThreads + threadIdx.x;
      x[k] = e < N ? key[e] : 0xFFFFFFFFu;
    }
#pragma unroll
    for (int k = 0; k < kAdaUnroll; ++k) f(x[k]);
  }
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__global__ __launch_bounds__(kAdaThreads) void adaptive_kernel(const float* __restrict__ pooled,
                                                               int H, int P, int64_t kk, int w,
                                                               int32_t* __restrict__ budgets) {
  __shared__ uint32_t hist[kAdaBins * kAdaCopies];
  __shared__ uint32_t scratch[kAdaThreads / 64];
  __shared__ uint32_t gt[kAdaMaxHeads], eq[kAdaMaxHeads];
  __shared__ uint32_t pick[2];
  const int l = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int64_t N = (int64_t)H * P;
  const uint32_t* key = reinterpret_cast<const uint32_t*>(pooled + (size_t)l * N);
  if (kk > N) kk = N;
  for (int h = tid; h < H; h += kAdaThreads) gt[h] = eq[h] = 0;

  // digits from the top: bits 30..20, 19..9, 8..0
  constexpr int kShift[3] = {20, 9, 0};
  constexpr int kBits[3] = {11, 11, 9};
  uint32_t prefix = 0;          // the digits of T found so far, in place
  uint32_t krem = (uint32_t)kk; // rank of T among the keys matching the prefix
  if (kk > 0) {
#pragma unroll
    for (int lev = 0; lev < 3; ++lev) {
      const int shift = kShift[lev], nb = 1 << kBits[lev], top = shift + kBits[lev];
      for (int b = tid; b < nb * kAdaCopies; b += kAdaThreads) hist[b] = 0;
      __syncthreads();
      const uint32_t want = prefix >> top;
      const int copy = lane & (kAdaCopies - 1);
      for_keys(key, N, [&](uint32_t x) {
        if ((x >> top) == want) atomicAdd(&hist[((x >> shift) & (nb - 1)) * kAdaCopies + copy], 1u);
      });
      // (no pick when the scores break the non-negative precondition: T = 0)
      if (tid == 0) pick[0] = pick[1] = 0u;
      __syncthreads();
      // suffix counts in descending bin order: thread t holds bins
      // nb-1-2t and nb-2-2t; T's digit is the bin where the count of keys at
      // or above it first reaches krem
      const int per = nb / kAdaThreads > 0 ? nb / kAdaThreads : 1;   // 2 or 1 bins
      uint32_t v[2] = {0u, 0u};
      const int b0 = nb - 1 - per * tid;
      auto bin = [&](int b) {
        uint32_t t = 0;
#pragma unroll
        for (int k = 0; k < kAdaCopies; ++k) t += hist[b * kAdaCopies + k];
        return t;
      };
      if (b0 >= 0) {
        v[0] = bin(b0);
        if (per == 2) v[1] = bin(b0 - 1);
      }
      uint32_t tot;
      const uint32_t before = block_exclusive_scan(v[0] + v[1], scratch, &tot);
      if (b0 >= 0) {
        if (before < krem && before + v[0] >= krem) {
          pick[0] = (uint32_t)b0;
          pick[1] = before;
        } else if (per == 2 && before + v[0] < krem && before + v[0] + v[1] >= krem) {
          pick[0] = (uint32_t)(b0 - 1);
          pick[1] = before + v[0];
        }
      }
      __syncthreads();
      prefix |= pick[0] << shift;
      krem -= pick[1];   // keys of higher digits already counted
      __syncthreads();   // pick and hist are rewritten by the next level
    }
  }
  const uint32_t T = prefix;

  // keys above T and equal to T, per head (one LDS add per wave and head)
  if (kk > 0) {
    for (int h = 0; h < H; ++h) {
      uint32_t a = 0, e = 0;
      for_keys(key + (size_t)h * P, P, [&](uint32_t x) {
        a += x != 0xFFFFFFFFu && x > T;
        e += x == T;
      });
      a = wave_sum(a);
      e = wave_sum(e);
      if (lane == 0) {
        if (a) atomicAdd(&gt[h], a);
        if (e) atomicAdd(&eq[h], e);
      }
    }
  }
  __syncthreads();
  if (tid == 0) {
    int64_t above = 0;
    for (int h = 0; h < H; ++h) above += gt[h];
    int64_t need = kk > 0 ? kk - above : 0;   // keys equal to T still to take
    for (int h = 0; h < H; ++h) {
      const int64_t tie = need > 0 ? (need < (int64_t)eq[h] ? need : (int64_t)eq[h]) : 0;
      need -= tie;
      budgets[(size_t)l * H + h] = w + (int32_t)(gt[h] + tie);
    }
  }
}

}  // namespace

hipError_t launch_adaptive_budgets(const float* pooled, int layers, int H, int P, int64_t kk,
                                   int w, int32_t* budgets, hipStream_t s) {
  if (H < 1 || H > kAdaMaxHeads) return hipErrorInvalidValue;
  hipLaunchKernelGGL(adaptive_kernel, dim3(layers), dim3(kAdaThreads), 0, s, pooled, H, P, kk, w,
                     budgets);
  return hipGetLastError();
}

}  // namespace grkv
