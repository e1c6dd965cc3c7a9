// Adaptive per-head budgets (the head-wise allocation of Ada-KV, with which
// the paper pairs GRKV in Sec. 4): inside each layer the H heads share
// H (c - w) selected tokens, taken as the highest pooled SnapKV scores over
// all heads of the layer (ties to the lower head, then the lower position),
// and head h keeps w plus the number of its tokens taken.
//
// One block per layer.  Pooled scores are non-negative, so their fp32 bit
// patterns order like the values: a bisection over the 31-bit key range finds
// the k-th largest key T with block-wide counts, then every head counts its
// keys above T and takes its share of the keys equal to T in head order.
#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

constexpr int kAdaThreads = 1024;
constexpr int kAdaMaxHeads = 128;

__device__ __forceinline__ uint32_t block_count(uint32_t v, uint32_t* red) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  uint32_t t = 0;
  for (int k = 0; k < kAdaThreads / 64; ++k) t += red[k];
  return t;
}

__global__ __launch_bounds__(kAdaThreads) void adaptive_kernel(const float* __restrict__ pooled,
                                                               int H, int P, int64_t kk, int w,
                                                               int32_t* __restrict__ budgets) {
  __shared__ uint32_t red[kAdaThreads / 64];
  __shared__ uint32_t gt[kAdaMaxHeads], eq[kAdaMaxHeads];
  const int l = blockIdx.x, tid = threadIdx.x;
  const int64_t N = (int64_t)H * P;
  const uint32_t* key = reinterpret_cast<const uint32_t*>(pooled + (size_t)l * N);
  if (kk > N) kk = N;
  for (int h = tid; h < H; h += kAdaThreads) gt[h] = eq[h] = 0;
  uint32_t T = 0;
  if (kk > 0) {
    // invariant: count(key >= lo) >= kk, count(key >= hi) < kk
    uint32_t lo = 0, hi = 0x7F800001u;
    while (hi - lo > 1) {
      const uint32_t mid = lo + (hi - lo) / 2;
      uint32_t c = 0;
      for (int64_t e = tid; e < N; e += kAdaThreads) c += key[e] >= mid;
      if (block_count(c, red) >= (uint32_t)kk) lo = mid;
      else hi = mid;
    }
    T = lo;
  }
  __syncthreads();
  if (kk > 0) {
    for (int64_t e = tid; e < N; e += kAdaThreads) {
      const uint32_t x = key[e];
      const int h = (int)(e / P);
      if (x > T) atomicAdd(&gt[h], 1u);
      else if (x == T) atomicAdd(&eq[h], 1u);
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
