// Device-side helpers for the gfx950 kernels: MFMA fragments, bf16 packing,
// wave reductions and block scans.  64-wide wavefronts throughout.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace grkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16;

// 16x16 output tile, K = 32 bf16 (gfx950 double-rate bf16 MFMA).
// Operand layout: lane l holds A[l%16][8*(l/16) .. +8) and B[8*(l/16) .. +8)[l%16];
// result: lane l holds D[4*(l/16) + i][l%16], i = 0..3.  Any permutation of the
// K index applied identically to A and B leaves the product unchanged.
__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// The same tile shape with fp16 operands.
__device__ __forceinline__ f32x4 mfma_f16(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// 16x16 output tile, K = 4 fp32: lane l holds A[l%16][l/16], B[l/16][l%16].
__device__ __forceinline__ f32x4 mfma_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ float bf16_to_f32(u16 b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Round-to-nearest-even split of 8 floats into bf16 hi and lo parts,
// x ~= hi + lo with about 16 significant bits.  Pairs go through the packed
// conversion (two values per instruction); hi back to fp32 is a shift or a
// mask of the packed word.
__device__ __forceinline__ void split8(const float* x, bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const bf16x2 h = __builtin_convertvector((f32x2){x[i], x[i + 1]}, bf16x2);
    const uint32_t hw = __builtin_bit_cast(uint32_t, h);
    const float h0 = __uint_as_float(hw << 16), h1 = __uint_as_float(hw & 0xffff0000u);
    const bf16x2 l = __builtin_convertvector((f32x2){x[i] - h0, x[i + 1] - h1}, bf16x2);
    hi[i] = h[0];
    hi[i + 1] = h[1];
    lo[i] = l[0];
    lo[i + 1] = l[1];
  }
}

// The same split for two floats: returns the packed hi pair (a in the low
// half) and stores the packed lo pair.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b, uint32_t* lo) {
  const bf16x2 h = __builtin_convertvector((f32x2){a, b}, bf16x2);
  const uint32_t hw = __builtin_bit_cast(uint32_t, h);
  const float a0 = __uint_as_float(hw << 16), b0 = __uint_as_float(hw & 0xffff0000u);
  *lo = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a - a0, b - b0}, bf16x2));
  return hw;
}

// Round-to-nearest-even conversion of 8 floats to fp16.
__device__ __forceinline__ f16x8 to_f16x8(const float* x) {
  f16x8 h;
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const f16x2 p = __builtin_convertvector((f32x2){x[i], x[i + 1]}, f16x2);
    h[i] = p[0];
    h[i + 1] = p[1];
  }
  return h;
}

// Two bf16 values (one 32-bit word) to two fp16 values, round to nearest even
// (exact when the magnitudes lie in fp16's normal range).
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
  const f32x2 f = {__uint_as_float(w << 16), __uint_as_float(w & 0xffff0000u)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, f16x2));
}

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// LDS transpose read of 4 x 16-bit values: within a 16-lane group, lane
// 4e + q supplies the address of row e, elements 4q..4q+3 (8 bytes), and
// lane i receives element i of the four rows (rows 0..3 in order).
__device__ __forceinline__ v4i16 ds_read_tr16(const void* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left at maximum).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier for the tile ring.  It waits for this wave's own LDS
// reads and writes and synchronises the waves; it does not wait for the
// vector-memory counter, so tile loads already in flight stay in flight (a
// fence-based barrier counts the LDS writes of those loads as pending local
// stores and would drain them).  The memory clobber keeps the compiler from
// moving LDS accesses across it.  Completion of the tile about to be read is
// established before the barrier by an explicit s_waitcnt on vmcnt.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Sum over the 16 lanes that share l/16 (lanes differing in bits 0..3).
__device__ __forceinline__ float sum16(float v) {
  v += __shfl_xor(v, 1);
  v += __shfl_xor(v, 2);
  v += __shfl_xor(v, 4);
  v += __shfl_xor(v, 8);
  return v;
}

// The same 16-lane sum on the VALU through DPP (no LDS traffic): swap within
// pairs, within quads, mirror within half-rows, mirror within the row; every
// lane of the 16-lane row ends with the row total.
__device__ __forceinline__ float sum16_dpp(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));
  return v;
}

// Reductions over the 4 lanes that share l%16 (lanes differing in bits 4..5).
__device__ __forceinline__ float max_over_groups(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}
__device__ __forceinline__ double sum_over_groups(double v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

// Exclusive prefix sum of one value per thread over the whole block
// (blockDim.x a multiple of 64, at most 1024).  `scratch` holds 16 words.
// Every thread receives the block total in *total.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* scratch,
                                                         uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    uint32_t t = __shfl_up(incl, off);
    if (lane >= off) incl += t;
  }
  if (lane == 63) scratch[wave] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
  for (int k = 0; k < nwaves; ++k) {
    uint32_t s = scratch[k];
    if (k < wave) before += s;
    all += s;
  }
  __syncthreads();
  *total = all;
  return before + incl - v;
}

}  // namespace grkv
