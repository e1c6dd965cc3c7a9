// Key-step operator pass (Sec. 3.4 "Key step", Eq. 9-10; App. D.2) on an LDS
// tile ring, for units of up to 128 window rows (padded to 128) and d = 128:
// the kOp and kFinal passes of the first alternating step (K_cur = K0), with
// the contract of key_pass in key.hip.
//
//  * Products are taken transposed, keys x rows: B^T = V* p^T (the V* tile as
//    the A operand, the direction p as B).  X^T, D^T and A^T = D^T W
//    (W = Q Q^T / d is symmetric) then share one layout, and H^T = X^T o A^T
//    is already the B operand of out^T += V*^T H^T once the keys of an
//    operand are ordered {4g .. 4g+3, 16+4g .. 16+4g+3} (g = lane / 16).
//  * X (the retained-set softmax weights at K0 against the retained LSE, zero
//    at invisible and fixed slots) does not change over the conjugate-gradient
//    iterations: key_x writes it once per key step, tile by tile in the lane
//    order the passes read it in, and the passes stream it instead of K0.
//    V* is split once per key step into bf16 hi and lo tensors (key_prep).
//  * One block per (unit, split) of 8 waves in two roles, one of each per
//    SIMD.  Producer waves 0-3 (rows 32w .. 32w+31) run phase A of a tile:
//    B^T and D^T = X^T o (B^T - s); consumer waves 4-7 (the same rows) run
//    phase B of the tile before: A^T = D^T W, H^T, out^T.  Each role holds
//    only its own operands in registers (p, or W and the output), and the
//    MFMAs of one role run beside the operand packing of the other.
//  * A tile (X^T fp32, V* hi, V* lo) goes from HBM straight into a four-stage
//    LDS ring (direct loads, no register staging); two tiles stay in flight
//    while two are read.  V*^T operands come from the row-major V* tiles by
//    the LDS transpose read.
//  * D (row-major, hi and lo) is handed to the consumers through a
//    double-buffered LDS tile; one barrier per interval publishes it, the next
//    ring stage and the stage that is refilled.
//  * Products of fp32 values use three bf16 MFMAs (hi*hi + hi*lo + lo*hi),
//    as in key.hip.
#include <math.h>

#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

constexpr int kRD = 128;                          // head dim
constexpr int kRMP = 128;                         // padded rows
constexpr int kRW = 8;                            // waves: 4 producers, 4 consumers
constexpr int kRTh = kRW * 64;
constexpr int kRTK = 32;                          // keys per tile
constexpr int kRTB = kRTK * kRD * 2;              // one bf16 tensor tile (8 KB)
constexpr int kRXB = kRMP * kRTK * 4;             // X^T of a tile (fp32, 16 KB)
constexpr int kRStage = kRXB + 2 * kRTB;          // X^T, V* hi, V* lo
constexpr int kRDB = kRMP * kRTK * 2;             // one D tile, hi or lo (8 KB)
constexpr int kRLoads = kRStage / 1024 / kRW;     // tile loads per wave per tile (4)

// 16-byte chunk permutation inside a 256-byte V* tile row (key row r): the
// rows are read 16 rows x one chunk and also by the transpose read as 8 rows x
// two adjacent chunks per half wave, which 2 (r mod 8) + (r / 8 mod 2) keeps
// on distinct banks in both.
__device__ __forceinline__ int vswz(int r) { return ((r & 7) << 1) | ((r >> 3) & 1); }
// 8-byte unit permutation inside a 64-byte D row (query row R): the row
// writes (16 rows x 2 units per half wave) and the transpose reads (8 rows x
// 4 units) both land on distinct banks.
__device__ __forceinline__ int dswz(int R) { return ((R >> 2) & 3) << 1; }

struct RingArgs {
  const u16* q;        // [U][m][d]
  const u16* k0;       // [U][c][d]
  const float* xs;     // [U][ceil(c / 32)][4096] X^T tiles (key_x)
  const u16* vh;       // [U][c][d] V* hi
  const u16* vl;       // [U][c][d] V* lo
  const float* lse2;   // [U][mp]
  const float* Fm;     // [U][mp][d]
  const float* W;      // [U][mp][mp]
  float* dir;          // [U][mp][d] direction p (kOp) or alpha (kFinal)
  float* sdot;         // [U][mp] rowdot(F, p) (kOp)
  double* cg;          // [U][4] {r.r, r0.r0, iterations, state}
  float* opart;        // [U][S][mp][d]
  float* hpart;        // [U][S][mp]
  float* kstar;        // [U][c][d]
  float* cg_info;      // [U][4] or null
  int m, w, c, ntc, S, chunk, causal;   // ntc = ceil(c / 32)
  float scale_log2, inv_sqrt_d;
  // kOp with one split per unit (fuse): the conjugate-gradient update of
  // key_cg runs in the pass's epilogue, on alpha, r, p (= dir) and sdot
  int fuse, max_iter;
  float lam_k, tol;
  float* alpha;        // [U][mp][d]
  float* r;            // [U][mp][d]
};

__device__ __forceinline__ bf16x8 cat8(v4i16 a, v4i16 b) {
  return __builtin_bit_cast(bf16x8, (v8i16){a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]});
}

__device__ __forceinline__ uint32_t lds_off(const void* p) {
  return (uint32_t)(uintptr_t)(lds_void*)p;
}

// 16 bytes per lane from HBM straight into LDS: lane source base + voff
// (base wave-uniform, voff a per-lane byte offset), the wave's 1 KB landing
// at the wave-uniform LDS byte offset lds.  Written as inline assembly so that the
// compiler does not track these loads: tracked, they make it wait for every
// outstanding LDS access before each use of one (it no longer counts LDS
// accesses in order) and order accesses to other LDS buffers after them.  The
// ring's own waits (vmcnt, then a barrier) establish completion.
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory", "m0");
}

template <bool FINAL>
__global__ __launch_bounds__(kRTh) void key_ring_kernel(RingArgs a) {
  __shared__ __attribute__((aligned(16))) char stg0[kRStage];
  __shared__ __attribute__((aligned(16))) char stg1[kRStage];
  __shared__ __attribute__((aligned(16))) char stg2[kRStage];
  __shared__ __attribute__((aligned(16))) char stg3[kRStage];
  __shared__ __attribute__((aligned(16))) char dbuf0[2 * kRDB];   // D hi, then D lo
  __shared__ __attribute__((aligned(16))) char dbuf1[2 * kRDB];

  const int u = blockIdx.y, s = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g = lane >> 4;
  const int state = (int)a.cg[u * 4 + 3];
  const int c = a.c, j0 = s * a.chunk, j1 = min(c, j0 + a.chunk);
  if (FINAL && s == 0 && tid == 0 && a.cg_info) {
    const double rr = a.cg[u * 4 + 0], rr0 = a.cg[u * 4 + 1];
    a.cg_info[u * 4 + 0] = (float)a.cg[u * 4 + 2];
    a.cg_info[u * 4 + 1] = rr0 > 0 ? (float)sqrt(rr / rr0) : 0.f;
    a.cg_info[u * 4 + 2] = (float)(state == kKeyRunning ? kKeyMaxIter : state);
    a.cg_info[u * 4 + 3] = (float)sqrt(rr0);
  }
  if (!FINAL && state != kKeyRunning) return;
  if (FINAL && state == kKeySkipped) {
    for (int e = tid; e < (j1 - j0) * kRD; e += kRTh) {
      const size_t o = ((size_t)u * c + j0) * kRD + e;
      a.kstar[o] = bf16_to_f32(a.k0[o]);
    }
    return;
  }
  const int ntiles = j1 > j0 ? (j1 - j0 + kRTK - 1) / kRTK : 0;
  if (ntiles == 0) {
    if constexpr (!FINAL) {
      for (int e = tid; e < kRMP * kRD; e += kRTh)
        a.opart[((size_t)u * a.S + s) * kRMP * kRD + e] = 0.f;
      for (int e = tid; e < kRMP; e += kRTh) a.hpart[((size_t)u * a.S + s) * kRMP + e] = 0.f;
    }
    return;
  }
  const bool producer = wave < 4;
  const int rw = producer ? wave : wave - 4;   // row group of the wave
  const int row0 = 32 * rw;
  const int e = l16 >> 2, qq = l16 & 3;
  const int last = ntiles - 1;

  // tile t of the split into a stage (X^T, V* hi, V* lo: 32 wave loads of
  // 1 KB, four per wave): a uniform base (the tile's start) plus each lane's
  // byte offset; V* rows past the split's end are clamped to its last key
  // (finite data; X is zero there)
  const int tg0 = j0 / kRTK;   // first tile of the split (splits are whole tiles)
  auto issue = [&](int t, char* stage) {
    const int tile0 = j0 + t * kRTK;
#pragma unroll
    for (int it = 0; it < kRLoads; ++it) {
      const int instr = wave * kRLoads + it;      // 0..31
      if (instr < kRXB / 1024) {
        const float* base = a.xs + ((size_t)u * a.ntc + tg0 + t) * (kRXB / 4);
        dma16(base, (uint32_t)(instr * 1024 + lane * 16), lds_off(stage) + instr * 1024);
      } else {
        const int vi = instr - kRXB / 1024, tensor = vi >> 3, part = vi & 7;
        const int r = part * 4 + (lane >> 4), pos = lane & 15;
        const u16* base = (tensor == 0 ? a.vh : a.vl) + ((size_t)u * c + tile0) * kRD;
        const int rr = min(tile0 + r, j1 - 1) - tile0;
        const uint32_t vo = (uint32_t)((rr * kRD + (pos ^ vswz(r)) * 8) * 2);
        dma16(base, vo, lds_off(stage) + kRXB + tensor * kRTB + part * 1024);
      }
    }
  };

  // consumers: out^T of their rows and the row sums of H (phase B)
  f32x4 oacc[FINAL ? 1 : 2][kRD / 16];
#pragma unroll
  for (int rt = 0; rt < (FINAL ? 1 : 2); ++rt)
#pragma unroll
    for (int dt = 0; dt < kRD / 16; ++dt) oacc[rt][dt] = zero4();
  float hs[2] = {0.f, 0.f};

  if (producer) {
    // ---------------------------------------------------------------- phase A
    bf16x8 ph[2][kRD / 32], pl[2][kRD / 32];
    float sd[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const int row = row0 + 16 * rt + l16;
      const float* pr = a.dir + ((size_t)u * kRMP + row) * kRD;
      const float* fr = a.Fm + ((size_t)u * kRMP + row) * kRD;
      float acc = 0.f;
#pragma unroll
      for (int ks = 0; ks < kRD / 32; ++ks) {
        const float4 x0 = *reinterpret_cast<const float4*>(pr + ks * 32 + 8 * g);
        const float4 x1 = *reinterpret_cast<const float4*>(pr + ks * 32 + 8 * g + 4);
        const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
        split8(x, ph[rt][ks], pl[rt][ks]);
        if constexpr (FINAL) {
          const float4 f0 = *reinterpret_cast<const float4*>(fr + ks * 32 + 8 * g);
          const float4 f1 = *reinterpret_cast<const float4*>(fr + ks * 32 + 8 * g + 4);
          acc += x0.x * f0.x + x0.y * f0.y + x0.z * f0.z + x0.w * f0.w;
          acc += x1.x * f1.x + x1.y * f1.y + x1.z * f1.z + x1.w * f1.w;
        }
      }
      if constexpr (FINAL) {
        acc += __shfl_xor(acc, 16);
        acc += __shfl_xor(acc, 32);
        sd[rt] = acc;
      } else {
        sd[rt] = a.sdot[(size_t)u * kRMP + row];
      }
    }
    uint32_t vofs[kRD / 32];   // operand chunk 4ks + g of key row l16
#pragma unroll
    for (int ks = 0; ks < kRD / 32; ++ks)
      vofs[ks] = (uint32_t)(kRXB + l16 * 256 + 16 * ((4 * ks + g) ^ vswz(l16)));
    // D row writes: row row0 + l16 (+16 per row tile), keys 16kt + 4g .. +3
    uint32_t dwo[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int R = row0 + l16;
      dwo[kt] = (uint32_t)(R * 64 + 8 * ((4 * kt + g) ^ dswz(R)));
    }
    const uint32_t xo = (uint32_t)(rw * 4096 + lane * 16);   // this lane's X^T slots

    // Phase A of a tile from stage sa: B^T - s (lane holds
    // [key 16kt + 4g + i][row 16rt + l16]) and D^T = X^T o (B^T - s); D rows
    // to LDS.
    auto phase_a = [&](const char* sa, char* dw) {
      // B^T accumulates from -s, so that it ends as B^T - s
      f32x4 bt[2][2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) bt[kt][rt] = f32x4{-sd[rt], -sd[rt], -sd[rt], -sd[rt]};
      // steps (ks, kt), the operands of the next step read before the MFMAs
      // of this one
      uint4 vhf[2], vlf[2];
      auto rd = [&](int step, int b) {
        const int ks = step >> 1, kt = step & 1;
        vhf[b] = *reinterpret_cast<const uint4*>(sa + vofs[ks] + kt * 4096);
        vlf[b] = *reinterpret_cast<const uint4*>(sa + kRTB + vofs[ks] + kt * 4096);
      };
      rd(0, 0);
#pragma unroll
      for (int step = 0; step < 2 * (kRD / 32); ++step) {
        const int ks = step >> 1, kt = step & 1, b = step & 1;
        if (step + 1 < 2 * (kRD / 32)) rd(step + 1, b ^ 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          bt[kt][rt] = mfma_bf16(as_bf16x8(vhf[b]), ph[rt][ks], bt[kt][rt]);
          bt[kt][rt] = mfma_bf16(as_bf16x8(vlf[b]), ph[rt][ks], bt[kt][rt]);
          bt[kt][rt] = mfma_bf16(as_bf16x8(vhf[b]), pl[rt][ks], bt[kt][rt]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          const f32x4 x = *reinterpret_cast<const f32x4*>(sa + xo + (2 * kt + rt) * 1024);
          float dv[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) dv[i] = x[i] * bt[kt][rt][i];
          uint32_t l0, l1;
          const uint32_t h0 = pack_bf16x2(dv[0], dv[1], &l0);
          const uint32_t h1 = pack_bf16x2(dv[2], dv[3], &l1);
          *reinterpret_cast<uint2*>(dw + rt * 1024 + dwo[kt]) = make_uint2(h0, h1);
          *reinterpret_cast<uint2*>(dw + kRDB + rt * 1024 + dwo[kt]) = make_uint2(l0, l1);
        }
    };

    // tiles 0 and 1 in flight, then interval 0 (phase A of tile 0, tile 2
    // issued); intervals k = 1 .. ntiles-1 in whole groups of four as
    // straight-line code (every access names its ring stage and buffers at
    // compile time), then the remaining zero to three
    wait_vmcnt<0>();   // the constants are in registers before the ring starts
    issue(0, stg0);
    issue(min(1, last), stg1);
    wait_vmcnt<kRLoads>();
    lds_barrier();
    auto interval = [&](int k, const char* sa, char* refill, char* dw) {
      issue(min(k + 2, last), refill);
      phase_a(sa, dw);
      // every interval issues one tile, so exactly one later tile's loads
      // may still be in flight once the next tile has landed
      wait_vmcnt<kRLoads>();
      lds_barrier();
    };
    interval(0, stg0, stg2, dbuf0);
    int k = 1;
    for (; k + 4 <= ntiles; k += 4) {
      interval(k + 0, stg1, stg3, dbuf1);
      interval(k + 1, stg2, stg0, dbuf0);
      interval(k + 2, stg3, stg1, dbuf1);
      interval(k + 3, stg0, stg2, dbuf0);
    }
    if (k < ntiles) interval(k, stg1, stg3, dbuf1);
    if (k + 1 < ntiles) interval(k + 1, stg2, stg0, dbuf0);
    if (k + 2 < ntiles) interval(k + 2, stg3, stg1, dbuf1);
    // the clamped loads past the end land before the block's LDS is released
    wait_vmcnt<0>();
  } else {

  // ------------------------------------------------------------------ phase B
  // kOp: W rows (B operand of A^T = D^T W), columns 32kb + 8g .. +7
  bf16x8 wh[FINAL ? 1 : 2][kRMP / 32], wl[FINAL ? 1 : 2][kRMP / 32];
  // kFinal: Q columns 16 (2 rw + dd) + l16 at rows 32kb + 8g .. +7 (A operand
  // of dK^T = Q^T D)
  bf16x8 qt[FINAL ? 2 : 1][kRMP / 32];
  if constexpr (!FINAL) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const float* wr = a.W + ((size_t)u * kRMP + row0 + 16 * rt + l16) * kRMP;
#pragma unroll
      for (int kb = 0; kb < kRMP / 32; ++kb) {
        const float4 x0 = *reinterpret_cast<const float4*>(wr + 32 * kb + 8 * g);
        const float4 x1 = *reinterpret_cast<const float4*>(wr + 32 * kb + 8 * g + 4);
        const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
        split8(x, wh[rt][kb], wl[rt][kb]);
      }
    }
  } else {
#pragma unroll
    for (int dd = 0; dd < 2; ++dd) {
      const int col = 16 * (2 * rw + dd) + l16;
#pragma unroll
      for (int kb = 0; kb < kRMP / 32; ++kb) {
        u16 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int r = 32 * kb + 8 * g + j;
          v[j] = r < a.m ? a.q[((size_t)u * a.m + r) * kRD + col] : (u16)0;
        }
        qt[dd][kb] = __builtin_bit_cast(bf16x8, v);
      }
    }
  }
  uint32_t vtofs[kRD / 16];   // V* transpose read: key row 4g + e, columns 16 dt + 4qq .. +3
  {
    const int vr = 4 * g + e;
#pragma unroll
    for (int dt = 0; dt < kRD / 16; ++dt)
      vtofs[dt] = (uint32_t)(kRXB + vr * 256 + 16 * ((2 * dt + (qq >> 1)) ^ vswz(vr)) + 8 * (qq & 1));
  }
  // D transpose reads: row 8g + 4h + e (+32 per kb), keys 16kt + 4qq .. +3
  uint32_t dro[2][2];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int R2 = 8 * g + 4 * h + e;
      dro[kt][h] = (uint32_t)(R2 * 64 + 8 * ((4 * kt + qq) ^ dswz(R2)));
    }
  const uint32_t xro = (uint32_t)(rw * 4096 + lane * 16);

  // D^T fragments of row block kb (keys 16kt + l16, rows 32kb + 8g .. +7)
  auto dfrag = [&](const char* dr, int kt, int kb, bf16x8& dh, bf16x8& dl) {
    const char* dp = dr + kb * 2048;
    dh = cat8(ds_read_tr16(dp + dro[kt][0]), ds_read_tr16(dp + dro[kt][1]));
    dl = cat8(ds_read_tr16(dp + kRDB + dro[kt][0]), ds_read_tr16(dp + kRDB + dro[kt][1]));
  };
  // kFinal: K0 of the lane's four d columns at the keys of (kt, dd), for the
  // tile in phase B.  Issued as inline assembly, ahead of the interval's tile
  // loads, and completed by a counted wait that names these registers.
  uint64_t k0r[2][2];
  auto k0load = [&](int t) {
    if constexpr (FINAL) {
      const int tile0 = j0 + t * kRTK;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int dd = 0; dd < 2; ++dd) {
          const int key = min(tile0 + 16 * kt + l16, j1 - 1);
          const u16* p = a.k0 + ((size_t)u * c + key) * kRD + 16 * (2 * rw + dd) + 4 * g;
          asm volatile("global_load_dwordx2 %0, %1, off" : "=v"(k0r[kt][dd]) : "v"(p) : "memory");
        }
    }
  };
  // Phase B of tile t: D_t from dr, X^T and V* from stage sb (tail: the last
  // interval, with no tile loads after the K0 loads).
  auto phase_b = [&](int t, const char* sb, const char* dr, bool tail) {
    if constexpr (!FINAL) {
      // A^T = D^T W in the layout of X^T, steps (kb, kt), the D^T fragments
      // of the next step read before the MFMAs of this one
      f32x4 at[2][2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) at[kt][rt] = zero4();
      bf16x8 dh[2], dl[2];
      dfrag(dr, 0, 0, dh[0], dl[0]);
#pragma unroll
      for (int step = 0; step < 2 * (kRMP / 32); ++step) {
        const int kb = step >> 1, kt = step & 1, b = step & 1;
        if (step + 1 < 2 * (kRMP / 32)) dfrag(dr, (step + 1) & 1, (step + 1) >> 1, dh[b ^ 1], dl[b ^ 1]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          at[kt][rt] = mfma_bf16(dh[b], wh[rt][kb], at[kt][rt]);
          at[kt][rt] = mfma_bf16(dl[b], wh[rt][kb], at[kt][rt]);
          at[kt][rt] = mfma_bf16(dh[b], wl[rt][kb], at[kt][rt]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // V*^T fragments of column block dt (keys ordered as the H^T operand)
      bf16x8 th[2], tl[2];
      auto vfrag = [&](int dt, int b) {
        const char* vp = sb + vtofs[dt];
        th[b] = cat8(ds_read_tr16(vp), ds_read_tr16(vp + 4096));
        tl[b] = cat8(ds_read_tr16(vp + kRTB), ds_read_tr16(vp + kRTB + 4096));
      };
      // X^T of the tile and the first V*^T fragments
      f32x4 xv[2][2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
          xv[kt][rt] = *reinterpret_cast<const f32x4*>(sb + xro + (2 * kt + rt) * 1024);
      vfrag(0, 0);
      // H^T = X^T o A^T as the B operand (keys 4g + j, then 16 + 4g + j)
      bf16x8 hh[2], hl[2];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        float x8[8];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float h = xv[kt][rt][i] * at[kt][rt][i];
            x8[4 * kt + i] = h;
            hs[rt] += h;
          }
        split8(x8, hh[rt], hl[rt]);
      }
      // out^T [d x rows] += V*^T H^T over the tile's 32 keys
#pragma unroll
      for (int dt = 0; dt < kRD / 16; ++dt) {
        const int b = dt & 1;
        if (dt + 1 < kRD / 16) vfrag(dt + 1, b ^ 1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          oacc[rt][dt] = mfma_bf16(th[b], hh[rt], oacc[rt][dt]);
          oacc[rt][dt] = mfma_bf16(th[b], hl[rt], oacc[rt][dt]);
          oacc[rt][dt] = mfma_bf16(tl[b], hh[rt], oacc[rt][dt]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      // dK^T [d x keys] = Q^T D / sqrt(d) for the d columns 16 (2 rw + dd) + ..;
      // lane holds dK[key 16kt + l16][d 16 (2 rw + dd) + 4g + i].  K* = K0 + dK
      // (fixed keys: D = 0, K* = K0 exactly), K0 from the loads issued at the
      // start of the interval (before the tile loads, so that only those may
      // still be in flight once it has landed)
      f32x4 acc[2][2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int dd = 0; dd < 2; ++dd) acc[kt][dd] = zero4();
#pragma unroll
      for (int kb = 0; kb < kRMP / 32; ++kb)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          bf16x8 dh, dl;
          dfrag(dr, kt, kb, dh, dl);
#pragma unroll
          for (int dd = 0; dd < 2; ++dd) {
            acc[kt][dd] = mfma_bf16(qt[dd][kb], dh, acc[kt][dd]);
            acc[kt][dd] = mfma_bf16(qt[dd][kb], dl, acc[kt][dd]);
          }
        }
      if (tail)
        asm volatile("s_waitcnt vmcnt(0)" : "+v"(k0r[0][0]), "+v"(k0r[0][1]), "+v"(k0r[1][0]),
                     "+v"(k0r[1][1]));
      else
        asm volatile("s_waitcnt vmcnt(%4)"
                     : "+v"(k0r[0][0]), "+v"(k0r[0][1]), "+v"(k0r[1][0]), "+v"(k0r[1][1])
                     : "n"(kRLoads));
      const int tile0 = j0 + t * kRTK;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int key = tile0 + 16 * kt + l16;
        if (key < j1) {
#pragma unroll
          for (int dd = 0; dd < 2; ++dd) {
            const uint64_t kv = k0r[kt][dd];
            const f32x4 o = {bf16_to_f32((u16)kv) + acc[kt][dd][0] * a.inv_sqrt_d,
                             bf16_to_f32((u16)(kv >> 16)) + acc[kt][dd][1] * a.inv_sqrt_d,
                             bf16_to_f32((u16)(kv >> 32)) + acc[kt][dd][2] * a.inv_sqrt_d,
                             bf16_to_f32((u16)(kv >> 48)) + acc[kt][dd][3] * a.inv_sqrt_d};
            *reinterpret_cast<f32x4*>(a.kstar + ((size_t)u * c + key) * kRD + 16 * (2 * rw + dd) +
                                      4 * g) = o;
          }
        }
      }
    }
  };

  // the same intervals as the producers: interval 0 only issues; interval k
  // runs phase B of tile k-1; the last one (k = ntiles) needs no barrier
  wait_vmcnt<0>();
  issue(0, stg0);
  issue(min(1, last), stg1);
  wait_vmcnt<kRLoads>();
  lds_barrier();
  issue(min(2, last), stg2);
  wait_vmcnt<kRLoads>();
  lds_barrier();
  auto interval = [&](int k, const char* sb, char* refill, const char* dr) {
    k0load(k - 1);
    issue(min(k + 2, last), refill);
    phase_b(k - 1, sb, dr, false);
    wait_vmcnt<kRLoads>();
    lds_barrier();
  };
  int k = 1;
  for (; k + 4 <= ntiles; k += 4) {
    interval(k + 0, stg0, stg3, dbuf0);
    interval(k + 1, stg1, stg0, dbuf1);
    interval(k + 2, stg2, stg1, dbuf0);
    interval(k + 3, stg3, stg2, dbuf1);
  }
  if (k < ntiles) interval(k, stg0, stg3, dbuf0);
  if (k + 1 < ntiles) interval(k + 1, stg1, stg0, dbuf1);
  if (k + 2 < ntiles) interval(k + 2, stg2, stg1, dbuf0);
  // the last interval: phase B of tile ntiles-1, after every load has landed
  // (its stage and buffers are picked at run time)
  wait_vmcnt<0>();
  {
    const char* sb = (last & 3) == 0 ? stg0 : (last & 3) == 1 ? stg1 : (last & 3) == 2 ? stg2 : stg3;
    const char* dr = (last & 1) ? dbuf1 : dbuf0;
    k0load(last);
    phase_b(last, sb, dr, true);
  }
  }   // roles

  if constexpr (!FINAL) {
    // row sums of H over the whole split (the lanes of a row hold parts)
    float hrow[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      float h = hs[rt];
      h += __shfl_xor(h, 16);
      h += __shfl_xor(h, 32);
      hrow[rt] = h;
    }
    if (!a.fuse) {
      if (!producer) {
        // lane holds out^T [16dt + 4g + i][row 16rt + l16]
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          const int row = row0 + 16 * rt + l16;
          float* op = a.opart + (((size_t)u * a.S + s) * kRMP + row) * kRD;
#pragma unroll
          for (int dt = 0; dt < kRD / 16; ++dt)
            *reinterpret_cast<float4*>(op + 16 * dt + 4 * g) =
                make_float4(oacc[rt][dt][0], oacc[rt][dt][1], oacc[rt][dt][2], oacc[rt][dt][3]);
          if (g == 0) a.hpart[((size_t)u * a.S + s) * kRMP + row] = hrow[rt];
        }
      }
      return;
    }
    // One split holds the whole unit: the conjugate-gradient update of
    // key_cg, spread over all eight waves.  Each thread takes 32 consecutive
    // elements of one row (row tid / 4, columns 32 (tid % 4) ..) and loads
    // its p, F, alpha and r at once, before the barrier; the consumers pass
    // out (rows in stg0 / stg1, 16-byte chunks XOR-swizzled by the row) and
    // the row sums of H (dbuf0) through the now idle ring.  Then
    // Ap = out + lambda_k p - (H 1) o F; alpha += a p, r -= a Ap with
    // a = r.r / p.Ap; p = r + (r'.r' / r.r) p and s = rowdot(F, p) for the
    // next pass.  Sums in fp64, block sums through dbuf1.
    constexpr int kEl = kRMP * kRD / kRTh;   // 32 elements per thread
    const int er = tid >> 2, ec = (tid & 3) * kEl;
    const size_t eo = ((size_t)u * kRMP + er) * kRD + ec;
    f32x4 pv[kEl / 4], fv[kEl / 4], av[kEl / 4], rv[kEl / 4];
    auto prefetch = [&]() {
#pragma unroll
      for (int k = 0; k < kEl / 4; ++k) {
        pv[k] = *reinterpret_cast<const f32x4*>(a.dir + eo + 4 * k);
        fv[k] = *reinterpret_cast<const f32x4*>(a.Fm + eo + 4 * k);
        av[k] = *reinterpret_cast<const f32x4*>(a.alpha + eo + 4 * k);
        rv[k] = *reinterpret_cast<const f32x4*>(a.r + eo + 4 * k);
      }
    };
    const double rr = a.cg[u * 4 + 0], rr0 = a.cg[u * 4 + 1];
    const int it = (int)a.cg[u * 4 + 2] + 1;
    float* hbuf = reinterpret_cast<float*>(dbuf0);
    double* red = reinterpret_cast<double*>(dbuf1);
    // out[row][col] in stg0 (rows < 64) or stg1, at (row % 64) * kRD +
    // 4 * ((col / 4) ^ (row % 16)) + col % 4
    auto oaddr = [&](int row, int ch) {
      float* base = reinterpret_cast<float*>(row < 64 ? stg0 : stg1);
      return base + (row & 63) * kRD + 4 * (ch ^ (row & 15));
    };
    // (the producers, done first, load theirs while the consumers finish;
    // the consumers load theirs once out has left their registers)
    if (producer) prefetch();
    lds_barrier();   // every wave is past its last ring access
    if (!producer) {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        const int row = row0 + 16 * rt + l16;
#pragma unroll
        for (int dt = 0; dt < kRD / 16; ++dt)
          *reinterpret_cast<f32x4*>(oaddr(row, 4 * dt + g)) = oacc[rt][dt];
        if (g == 0) hbuf[row] = hrow[rt];
      }
      prefetch();
    }
    auto block_sum8 = [&](double v, int slot) {
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
      if (lane == 0) red[slot * kRW + wave] = v;
      lds_barrier();
      double t = 0.0;
#pragma unroll
      for (int k = 0; k < kRW; ++k) t += red[slot * kRW + k];
      return t;
    };
    lds_barrier();
    f32x4 ap[kEl / 4];
    double part = 0.0;
    {
      const float h = hbuf[er];
#pragma unroll
      for (int k = 0; k < kEl / 4; ++k) {
        const f32x4 o = *reinterpret_cast<const f32x4*>(oaddr(er, ec / 4 + k));
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ap[k][i] = o[i] + a.lam_k * pv[k][i] - h * fv[k][i];
          part += (double)(pv[k][i] * ap[k][i]);
        }
      }
    }
    const double pap = block_sum8(part, 0);
    if (!(pap > 0)) {
      if (tid == 0) a.cg[u * 4 + 3] = kKeyBreakdown;
      return;
    }
    const float step = (float)(rr / pap);
    part = 0.0;
#pragma unroll
    for (int k = 0; k < kEl / 4; ++k) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        av[k][i] += step * pv[k][i];
        rv[k][i] -= step * ap[k][i];
        part += (double)(rv[k][i] * rv[k][i]);
      }
      *reinterpret_cast<f32x4*>(a.alpha + eo + 4 * k) = av[k];
      *reinterpret_cast<f32x4*>(a.r + eo + 4 * k) = rv[k];
    }
    const double rn = block_sum8(part, 1);
    int st = kKeyRunning;
    if (sqrt(rn) <= (double)a.tol * sqrt(rr0)) st = kKeyConverged;
    else if (it >= a.max_iter) st = kKeyMaxIter;
    if (st == kKeyRunning) {
      const float beta = (float)(rn / rr);
      float sdr = 0.f;
#pragma unroll
      for (int k = 0; k < kEl / 4; ++k) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pv[k][i] = rv[k][i] + beta * pv[k][i];
          sdr += fv[k][i] * pv[k][i];
        }
        *reinterpret_cast<f32x4*>(a.dir + eo + 4 * k) = pv[k];
      }
      // the four threads of a row are adjacent lanes
      sdr += __shfl_xor(sdr, 1);
      sdr += __shfl_xor(sdr, 2);
      if ((tid & 3) == 0) a.sdot[(size_t)u * kRMP + er] = sdr;
    }
    if (tid == 0) {
      a.cg[u * 4 + 0] = rn;
      a.cg[u * 4 + 2] = it;
      a.cg[u * 4 + 3] = st;
    }
  }
}

// V* to bf16 hi + lo.
__global__ __launch_bounds__(256) void key_prep_kernel(const float* __restrict__ v,
                                                       u16* __restrict__ vh, u16* __restrict__ vl,
                                                       size_t n4) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n4;
       i += (size_t)gridDim.x * blockDim.x) {
    const float4 x = reinterpret_cast<const float4*>(v)[i];
    uint32_t l0, l1;
    const uint32_t h0 = pack_bf16x2(x.x, x.y, &l0), h1 = pack_bf16x2(x.z, x.w, &l1);
    reinterpret_cast<uint2*>(vh)[i] = make_uint2(h0, h1);
    reinterpret_cast<uint2*>(vl)[i] = make_uint2(l0, l1);
  }
}

// X^T tiles of the retained set at K0: X = 2^(Q K0^T log2(e) / sqrt(d) - LSE)
// against the retained log-sum-exp (the value step's retained-set softmax),
// zero at slots a row cannot see (past c, or later window positions) and at
// fixed slots.  Tile t of unit u holds keys 32t .. 32t+31 as 16 floats per
// lane of the ring kernel's producer waves: float (((rw * 4 + 2kt + rt) * 64
// + lane) * 4 + i) is X[row 32rw + 16rt + l16][key 32t + 16kt + 4g + i].
// One block of 4 waves (32 rows each) per kXTiles tiles of a unit.
constexpr int kXTiles = 1;

__global__ __launch_bounds__(256) void key_x_kernel(const u16* __restrict__ q,
                                                    const u16* __restrict__ k0,
                                                    const float* __restrict__ lse2,
                                                    const uint8_t* __restrict__ fixed,
                                                    float* __restrict__ xs, int m, int w, int c,
                                                    int ntc, int causal, float scale_log2) {
  const int u = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  uint4 qb[2][kRD / 32];
  float nl[2];
  int vlim[2];
  // (rows past m read row m - 1, in bounds, and are masked: loads without
  // branches are in flight together)
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    const int row = 32 * wave + 16 * rt + l16;
    const bool ok = row < m;
    const u16* qr = q + ((size_t)u * m + min(row, m - 1)) * kRD;
#pragma unroll
    for (int ks = 0; ks < kRD / 32; ++ks) {
      const uint4 v = *reinterpret_cast<const uint4*>(qr + ks * 32 + 8 * g);
      qb[rt][ks] = ok ? v : make_uint4(0, 0, 0, 0);
    }
    const float l2 = lse2[(size_t)u * kRMP + row];   // row < kRMP: in bounds
    nl[rt] = ok ? -l2 : -__builtin_huge_valf();
    // one past the last slot the row sees (the window is the last w slots)
    vlim[rt] = causal ? min(c, c - w + row % w + 1) : c;
  }
  const int t0 = blockIdx.x * kXTiles;
  for (int t = t0; t < min(t0 + kXTiles, ntc); ++t) {
    const int tile0 = t * kRTK;
    f32x4 st[2][2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int key = min(tile0 + 16 * kt + l16, c - 1);
      const u16* kr = k0 + ((size_t)u * c + key) * kRD;
      uint4 kf[kRD / 32];
#pragma unroll
      for (int ks = 0; ks < kRD / 32; ++ks) kf[ks] = *reinterpret_cast<const uint4*>(kr + ks * 32 + 8 * g);
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        st[kt][rt] = zero4();
#pragma unroll
        for (int ks = 0; ks < kRD / 32; ++ks)
          st[kt][rt] = mfma_bf16(as_bf16x8(kf[ks]), as_bf16x8(qb[rt][ks]), st[kt][rt]);
      }
    }
    float* xt = xs + ((size_t)u * ntc + t) * (kRXB / 4);
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      bool fx[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = tile0 + 16 * kt + 4 * g + i;
        const uint8_t f = fixed[(size_t)u * c + min(key, c - 1)];   // loaded without a branch
        fx[i] = (key >= c) | (f != 0);
      }
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        f32x4 x;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = tile0 + 16 * kt + 4 * g + i;
          x[i] = (!fx[i] && key < vlim[rt])
                     ? __builtin_amdgcn_exp2f(fmaf(st[kt][rt][i], scale_log2, nl[rt]))
                     : 0.f;
        }
        *reinterpret_cast<f32x4*>(xt + ((wave * 4 + 2 * kt + rt) * 64 + lane) * 4) = x;
      }
    }
  }
}

}  // namespace

bool key_ring_supported(const Plan& p) {
  return p.mp == kRMP && p.d == kRD && p.dtype == GRKV_BF16;
}

size_t key_x_bytes(const Plan& p) {
  return (size_t)p.U * ((p.c + kRTK - 1) / kRTK) * kRXB;
}

hipError_t launch_key_prep(const Plan& p, const KeyArgs& a, hipStream_t s) {
  const size_t n4 = (size_t)p.U * p.c * p.d / 4;
  size_t blocks = (n4 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(key_prep_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a.vs, a.vh, a.vl, n4);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int ntc = (p.c + kRTK - 1) / kRTK;
  hipLaunchKernelGGL(key_x_kernel, dim3((ntc + kXTiles - 1) / kXTiles, p.U), dim3(256), 0, s, a.q,
                     a.k0, a.lse2, a.fixed, a.xs, p.m, p.w, p.c, ntc,
                     p.opt.causal_window ? 1 : 0,
                     (float)(1.4426950408889634 / sqrt((double)kRD)));
  return hipGetLastError();
}

hipError_t launch_key_ring(const Plan& p, const KeyArgs& ka, bool final, int S, int chunk,
                           float* dir, bool fuse, hipStream_t s) {
  RingArgs a;
  a.q = ka.q;
  a.k0 = ka.k0;
  a.xs = ka.xs;
  a.vh = ka.vh;
  a.vl = ka.vl;
  a.lse2 = ka.lse2;
  a.Fm = ka.Fm;
  a.W = ka.W;
  a.dir = dir;
  a.sdot = ka.sdot;
  a.cg = ka.cg;
  a.opart = ka.opart;
  a.hpart = ka.hpart;
  a.kstar = ka.kstar;
  a.cg_info = ka.cg_info;
  a.m = p.m;
  a.w = p.w;
  a.c = p.c;
  a.ntc = (p.c + kRTK - 1) / kRTK;
  a.S = S;
  a.chunk = chunk;
  a.causal = p.opt.causal_window ? 1 : 0;
  a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)kRD));
  a.inv_sqrt_d = (float)(1.0 / sqrt((double)kRD));
  a.fuse = fuse && !final && S == 1 ? 1 : 0;
  a.max_iter = ka.max_iter;
  a.lam_k = ka.lam_k;
  a.tol = ka.tol;
  a.alpha = ka.alpha;
  a.r = ka.r;
  if (chunk % kRTK != 0) return hipErrorInvalidValue;   // splits are whole tiles
  if (final)
    hipLaunchKernelGGL(key_ring_kernel<true>, dim3(S, p.U), dim3(kRTh), 0, s, a);
  else
    hipLaunchKernelGGL(key_ring_kernel<false>, dim3(S, p.U), dim3(kRTh), 0, s, a);
  return hipGetLastError();
}

}  // namespace grkv
