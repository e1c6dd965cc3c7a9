// Key-step operator pass (Sec. 3.4 "Key step", Eq. 9-10; App. D.2) on an LDS
// tile ring, for units of up to 128 window rows (padded to 128) and d = 128:
// the kOp and kFinal passes of the first alternating step (K_cur = K0), with
// the contract of key_pass in key.hip.
//
//  * Products are taken transposed, keys x rows: S^T = K Q^T and
//    B^T = V* p^T (K and V* tiles as the A operand, Q and the direction p as
//    B).  X^T, D^T and A^T = D^T W (W = Q Q^T / d is symmetric) then share one
//    layout, and H^T = X^T o A^T is already the B operand of
//    out^T += V*^T H^T once the keys of an operand are ordered
//    {4g .. 4g+3, 16+4g .. 16+4g+3} (g = lane / 16).
//  * One block per (unit, split) of 8 waves in two roles, one of each per
//    SIMD.  Producer waves 0-3 (rows 32w .. 32w+31) run phase A of a tile:
//    S^T, B^T, X^T and D^T; consumer waves 4-7 (the same rows) run phase B of
//    the tile before: A^T = D^T W, H^T, out^T.  Each role holds only its own
//    operands in registers (Q and p, or W and the output), and the MFMAs of
//    one role run beside the exponentials and operand packing of the other.
//  * V* is split once per key step into bf16 hi and lo tensors (key_prep), so
//    a tile is three bf16 tensors (K0, V* hi, V* lo) that go from HBM straight
//    into a four-stage LDS ring (global_load_lds, no register staging); two
//    tiles stay in flight while two are read.  V*^T operands come from the
//    row-major V* tiles by the LDS transpose read.
//  * D (row-major, hi and lo) and X^T (in the producer lanes' own order) are
//    handed over through double-buffered LDS; one barrier per interval
//    publishes them, the next ring stage and the stage that is refilled.
//  * The fixed flags of a tile are one 32-bit word (built by key_prep), read
//    by a scalar load.
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
constexpr int kRStage = 3 * kRTB;                 // K0, V* hi, V* lo
constexpr int kRDB = kRMP * kRTK * 2;             // one D tile, hi or lo (8 KB)
constexpr int kRXB = 4 * 16 * 64 * 4;             // X^T of a tile, 16 floats per producer lane
constexpr int kRLoads = 3 * (kRTB / 1024) / kRW;  // tile loads per wave per tile (3)

// 16-byte chunk permutations inside a 256-byte tile row (key row r).  K rows
// are read 16 rows x one chunk (r mod 16 keeps those on distinct banks); V*
// rows are read that way and also by the transpose read as 8 rows x two
// adjacent chunks per half wave, which 2 (r mod 8) + (r / 8 mod 2) serves both.
__device__ __forceinline__ int kswz(int r) { return r & 15; }
__device__ __forceinline__ int vswz(int r) { return ((r & 7) << 1) | ((r >> 3) & 1); }
// 8-byte unit permutation inside a 64-byte D row (query row R): the row
// writes (16 rows x 2 units per half wave) and the transpose reads (8 rows x
// 4 units) both land on distinct banks.
__device__ __forceinline__ int dswz(int R) { return ((R >> 2) & 3) << 1; }

struct RingArgs {
  const u16* q;        // [U][m][d]
  const u16* k0;       // [U][c][d]
  const u16* vh;       // [U][c][d] V* hi
  const u16* vl;       // [U][c][d] V* lo
  const float* lse2;   // [U][mp]
  const float* Fm;     // [U][mp][d]
  const float* W;      // [U][mp][mp]
  const float* dir;    // [U][mp][d] direction p (kOp) or alpha (kFinal)
  const float* sdot;   // [U][mp] rowdot(F, p) (kOp)
  const double* cg;
  float* opart;        // [U][S][mp][d]
  float* hpart;        // [U][S][mp]
  float* kstar;        // [U][c][d]
  float* cg_info;      // [U][4] or null
  int m, w, c, nw, S, chunk, causal;
  float scale_log2, inv_sqrt_d;
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

// fixbits [U][nw]: bit j of word t set when slot 32t + j is fixed (a separate
// read-only argument, so that its wave-uniform reads are scalar loads).
template <bool FINAL>
__global__ __launch_bounds__(kRTh) void key_ring_kernel(RingArgs a,
                                                        const uint32_t* __restrict__ fixbits) {
  __shared__ __attribute__((aligned(16))) char stg0[kRStage];
  __shared__ __attribute__((aligned(16))) char stg1[kRStage];
  __shared__ __attribute__((aligned(16))) char stg2[kRStage];
  __shared__ __attribute__((aligned(16))) char stg3[kRStage];
  __shared__ __attribute__((aligned(16))) char dbuf0[2 * kRDB];   // D hi, then D lo
  __shared__ __attribute__((aligned(16))) char dbuf1[2 * kRDB];
  __shared__ __attribute__((aligned(16))) char xbuf0[kRXB];
  __shared__ __attribute__((aligned(16))) char xbuf1[kRXB];

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

  // tile t of the split into a stage (K0, V* hi, V* lo: 24 wave loads of
  // 1 KB, three per wave), rows past the split's end clamped to its last key
  // (finite data, masked below)
  // tile t of the split into a stage (K0, V* hi, V* lo: 24 wave loads of
  // 1 KB, three per wave): a uniform base (the tile's first row) plus each
  // lane's byte offset (its row and chunk); rows past the split's end are
  // clamped to its last key (finite data, masked below)
  auto issue = [&](int t, char* stage) {
    const int tile0 = j0 + t * kRTK;
#pragma unroll
    for (int it = 0; it < kRLoads; ++it) {
      const int instr = wave * kRLoads + it;      // 0..23
      const int tensor = instr >> 3, part = instr & 7;
      const int r = part * 4 + (lane >> 4), pos = lane & 15;
      const u16* base = (tensor == 0 ? a.k0 : tensor == 1 ? a.vh : a.vl) + ((size_t)u * c + tile0) * kRD;
      const int rr = min(tile0 + r, j1 - 1) - tile0;
      const uint32_t vo = (uint32_t)((rr * kRD + (pos ^ (tensor == 0 ? kswz(r) : vswz(r))) * 8) * 2);
      dma16(base, vo, lds_off(stage) + tensor * kRTB + part * 1024);
    }
  };

  if (producer) {
    // ---------------------------------------------------------------- phase A
    uint4 qb[2][kRD / 32];
    bf16x8 ph[2][kRD / 32], pl[2][kRD / 32];
    float sd[2], nl[2];
    int vlim[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const int row = row0 + 16 * rt + l16;
      const bool ok = row < a.m;
      const u16* qr = a.q + ((size_t)u * a.m + row) * kRD;
      const float* pr = a.dir + ((size_t)u * kRMP + row) * kRD;
      const float* fr = a.Fm + ((size_t)u * kRMP + row) * kRD;
      float acc = 0.f;
#pragma unroll
      for (int ks = 0; ks < kRD / 32; ++ks) {
        qb[rt][ks] = ok ? *reinterpret_cast<const uint4*>(qr + ks * 32 + 8 * g) : make_uint4(0, 0, 0, 0);
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
      nl[rt] = ok ? -a.lse2[(size_t)u * kRMP + row] : -__builtin_huge_valf();
      // one past the last slot the row sees: the split's end, or its own
      // window position (the window is the last w retained slots)
      vlim[rt] = a.causal ? min(j1, c - a.w + row % a.w + 1) : j1;
    }
    uint32_t kofs[kRD / 32], vofs[kRD / 32];   // operand chunk 4ks + g of key row l16
#pragma unroll
    for (int ks = 0; ks < kRD / 32; ++ks) {
      kofs[ks] = (uint32_t)(l16 * 256 + 16 * ((4 * ks + g) ^ kswz(l16)));
      vofs[ks] = (uint32_t)(kRTB + l16 * 256 + 16 * ((4 * ks + g) ^ vswz(l16)));
    }
    // D row writes: row row0 + l16 (+16 per row tile), keys 16kt + 4g .. +3
    uint32_t dwo[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int R = row0 + l16;
      dwo[kt] = (uint32_t)(R * 64 + 8 * ((4 * kt + g) ^ dswz(R)));
    }
    const uint32_t xwo = (uint32_t)(rw * 4096 + lane * 16);
    const uint32_t* fb = fixbits + (size_t)u * a.nw + j0 / kRTK;

    // Phase A of tile t from stage sa: S^T and B^T (lane holds
    // [key 16kt + 4g + i][row 16rt + l16]), X^T = softmax weights against the
    // retained LSE, D^T = X^T o (B^T - s) with the fixed keys' columns zero;
    // D rows and X^T to LDS.
    auto phase_a = [&](int t, uint32_t fx, const char* sa, char* dw, char* xw) {
      // B^T accumulates from -s, so that it ends as B^T - s
      f32x4 st[2][2], bt[2][2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          st[kt][rt] = zero4();
          bt[kt][rt] = f32x4{-sd[rt], -sd[rt], -sd[rt], -sd[rt]};
        }
      // steps (ks, kt), the operands of the next step read before the MFMAs
      // of this one
      uint4 kf[2], vhf[2], vlf[2];
      auto rd = [&](int step, int b) {
        const int ks = step >> 1, kt = step & 1;
        kf[b] = *reinterpret_cast<const uint4*>(sa + kofs[ks] + kt * 4096);
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
          st[kt][rt] = mfma_bf16(as_bf16x8(kf[b]), as_bf16x8(qb[rt][ks]), st[kt][rt]);
          bt[kt][rt] = mfma_bf16(as_bf16x8(vhf[b]), ph[rt][ks], bt[kt][rt]);
          bt[kt][rt] = mfma_bf16(as_bf16x8(vlf[b]), ph[rt][ks], bt[kt][rt]);
          bt[kt][rt] = mfma_bf16(as_bf16x8(vhf[b]), pl[rt][ks], bt[kt][rt]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      const int tile0 = j0 + t * kRTK;
      float xk[2][2][4];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const int kb0 = 16 * kt + 4 * g;              // the lane's first key in the tile
        const uint32_t fr4 = (fx >> kb0) & 0xfu;      // fixed flags of its four keys
        float dv[2][4];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          // keys i < nvis of the four are live and visible to the row; X is
          // zero at the others and at fixed keys (whose D^T and H^T rows
          // vanish either way)
          const int nvis = vlim[rt] - tile0 - kb0;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool keep = i < nvis && ((fr4 >> i) & 1u) == 0;
            const float x =
                keep ? __builtin_amdgcn_exp2f(fmaf(st[kt][rt][i], a.scale_log2, nl[rt])) : 0.f;
            xk[kt][rt][i] = x;
            dv[rt][i] = x * bt[kt][rt][i];
          }
        }
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          uint32_t l0, l1;
          const uint32_t h0 = pack_bf16x2(dv[rt][0], dv[rt][1], &l0);
          const uint32_t h1 = pack_bf16x2(dv[rt][2], dv[rt][3], &l1);
          *reinterpret_cast<uint2*>(dw + rt * 1024 + dwo[kt]) = make_uint2(h0, h1);
          *reinterpret_cast<uint2*>(dw + kRDB + rt * 1024 + dwo[kt]) = make_uint2(l0, l1);
        }
      }
      // X^T: 16 floats per lane, slot (2kt + rt) of 4, each a 1 KB row of lanes
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          *reinterpret_cast<f32x4*>(xw + xwo + (2 * kt + rt) * 1024) =
              f32x4{xk[kt][rt][0], xk[kt][rt][1], xk[kt][rt][2], xk[kt][rt][3]};
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
    auto interval = [&](int k, const char* sa, char* refill, char* dw, char* xw) {
      issue(min(k + 2, last), refill);
      phase_a(k, fb[k], sa, dw, xw);
      // every interval issues one tile, so exactly one later tile's loads
      // may still be in flight once the next tile has landed
      wait_vmcnt<kRLoads>();
      lds_barrier();
    };
    interval(0, stg0, stg2, dbuf0, xbuf0);
    int k = 1;
    for (; k + 4 <= ntiles; k += 4) {
      interval(k + 0, stg1, stg3, dbuf1, xbuf1);
      interval(k + 1, stg2, stg0, dbuf0, xbuf0);
      interval(k + 2, stg3, stg1, dbuf1, xbuf1);
      interval(k + 3, stg0, stg2, dbuf0, xbuf0);
    }
    if (k < ntiles) interval(k, stg1, stg3, dbuf1, xbuf1);
    if (k + 1 < ntiles) interval(k + 1, stg2, stg0, dbuf0, xbuf0);
    if (k + 2 < ntiles) interval(k + 2, stg3, stg1, dbuf1, xbuf1);
    // the clamped loads past the end land before the block's LDS is released
    wait_vmcnt<0>();
    return;
  }

  // ------------------------------------------------------------------ phase B
  // kOp: W rows (B operand of A^T = D^T W), columns 32kb + 8g .. +7
  bf16x8 wh[FINAL ? 1 : 2][kRMP / 32], wl[FINAL ? 1 : 2][kRMP / 32];
  // kFinal: Q columns 16 (2 rw + dd) + l16 at rows 32kb + 8g .. +7 (B operand
  // of dK = D^T Q)
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
      vtofs[dt] = (uint32_t)(kRTB + vr * 256 + 16 * ((2 * dt + (qq >> 1)) ^ vswz(vr)) + 8 * (qq & 1));
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

  f32x4 oacc[FINAL ? 1 : 2][kRD / 16];
#pragma unroll
  for (int rt = 0; rt < (FINAL ? 1 : 2); ++rt)
#pragma unroll
    for (int dt = 0; dt < kRD / 16; ++dt) oacc[rt][dt] = zero4();
  float hs[2] = {0.f, 0.f};

  // D^T fragments of row block kb (keys 16kt + l16, rows 32kb + 8g .. +7)
  auto dfrag = [&](const char* dr, int kt, int kb, bf16x8& dh, bf16x8& dl) {
    const char* dp = dr + kb * 2048;
    dh = cat8(ds_read_tr16(dp + dro[kt][0]), ds_read_tr16(dp + dro[kt][1]));
    dl = cat8(ds_read_tr16(dp + kRDB + dro[kt][0]), ds_read_tr16(dp + kRDB + dro[kt][1]));
  };
  // Phase B of tile t: D_t from dr, X^T from xr, the tile's V* (or K0) from
  // stage sb.
  auto phase_b = [&](int t, const char* sb, const char* dr, const char* xr) {
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
          xv[kt][rt] = *reinterpret_cast<const f32x4*>(xr + xro + (2 * kt + rt) * 1024);
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
      // dK [keys x d] = D^T Q / sqrt(d) for the d columns 16 (2 rw + dd) + l16;
      // K* = K0 + dK (fixed keys: D^T = 0, K* = K0 exactly)
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
            acc[kt][dd] = mfma_bf16(dh, qt[dd][kb], acc[kt][dd]);
            acc[kt][dd] = mfma_bf16(dl, qt[dd][kb], acc[kt][dd]);
          }
        }
      const int tile0 = j0 + t * kRTK;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int dd = 0; dd < 2; ++dd) {
          const int col = 16 * (2 * rw + dd) + l16;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = 16 * kt + 4 * g + i;
            const int key = tile0 + r;
            if (key < j1) {
              const u16 k0v = *reinterpret_cast<const u16*>(
                  sb + r * 256 + 16 * ((col >> 3) ^ kswz(r)) + 2 * (col & 7));
              a.kstar[((size_t)u * c + key) * kRD + col] =
                  bf16_to_f32(k0v) + acc[kt][dd][i] * a.inv_sqrt_d;
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
  auto interval = [&](int k, const char* sb, char* refill, const char* dr, const char* xr) {
    issue(min(k + 2, last), refill);
    phase_b(k - 1, sb, dr, xr);
    wait_vmcnt<kRLoads>();
    lds_barrier();
  };
  int k = 1;
  for (; k + 4 <= ntiles; k += 4) {
    interval(k + 0, stg0, stg3, dbuf0, xbuf0);
    interval(k + 1, stg1, stg0, dbuf1, xbuf1);
    interval(k + 2, stg2, stg1, dbuf0, xbuf0);
    interval(k + 3, stg3, stg2, dbuf1, xbuf1);
  }
  if (k < ntiles) interval(k, stg0, stg3, dbuf0, xbuf0);
  if (k + 1 < ntiles) interval(k + 1, stg1, stg0, dbuf1, xbuf1);
  if (k + 2 < ntiles) interval(k + 2, stg2, stg1, dbuf0, xbuf0);
  // the last interval: phase B of tile ntiles-1, after every load has landed
  // (its stage and buffers are picked at run time)
  wait_vmcnt<0>();
  {
    const char* sb = (last & 3) == 0 ? stg0 : (last & 3) == 1 ? stg1 : (last & 3) == 2 ? stg2 : stg3;
    const char* dr = (last & 1) ? dbuf1 : dbuf0;
    const char* xr = (last & 1) ? xbuf1 : xbuf0;
    phase_b(last, sb, dr, xr);
  }

  if constexpr (!FINAL) {
    // lane holds out^T [16dt + 4g + i][row 16rt + l16]
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const int row = row0 + 16 * rt + l16;
      float* op = a.opart + (((size_t)u * a.S + s) * kRMP + row) * kRD;
#pragma unroll
      for (int dt = 0; dt < kRD / 16; ++dt)
        *reinterpret_cast<float4*>(op + 16 * dt + 4 * g) =
            make_float4(oacc[rt][dt][0], oacc[rt][dt][1], oacc[rt][dt][2], oacc[rt][dt][3]);
      float h = hs[rt];
      h += __shfl_xor(h, 16);
      h += __shfl_xor(h, 32);
      if (g == 0) a.hpart[((size_t)u * a.S + s) * kRMP + row] = h;
    }
  }
}

// V* to bf16 hi + lo, and the fixed flags to one bit per slot (bit j of word
// t is slot 32t + j; slots past c count as fixed).
__global__ __launch_bounds__(256) void key_prep_kernel(const float* __restrict__ v,
                                                       u16* __restrict__ vh, u16* __restrict__ vl,
                                                       size_t n4, const uint8_t* __restrict__ fixed,
                                                       uint32_t* __restrict__ bits, int U, int c,
                                                       int nw) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  const size_t t0 = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  for (size_t i = t0; i < n4; i += stride) {
    const float4 x = reinterpret_cast<const float4*>(v)[i];
    uint32_t l0, l1;
    const uint32_t h0 = pack_bf16x2(x.x, x.y, &l0), h1 = pack_bf16x2(x.z, x.w, &l1);
    reinterpret_cast<uint2*>(vh)[i] = make_uint2(h0, h1);
    reinterpret_cast<uint2*>(vl)[i] = make_uint2(l0, l1);
  }
  for (size_t i = t0; i < (size_t)U * nw; i += stride) {
    const int u = (int)(i / nw), t = (int)(i % nw);
    uint32_t b = 0;
    for (int j = 0; j < 32; ++j) {
      const int slot = 32 * t + j;
      if (slot >= c || fixed[(size_t)u * c + slot]) b |= 1u << j;
    }
    bits[i] = b;
  }
}

}  // namespace

bool key_ring_supported(const Plan& p) {
  return p.mp == kRMP && p.d == kRD && p.dtype == GRKV_BF16;
}

size_t key_fixbits_words(const Plan& p) { return (size_t)(p.c + kRTK - 1) / kRTK; }

hipError_t launch_key_prep(const Plan& p, const KeyArgs& a, hipStream_t s) {
  const size_t n4 = (size_t)p.U * p.c * p.d / 4;
  size_t blocks = (n4 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(key_prep_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a.vs, a.vh, a.vl,
                     n4, a.fixed, a.fixbits, p.U, p.c, (int)key_fixbits_words(p));
  return hipGetLastError();
}

hipError_t launch_key_ring(const Plan& p, const KeyArgs& ka, bool final, int S, int chunk,
                           const float* dir, hipStream_t s) {
  RingArgs a;
  a.q = ka.q;
  a.k0 = ka.k0;
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
  a.nw = (int)key_fixbits_words(p);
  a.S = S;
  a.chunk = chunk;
  a.causal = p.opt.causal_window ? 1 : 0;
  a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)kRD));
  a.inv_sqrt_d = (float)(1.0 / sqrt((double)kRD));
  if (final)
    hipLaunchKernelGGL(key_ring_kernel<true>, dim3(S, p.U), dim3(kRTh), 0, s, a, ka.fixbits);
  else
    hipLaunchKernelGGL(key_ring_kernel<false>, dim3(S, p.U), dim3(kRTh), 0, s, a, ka.fixbits);
  return hipGetLastError();
}

}  // namespace grkv
