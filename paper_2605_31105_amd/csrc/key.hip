// Key step of GRKV on the bf16 path: the local linearized dual ridge update of
// the free retained keys (Sec. 3.4 "Key step" and "Linearized dual solution",
// Eq. 9-10; Algorithm 1, key step; App. D.2 and D.3), run after the value step
// with the merged values V* held fixed and K_cur = K0 (one alternating step).
//
// With X = softmax(Q K0^T / sqrt(d)) (the retained-set attention of the value
// step), F = X V* = f(K0) and W = Q Q^T / d, the operator of the dual system
// is applied matrix-free:
//   J_G^T a : D = X o (a V*^T - rowdot(F, a) 1^T) with the fixed columns zeroed,
//             dK_j = sum_r D_rj q_r / sqrt(d);
//   J_G dK  : H = X o (W D) (the logit change is Q dK^T / sqrt(d) = W D),
//             J_G dK = H V* - diag(H 1) F;
// so (J_G J_G^T + lambda_k I) a needs no stored Jacobian.  The right-hand side
// is E = Y - f(K0), which after the value step equals lambda_v Z in closed
// form (Y - X V* = lambda_v Z), so F = Y - lambda_v Z as well.  The system is
// solved by conjugate gradients from a = 0 (App. D.2); K* = K0 + J_G^T a.
//
// Kernels: key_init (one block per unit: F, E, W, CG state), key_pass (the
// operator, or the final J_G^T a, over the retained keys in splits), key_cg
// (one block per unit: combines the split partials, one CG update).  The
// host enqueues max_iter pairs of key_pass + key_cg; a unit that has converged
// makes both return at once.
//
// key_pass: a block holds all m rows of one unit and a split of its retained
// keys, one wave per 16 rows.  Keys come in tiles of 32: K0 rows (bf16) and V*
// rows split into bf16 hi + lo parts are staged in LDS, V* also transposed.  A
// wave computes, for its 16 rows, S = Q K^T and B = a V*^T on the MFMA (the
// result holds each lane's key column), D = X o (B - s), and writes D to LDS
// transposed for the other waves; then A = W D (W rows in registers, D from
// LDS) arrives in the same layout as X, so H = X o A needs no second product.
// H goes through a small per-wave LDS area into the operand layout of
// out^T += V*^T H^T.  Products of fp32 values use three bf16 MFMAs
// (hi*hi + hi*lo + lo*hi).
#include <math.h>

#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

constexpr int kKT = 32;   // retained keys per tile (the key orders below assume 32)
constexpr int kKeyEarlyIters = 13;  // CG iterations run with the fewest splits
constexpr int kKeyRingEarlyIters = 16;  // the same for the ring passes
constexpr int kInitBatch = 8;           // key_init: elements a thread loads together
constexpr int kCgBatch = 4;             // key_cg: split partials a thread loads together

// Position, inside a block of 32, of the index a lane holds as element j of an
// MFMA operand when the operand comes from an MFMA result: elements
// {4g + i} and {16 + 4g + i} (i < 4) of group g become 8g + i and 8g + 4 + i,
// so the eight values of a lane sit next to each other.
__device__ __forceinline__ int kperm(int x) {
  const int b = x & ~31, o = x & 31;
  return b + ((o & 15) >> 2) * 8 + (o >> 4) * 4 + (o & 3);
}

__device__ __forceinline__ float dot4(float4 a, float4 b) {
  return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
}

__device__ __forceinline__ double block_sum(double v, double* red) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double t = 0;
  for (int k = 0; k < nw; ++k) t += red[k];
  return t;
}

// ------------------------------------------------------------------ init ----
template <int MP, int D>
__global__ __launch_bounds__(256) void key_init_kernel(
    const u16* __restrict__ q, const float* __restrict__ y, const float* __restrict__ zt,
    const float* __restrict__ stats_ws, float lam_v, int m, float* __restrict__ Fm,
    float* __restrict__ alpha, float* __restrict__ r, float* __restrict__ p,
    float* __restrict__ sdot, float* __restrict__ W, double* __restrict__ cg) {
  __shared__ double red[4];
  // E = lam_v Z and F = Y - E of this unit, rows padded by one float
  constexpr int ES = D + 1;
  __shared__ float Es[MP * ES], Fs[MP * ES];
  const int u = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g = lane >> 4;
  const bool skip = stats_ws[u * 4 + 3] != 0.f;
  // Z^T is [d][mp]: read along its rows (coalesced), store transposed.  A
  // thread loads kInitBatch elements before it uses them; every row of the
  // [mp]-row arrays is read (in bounds) and rows past m are masked.
  constexpr int NE = MP * D;
  static_assert(NE % (256 * kInitBatch) == 0, "whole batches");
  for (int e0 = tid; e0 < NE; e0 += 256 * kInitBatch) {
    float zv[kInitBatch];
#pragma unroll
    for (int b = 0; b < kInitBatch; ++b) zv[b] = zt[(size_t)u * D * MP + e0 + 256 * b];
#pragma unroll
    for (int b = 0; b < kInitBatch; ++b) {
      const int e = e0 + 256 * b, col = e / MP, row = e % MP;
      Es[row * ES + col] = (!skip && row < m) ? lam_v * zv[b] : 0.f;
    }
  }
  __syncthreads();
  double ee = 0;
  for (int e0 = tid; e0 < NE; e0 += 256 * kInitBatch) {
    float yv[kInitBatch];
#pragma unroll
    for (int b = 0; b < kInitBatch; ++b) yv[b] = y[(size_t)u * MP * D + e0 + 256 * b];
#pragma unroll
    for (int b = 0; b < kInitBatch; ++b) {
      const int e = e0 + 256 * b, row = e / D, col = e % D;
      const size_t o = (size_t)u * MP * D + e;
      const float E = Es[row * ES + col];
      const float F = row < m ? yv[b] - E : 0.f;
      Fs[row * ES + col] = F;
      Fm[o] = F;
      alpha[o] = 0.f;
      r[o] = E;
      p[o] = E;
      ee += (double)E * E;
    }
  }
  __syncthreads();
  // s = rowdot(F, p) for the first direction p = E, summed over the columns
  // in order (one thread per row, from LDS)
  for (int row = tid; row < MP; row += 256) {
    float acc = 0.f;
    if (!skip && row < m)
      for (int col = 0; col < D; ++col) acc += Fs[row * ES + col] * Es[row * ES + col];
    sdot[(size_t)u * MP + row] = acc;
  }
  // W = Q Q^T / d (bf16 products are exact; fp32 sums)
  const u16* qu = q + (size_t)u * m * D;
  for (int t = wave; t < (MP / 16) * (MP / 16); t += 4) {
    const int ta = t / (MP / 16), tb = t % (MP / 16);
    const int ra = ta * 16 + l16, rb = tb * 16 + l16;
    f32x4 acc = zero4();
    // (rows past m read row m - 1 and are masked: no branches around the loads)
    uint4 av[D / 32], bv[D / 32];
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      av[ks] = *reinterpret_cast<const uint4*>(qu + (size_t)min(ra, m - 1) * D + ks * 32 + 8 * g);
      bv[ks] = *reinterpret_cast<const uint4*>(qu + (size_t)min(rb, m - 1) * D + ks * 32 + 8 * g);
    }
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const uint4 a = ra < m ? av[ks] : make_uint4(0, 0, 0, 0);
      const uint4 b = rb < m ? bv[ks] : make_uint4(0, 0, 0, 0);
      acc = mfma_bf16(as_bf16x8(a), as_bf16x8(b), acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
      W[((size_t)u * MP + ta * 16 + 4 * g + i) * MP + tb * 16 + l16] = acc[i] * (1.f / D);
  }
  ee = block_sum(ee, red);
  if (tid == 0) {
    cg[u * 4 + 0] = ee;
    cg[u * 4 + 1] = ee;
    cg[u * 4 + 2] = 0;
    cg[u * 4 + 3] = skip ? kKeySkipped : ee == 0 ? kKeyConverged : kKeyRunning;
  }
}

// ------------------------------------------------------------------ pass ----
enum { kOp = 0, kFinal = 1, kJvp = 2 };   // key_pass modes

// LDS regions (bf16 elements).  KF: the current keys are fp32 (later
// alternating steps) and are held as bf16 hi + lo; JVP: the tile of
// G = K_cur - K0 (hi + lo) replaces D^T.
template <int MP, int D, int KM, bool KF>
struct KeyLds {
  static constexpr int KS = D + 8;     // row stride (bf16) of K, G and V rows
  static constexpr int TS = kKT + 8;   // row stride of V^T rows
  static constexpr int DS = MP + 8;    // row stride of D^T rows
  static constexpr int QS = MP + 8;    // row stride of Q^T rows
  static constexpr int HS = kKT + 8;   // row stride of a wave's H rows
  static constexpr int k = 0;                                   // K (hi)
  static constexpr int kl = k + kKT * KS;                       // K lo
  static constexpr int vh = kl + (KF ? kKT * KS : 0);
  static constexpr int vl = vh + kKT * KS;
  static constexpr int th = vl + kKT * KS;
  static constexpr int tl = th + D * TS;
  static constexpr int dh = tl + D * TS;                        // D^T hi / G hi
  static constexpr int dl = dh + kKT * (KM == kJvp ? KS : DS);  // D^T lo / G lo
  static constexpr int hh = dl + kKT * (KM == kJvp ? KS : DS);  // [NW][16][HS] H hi, then lo
  static constexpr int hl = hh + (KM == kFinal ? 0 : MP * HS);
  static constexpr int qt = hl + (KM == kFinal ? 0 : MP * HS);
  static constexpr int end = qt + (KM == kFinal ? D * QS : 0);
  static constexpr size_t bytes() { return (size_t)end * sizeof(u16) + kKT * (sizeof(int) + 1); }
};

// One pass over a split of the retained keys of unit blockIdx.y, with X from
// the current keys (K0 in bf16, or fp32 K_cur when KF) and the retained LSE.
//   kOp:    partial sums of H V* (opart) and H 1 (hpart) for the direction p,
//           H = X o (W D), D = X o (p V*^T - rowdot(F, p)) with fixed columns 0;
//   kJvp:   the same partials for H = X o (Q G^T / sqrt(d)), G = K_cur - K0
//           (the J_G G term of the right-hand side at later steps);
//   kFinal: K* = K0 + J_G^T alpha for the split's keys.
template <int MP, int D, int KM, bool KF>
__global__ __launch_bounds__(MP / 16 * 64) void key_pass_kernel(
    const u16* __restrict__ q, const u16* __restrict__ k0, const float* __restrict__ kcur,
    const float* __restrict__ vs, const float* __restrict__ lse2,
    const uint8_t* __restrict__ fixed, const int32_t* __restrict__ idx,
    const float* __restrict__ Fm, const float* __restrict__ W, const float* __restrict__ pv,
    const float* __restrict__ sdot_in, const double* __restrict__ cg, float* __restrict__ opart,
    float* __restrict__ hpart, float* __restrict__ kstar, float* __restrict__ cg_info, int m,
    int w, int64_t n, int c, int S, int chunk, int causal, float scale_log2, float inv_sqrt_d) {
  constexpr bool FINAL = KM == kFinal, JVP = KM == kJvp;
  constexpr int NW = MP / 16, NTH = NW * 64;
  constexpr int KCH = kKT * D / 8;            // 16-byte chunks of a bf16 K tile
  constexpr int KPT = (KCH + NTH - 1) / NTH;
  constexpr int KCH4 = kKT * D / 4;           // 4-element pieces of an fp32 K tile
  constexpr int KPT4 = (KCH4 + NTH - 1) / NTH;
  // V staging unit: keys {k, k + 16} x four columns, so that both the row-major
  // copy (8-byte pieces) and the transposed copy (4-byte pieces) are written
  // without 2-byte stores
  constexpr int VUN = 16 * (D / 4);
  constexpr int VPT = (VUN + NTH - 1) / NTH;
  constexpr float NEG_INF = -__builtin_huge_valf();
  using L = KeyLds<MP, D, KM, KF>;
  extern __shared__ __attribute__((aligned(16))) u16 sm[];
  int* kp_s = reinterpret_cast<int*>(sm + L::end);
  uint8_t* fx_s = reinterpret_cast<uint8_t*>(kp_s + kKT);

  const int u = blockIdx.y, s = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g = lane >> 4;
  const int state = (int)cg[u * 4 + 3];
  const int j0 = s * chunk, j1 = min(c, j0 + chunk);
  if (FINAL && s == 0 && tid == 0 && cg_info) {
    const double rr = cg[u * 4 + 0], rr0 = cg[u * 4 + 1];
    cg_info[u * 4 + 0] = (float)cg[u * 4 + 2];
    cg_info[u * 4 + 1] = rr0 > 0 ? (float)sqrt(rr / rr0) : 0.f;
    cg_info[u * 4 + 2] = (float)(state == kKeyRunning ? kKeyMaxIter : state);
    cg_info[u * 4 + 3] = (float)sqrt(rr0);
  }
  if (!FINAL && state != kKeyRunning) return;
  if (FINAL && state == kKeySkipped) {
    for (int e = tid; e < (j1 - j0) * D; e += NTH) {
      const size_t o = ((size_t)u * c + j0) * D + e;
      kstar[o] = bf16_to_f32(k0[o]);
    }
    return;
  }

  // register-staged tile loads
  const u16* ku = k0 + (size_t)u * c * D;
  const float* kf = KF ? kcur + (size_t)u * c * D : nullptr;
  const float* vu = vs + (size_t)u * c * D;
  uint4 kreg[KF ? 1 : KPT];
  float4 kfreg[KF ? KPT4 : 1];
  uint2 k0reg[JVP ? KPT4 : 1];
  float4 vreg[VPT][2];
  int kpreg = 0, fxreg = 1;
  // loads clamp the key into the split and zero what lies beyond it
  auto load_tile = [&](int t0) {
    if constexpr (KF) {
#pragma unroll
      for (int k = 0; k < KPT4; ++k) {
        const int e = min(tid + k * NTH, KCH4 - 1);
        const int key = e / (D / 4), ch = e % (D / 4);
        const size_t o = (size_t)min(t0 + key, j1 - 1) * D + ch * 4;
        const float4 v = *reinterpret_cast<const float4*>(kf + o);
        kfreg[k] = t0 + key < j1 ? v : make_float4(0.f, 0.f, 0.f, 0.f);
        if constexpr (JVP) {
          const uint2 b = *reinterpret_cast<const uint2*>(ku + o);
          k0reg[k] = t0 + key < j1 ? b : make_uint2(0, 0);
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < KPT; ++k) {
        const int e = min(tid + k * NTH, KCH - 1);
        const int key = e / (D / 8), ch = e % (D / 8);
        const uint4 v = *reinterpret_cast<const uint4*>(ku + (size_t)min(t0 + key, j1 - 1) * D + ch * 8);
        kreg[k] = t0 + key < j1 ? v : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int k = 0; k < VPT; ++k) {
      const int e = min(tid + k * NTH, VUN - 1);
      const int kp = e % 16, dq = e / 16;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int key = t0 + kp + 16 * h;
        const float4 v = *reinterpret_cast<const float4*>(vu + (size_t)min(key, j1 - 1) * D + 4 * dq);
        vreg[k][h] = key < j1 ? v : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
    if (tid < kKT) {
      const int key = t0 + tid, kc = min(key, j1 - 1);
      const int pv_ = idx[(size_t)u * c + kc];
      const int fv_ = fixed[(size_t)u * c + kc];
      kpreg = key < j1 ? pv_ : 0x7fffffff;
      fxreg = key < j1 ? fv_ : 1;
    }
  };
  auto store_tile = [&]() {
    if constexpr (KF) {
#pragma unroll
      for (int k = 0; k < KPT4; ++k) {
        const int e = tid + k * NTH;
        if (e < KCH4) {
          const int key = e / (D / 4), ch = e % (D / 4);
          const int o = key * L::KS + ch * 4;
          const float4 v = kfreg[k];
          uint32_t l0, l1;
          const uint32_t h0 = pack_bf16x2(v.x, v.y, &l0), h1 = pack_bf16x2(v.z, v.w, &l1);
          *reinterpret_cast<uint2*>(sm + L::k + o) = make_uint2(h0, h1);
          *reinterpret_cast<uint2*>(sm + L::kl + o) = make_uint2(l0, l1);
          if constexpr (JVP) {
            // G = K_cur - K0 (zero for fixed keys, which never move)
            const uint2 b = k0reg[k];
            const float gx = v.x - __uint_as_float(b.x << 16), gy = v.y - __uint_as_float(b.x & 0xffff0000u);
            const float gz = v.z - __uint_as_float(b.y << 16), gw = v.w - __uint_as_float(b.y & 0xffff0000u);
            uint32_t gl0, gl1;
            const uint32_t gh0 = pack_bf16x2(gx, gy, &gl0), gh1 = pack_bf16x2(gz, gw, &gl1);
            *reinterpret_cast<uint2*>(sm + L::dh + o) = make_uint2(gh0, gh1);
            *reinterpret_cast<uint2*>(sm + L::dl + o) = make_uint2(gl0, gl1);
          }
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < KPT; ++k) {
        const int e = tid + k * NTH;
        if (e < KCH) {
          const int key = e / (D / 8), ch = e % (D / 8);
          *reinterpret_cast<uint4*>(sm + L::k + key * L::KS + ch * 8) = kreg[k];
        }
      }
    }
#pragma unroll
    for (int k = 0; k < VPT; ++k) {
      const int e = tid + k * NTH;
      if (e < VUN) {
        const int kp = e % 16, dq = e / 16;
        uint32_t hi[2][2], lo[2][2];   // [key kp + 16h][column pair]
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          hi[h][0] = pack_bf16x2(vreg[k][h].x, vreg[k][h].y, &lo[h][0]);
          hi[h][1] = pack_bf16x2(vreg[k][h].z, vreg[k][h].w, &lo[h][1]);
          const int ro = (kp + 16 * h) * L::KS + 4 * dq;
          *reinterpret_cast<uint2*>(sm + L::vh + ro) = make_uint2(hi[h][0], hi[h][1]);
          *reinterpret_cast<uint2*>(sm + L::vl + ro) = make_uint2(lo[h][0], lo[h][1]);
        }
        // transposed: column 4dq + c holds (key kp, key kp + 16) at 2kp
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
          const int sh = (cc & 1) * 16;
          const uint32_t th_ = ((hi[0][cc >> 1] >> sh) & 0xffffu) | (((hi[1][cc >> 1] >> sh) & 0xffffu) << 16);
          const uint32_t tl_ = ((lo[0][cc >> 1] >> sh) & 0xffffu) | (((lo[1][cc >> 1] >> sh) & 0xffffu) << 16);
          const int to = (4 * dq + cc) * L::TS + 2 * kp;
          *reinterpret_cast<uint32_t*>(sm + L::th + to) = th_;
          *reinterpret_cast<uint32_t*>(sm + L::tl + to) = tl_;
        }
      }
    }
    if (tid < kKT) {
      kp_s[tid] = kpreg;
      fx_s[tid] = (uint8_t)fxreg;
    }
  };
  // the first tile's loads go out before the per-block constants
  if (j0 < j1) load_tile(j0);

  // per-wave constants: Q rows, the direction's rows (bf16 hi/lo), s = rowdot(F, dir)
  const int row = 16 * wave + l16;
  const u16* qu = q + (size_t)u * m * D;
  uint4 qa[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks)
    qa[ks] = row < m ? *reinterpret_cast<const uint4*>(qu + (size_t)row * D + ks * 32 + 8 * g)
                     : make_uint4(0, 0, 0, 0);
  bf16x8 pah[JVP ? 1 : D / 32], pal[JVP ? 1 : D / 32];
  float sdot = 0.f;
  if constexpr (!JVP) {
    const float* pr = pv + ((size_t)u * MP + row) * D;
    const float* fr = Fm + ((size_t)u * MP + row) * D;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const float4 a0 = *reinterpret_cast<const float4*>(pr + ks * 32 + 8 * g);
      const float4 a1 = *reinterpret_cast<const float4*>(pr + ks * 32 + 8 * g + 4);
      const float x[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      if constexpr (FINAL) {
        const float4 f0 = *reinterpret_cast<const float4*>(fr + ks * 32 + 8 * g);
        const float4 f1 = *reinterpret_cast<const float4*>(fr + ks * 32 + 8 * g + 4);
        sdot += a0.x * f0.x + a0.y * f0.y + a0.z * f0.z + a0.w * f0.w;
        sdot += a1.x * f1.x + a1.y * f1.y + a1.z * f1.z + a1.w * f1.w;
      }
      split8(x, pah[ks], pal[ks]);
    }
  }
  if constexpr (FINAL) {
    sdot += __shfl_xor(sdot, 16);
    sdot += __shfl_xor(sdot, 32);
  }
  // an MFMA result gives a lane rows 16w + 4g + i
  float s4[4], nl4[4];
  int rp4[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r4 = 16 * wave + 4 * g + i;
    if constexpr (FINAL)
      s4[i] = __shfl(sdot, 4 * g + i);
    else if constexpr (!JVP)
      s4[i] = sdot_in[(size_t)u * MP + r4];
    else
      s4[i] = 0.f;
    nl4[i] = r4 < m ? -lse2[(size_t)u * MP + r4] : NEG_INF;
    rp4[i] = r4 < m ? (int)(n - w + r4 % w) : -1;
  }

  bf16x8 wah[KM == kOp ? MP / 32 : 1], wal[KM == kOp ? MP / 32 : 1];
  if constexpr (KM == kOp) {
    // W row of this lane at the columns 32kb + {4g + i, 16 + 4g + i}
    const float* wr = W + ((size_t)u * MP + row) * MP;
#pragma unroll
    for (int kb = 0; kb < MP / 32; ++kb) {
      const float4 a = *reinterpret_cast<const float4*>(wr + 32 * kb + 4 * g);
      const float4 b = *reinterpret_cast<const float4*>(wr + 32 * kb + 16 + 4 * g);
      const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
      split8(x, wah[kb], wal[kb]);
    }
  }
  if constexpr (FINAL) {
    // Q^T in LDS, rows permuted by kperm: QT[dd][kperm(r)] = Q[r][dd]
    for (int e = tid; e < MP * (D / 8); e += NTH) {
      const int r = e % MP, ch = e / MP;   // neighbouring lanes: neighbouring rows
      const uint4 v = r < m ? *reinterpret_cast<const uint4*>(qu + (size_t)r * D + ch * 8)
                            : make_uint4(0, 0, 0, 0);
      const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
      u16* dst = sm + L::qt + (ch * 8) * L::QS + kperm(r);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        dst[(2 * k) * L::QS] = (u16)(wv[k] & 0xffffu);
        dst[(2 * k + 1) * L::QS] = (u16)(wv[k] >> 16);
      }
    }
  }

  f32x4 oacc[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) oacc[dt] = zero4();
  float hs4[4] = {0.f, 0.f, 0.f, 0.f};   // row sums of H, rows 16w + 4g + i

  for (int t0 = j0; t0 < j1; t0 += kKT) {
    __syncthreads();   // the previous tile is no longer read
    store_tile();
    __syncthreads();
    if (t0 + kKT < j1) load_tile(t0 + kKT);

    // S = Q K^T (and for kOp / kFinal B = dir V^T, D = X o (B - s) -> D^T in LDS)
    float xk[kKT / 16][4];   // X[16w + 4g + i][key 16kt + l16]
#pragma unroll
    for (int kt = 0; kt < kKT / 16; ++kt) {
      const int key = 16 * kt + l16;
      f32x4 sacc = zero4(), bacc = zero4();
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        const int o = key * L::KS + ks * 32 + 8 * g;
        const bf16x8 kk = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::k + o));
        sacc = mfma_bf16(as_bf16x8(qa[ks]), kk, sacc);
        if constexpr (KF) {
          const bf16x8 kl = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::kl + o));
          sacc = mfma_bf16(as_bf16x8(qa[ks]), kl, sacc);
        }
        if constexpr (!JVP) {
          const bf16x8 vh = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::vh + o));
          const bf16x8 vl = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::vl + o));
          bacc = mfma_bf16(pah[ks], vh, bacc);
          bacc = mfma_bf16(pah[ks], vl, bacc);
          bacc = mfma_bf16(pal[ks], vh, bacc);
        }
      }
      const int kpos = kp_s[key];
      const bool live = t0 + key < j1;
      const bool free_key = live && fx_s[key] == 0;
      float dv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool vis = live && (!causal || kpos <= rp4[i]);
        const float x = vis ? __builtin_amdgcn_exp2f(fmaf(sacc[i], scale_log2, nl4[i])) : 0.f;
        xk[kt][i] = x;
        dv[i] = free_key ? x * (bacc[i] - s4[i]) : 0.f;
      }
      if constexpr (!JVP) {
        uint32_t dl0, dl1;
        const uint32_t dh0 = pack_bf16x2(dv[0], dv[1], &dl0);
        const uint32_t dh1 = pack_bf16x2(dv[2], dv[3], &dl1);
        const int dp = key * L::DS + 32 * (wave >> 1) + 8 * g + 4 * (wave & 1);
        *reinterpret_cast<uint2*>(sm + L::dh + dp) = make_uint2(dh0, dh1);
        *reinterpret_cast<uint2*>(sm + L::dl + dp) = make_uint2(dl0, dl1);
      }
    }
    if constexpr (!JVP) __syncthreads();   // D^T of all rows is in LDS

    if constexpr (FINAL) {
      // dK [keys x d] = D^T Q / sqrt(d); K* = K0 + dK (fixed keys: dK = 0)
      for (int tl = wave; tl < (kKT / 16) * (D / 16); tl += NW) {
        const int kt = tl / (D / 16), dt = tl % (D / 16);
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < MP / 32; ++kb) {
          const int ao = (16 * kt + l16) * L::DS + 32 * kb + 8 * g;
          const bf16x8 ah = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::dh + ao));
          const bf16x8 al = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::dl + ao));
          const bf16x8 b = as_bf16x8(*reinterpret_cast<const uint4*>(
              sm + L::qt + (16 * dt + l16) * L::QS + 32 * kb + 8 * g));
          acc = mfma_bf16(ah, b, acc);
          acc = mfma_bf16(al, b, acc);
        }
        const int dd = 16 * dt + l16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = 16 * kt + 4 * g + i;
          if (t0 + key < j1) {
            const size_t o = ((size_t)u * c + t0 + key) * D + dd;
            const float base = KF ? bf16_to_f32(k0[o]) : bf16_to_f32(sm[L::k + key * L::KS + dd]);
            kstar[o] = base + acc[i] * inv_sqrt_d;
          }
        }
      }
    } else {
      // A = W D (kOp) or A = Q G^T / sqrt(d) (kJvp) for this wave's rows, and
      // H = X o A: lane holds [row 16w + 4g + i][key]
      const int hb = wave * 16 * L::HS;
      float hv[kKT / 16][4];
#pragma unroll
      for (int kt = 0; kt < kKT / 16; ++kt) {
        f32x4 aacc = zero4();
        if constexpr (JVP) {
#pragma unroll
          for (int ks = 0; ks < D / 32; ++ks) {
            const int o = (16 * kt + l16) * L::KS + ks * 32 + 8 * g;
            const bf16x8 gh = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::dh + o));
            const bf16x8 gl = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::dl + o));
            aacc = mfma_bf16(as_bf16x8(qa[ks]), gh, aacc);
            aacc = mfma_bf16(as_bf16x8(qa[ks]), gl, aacc);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) aacc[i] *= inv_sqrt_d;
        } else {
#pragma unroll
          for (int kb = 0; kb < MP / 32; ++kb) {
            const int ao = (16 * kt + l16) * L::DS + 32 * kb + 8 * g;
            const bf16x8 dh = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::dh + ao));
            const bf16x8 dl = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::dl + ao));
            aacc = mfma_bf16(wah[kb], dh, aacc);
            aacc = mfma_bf16(wal[kb], dh, aacc);
            aacc = mfma_bf16(wah[kb], dl, aacc);
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          hv[kt][i] = xk[kt][i] * aacc[i];
          hs4[i] += hv[kt][i];
        }
      }
      // the lane's keys l16 and 16 + l16 are adjacent in the H rows
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t lo;
        const uint32_t hi = pack_bf16x2(hv[0][i], hv[1][i], &lo);
        const int o = hb + (4 * g + i) * L::HS + 2 * l16;
        *reinterpret_cast<uint32_t*>(sm + L::hh + o) = hi;
        *reinterpret_cast<uint32_t*>(sm + L::hl + o) = lo;
      }
      // out^T [d x rows] += V*^T H^T over the tile's 32 keys (the H rows were
      // written by this wave alone, and its LDS accesses complete in order)
      const int ho = hb + l16 * L::HS + 8 * g;
      const bf16x8 hh = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::hh + ho));
      const bf16x8 hl = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::hl + ho));
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const int vo = (16 * dt + l16) * L::TS + 8 * g;
        const bf16x8 th = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::th + vo));
        const bf16x8 tl = as_bf16x8(*reinterpret_cast<const uint4*>(sm + L::tl + vo));
        oacc[dt] = mfma_bf16(th, hh, oacc[dt]);
        oacc[dt] = mfma_bf16(th, hl, oacc[dt]);
        oacc[dt] = mfma_bf16(tl, hh, oacc[dt]);
      }
    }
  }

  if constexpr (!FINAL) {
    // lane holds out[row][16dt + 4g + i]
    float* op = opart + (((size_t)u * S + s) * MP + row) * D;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
      *reinterpret_cast<float4*>(op + 16 * dt + 4 * g) =
          make_float4(oacc[dt][0], oacc[dt][1], oacc[dt][2], oacc[dt][3]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float h = sum16(hs4[i]);
      if (l16 == 0) hpart[((size_t)u * S + s) * MP + 16 * wave + 4 * g + i] = h;
    }
  }
}

// Right-hand side at a later alternating step: r = E + J_G G from the kJvp
// partials (J_G G = sum_s opart - (sum_s hpart) o F), then p = r, alpha = 0
// and the CG state.  key_init has already set F, E (in r) and the skip state.
template <int MP, int D>
__global__ __launch_bounds__(1024) void key_rhs_kernel(
    const float* __restrict__ opart, const float* __restrict__ hpart, int S,
    const float* __restrict__ Fm, float* __restrict__ r, float* __restrict__ p,
    float* __restrict__ sdot, double* __restrict__ cg) {
  constexpr int NTH = 1024, E4 = MP * D / 4, PER = (E4 + NTH - 1) / NTH, RW = D / 4;
  __shared__ float hsum[MP];
  __shared__ double red[16];
  const int u = blockIdx.x, tid = threadIdx.x;
  if ((int)cg[u * 4 + 3] == kKeySkipped) return;
  // split partials in batches of kCgBatch (clamped, summed in split order),
  // as in key_cg
  for (int i = tid; i < MP; i += NTH) {
    float h = 0.f;
    for (int k0 = 0; k0 < S; k0 += kCgBatch) {
      float hv[kCgBatch];
#pragma unroll
      for (int j = 0; j < kCgBatch; ++j) hv[j] = hpart[((size_t)u * S + min(k0 + j, S - 1)) * MP + i];
#pragma unroll
      for (int j = 0; j < kCgBatch; ++j)
        if (k0 + j < S) h += hv[j];
    }
    hsum[i] = h;
  }
  __syncthreads();
  const size_t base = (size_t)u * E4;
  const float4* __restrict__ op4 = reinterpret_cast<const float4*>(opart) + (size_t)u * S * E4;
  const float4* __restrict__ F4 = reinterpret_cast<const float4*>(Fm) + base;
  float4* __restrict__ r4 = reinterpret_cast<float4*>(r) + base;
  float4* __restrict__ p4 = reinterpret_cast<float4*>(p) + base;
  float4 rs[PER];   // r + the partials, in split order
#pragma unroll
  for (int k = 0; k < PER; ++k) rs[k] = r4[min(tid + k * NTH, E4 - 1)];
  for (int s0 = 0; s0 < S; s0 += kCgBatch) {
    float4 ov[kCgBatch][PER];
#pragma unroll
    for (int j = 0; j < kCgBatch; ++j)
#pragma unroll
      for (int k = 0; k < PER; ++k)
        ov[j][k] = op4[(size_t)min(s0 + j, S - 1) * E4 + min(tid + k * NTH, E4 - 1)];
#pragma unroll
    for (int j = 0; j < kCgBatch; ++j)
      if (s0 + j < S)
#pragma unroll
        for (int k = 0; k < PER; ++k) {
          rs[k].x += ov[j][k].x; rs[k].y += ov[j][k].y;
          rs[k].z += ov[j][k].z; rs[k].w += ov[j][k].w;
        }
  }
  double rr = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = tid + k * NTH;
    float4 re = make_float4(0.f, 0.f, 0.f, 0.f), f = re;
    if (e < E4) {
      const float4 v = rs[k];
      f = F4[e];
      const float h = hsum[e / RW];
      re = make_float4(v.x - h * f.x, v.y - h * f.y, v.z - h * f.z, v.w - h * f.w);
      r4[e] = re;
      p4[e] = re;
      rr += (double)dot4(re, re);
    }
    // row dot over the RW consecutive threads of a row (whole rows only)
    float sd = dot4(f, re);
#pragma unroll
    for (int off = 1; off < RW; off <<= 1) sd += __shfl_xor(sd, off);
    if (e < E4 && (e % RW) == 0) sdot[(size_t)u * MP + e / RW] = sd;
  }
  rr = block_sum(rr, red);
  if (tid == 0) {
    cg[u * 4 + 0] = rr;
    cg[u * 4 + 1] = rr;
    cg[u * 4 + 2] = 0;
    cg[u * 4 + 3] = rr == 0 ? kKeyConverged : kKeyRunning;
  }
}

// -------------------------------------------------------------------- cg ----
// One conjugate-gradient update per unit: Ap = sum_s opart - (sum_s hpart) o F
// + lambda_k p; alpha += a p; r -= a Ap; p = r + beta p; and the row dots
// s = rowdot(F, p) of the new direction for the next operator pass.

template <int MP, int D>
__global__ __launch_bounds__(1024) void key_cg_kernel(
    const float* __restrict__ opart, const float* __restrict__ hpart, int S,
    const float* __restrict__ Fm, float* __restrict__ alpha, float* __restrict__ r,
    float* __restrict__ p, float* __restrict__ sdot, double* __restrict__ cg, float lam_k,
    float tol, int max_iter) {
  constexpr int NTH = 1024, E4 = MP * D / 4, PER = (E4 + NTH - 1) / NTH, RW = D / 4;
  __shared__ float hsum[MP];
  __shared__ double red[16];
  const int u = blockIdx.x, tid = threadIdx.x;
  if ((int)cg[u * 4 + 3] != kKeyRunning) return;
  // the split partials are loaded kCgBatch splits at a time (indices past S
  // read split S - 1, in bounds, and are not summed) and summed in split
  // order: the loads of a batch are in flight together
  for (int i = tid; i < MP; i += NTH) {
    float h = 0.f;
    for (int k0 = 0; k0 < S; k0 += kCgBatch) {
      float hv[kCgBatch];
#pragma unroll
      for (int j = 0; j < kCgBatch; ++j) hv[j] = hpart[((size_t)u * S + min(k0 + j, S - 1)) * MP + i];
#pragma unroll
      for (int j = 0; j < kCgBatch; ++j)
        if (k0 + j < S) h += hv[j];
    }
    hsum[i] = h;
  }
  __syncthreads();
  const size_t base = (size_t)u * E4;
  const float4* __restrict__ op4 = reinterpret_cast<const float4*>(opart) + (size_t)u * S * E4;
  const float4* __restrict__ F4 = reinterpret_cast<const float4*>(Fm) + base;
  float4* __restrict__ a4 = reinterpret_cast<float4*>(alpha) + base;
  float4* __restrict__ r4 = reinterpret_cast<float4*>(r) + base;
  float4* __restrict__ p4 = reinterpret_cast<float4*>(p) + base;
  const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
  float4 osum[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) osum[k] = z4;
  for (int s0 = 0; s0 < S; s0 += kCgBatch) {
    float4 ov[kCgBatch][PER];
#pragma unroll
    for (int j = 0; j < kCgBatch; ++j)
#pragma unroll
      for (int k = 0; k < PER; ++k)
        ov[j][k] = op4[(size_t)min(s0 + j, S - 1) * E4 + min(tid + k * NTH, E4 - 1)];
#pragma unroll
    for (int j = 0; j < kCgBatch; ++j)
      if (s0 + j < S)
#pragma unroll
        for (int k = 0; k < PER; ++k) {
          osum[k].x += ov[j][k].x; osum[k].y += ov[j][k].y;
          osum[k].z += ov[j][k].z; osum[k].w += ov[j][k].w;
        }
  }
  float4 ap[PER], pp[PER], fv[PER];
  double pap = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = tid + k * NTH;
    ap[k] = pp[k] = fv[k] = z4;
    if (e < E4) {
      float4 v = osum[k];
      const float4 pe = p4[e], f = F4[e];
      const float h = hsum[e / RW];
      v.x += lam_k * pe.x - h * f.x;
      v.y += lam_k * pe.y - h * f.y;
      v.z += lam_k * pe.z - h * f.z;
      v.w += lam_k * pe.w - h * f.w;
      ap[k] = v;
      pp[k] = pe;
      fv[k] = f;
      pap += (double)dot4(pe, v);
    }
  }
  pap = block_sum(pap, red);
  const double rr = cg[u * 4 + 0], rr0 = cg[u * 4 + 1];
  const int it = (int)cg[u * 4 + 2] + 1;
  if (!(pap > 0)) {
    if (tid == 0) cg[u * 4 + 3] = kKeyBreakdown;
    return;
  }
  const float a = (float)(rr / pap);
  float4 rv[PER];
  double rn = 0;
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = tid + k * NTH;
    rv[k] = z4;
    if (e < E4) {
      float4 al = a4[e], re = r4[e];
      al.x += a * pp[k].x; al.y += a * pp[k].y; al.z += a * pp[k].z; al.w += a * pp[k].w;
      re.x -= a * ap[k].x; re.y -= a * ap[k].y; re.z -= a * ap[k].z; re.w -= a * ap[k].w;
      a4[e] = al;
      r4[e] = re;
      rv[k] = re;
      rn += (double)dot4(re, re);
    }
  }
  rn = block_sum(rn, red);
  int st = kKeyRunning;
  if (sqrt(rn) <= (double)tol * sqrt(rr0)) st = kKeyConverged;
  else if (it >= max_iter) st = kKeyMaxIter;
  if (st == kKeyRunning) {
    const float beta = (float)(rn / rr);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = tid + k * NTH;
      float4 pn = z4;
      if (e < E4) {
        pn = make_float4(rv[k].x + beta * pp[k].x, rv[k].y + beta * pp[k].y,
                         rv[k].z + beta * pp[k].z, rv[k].w + beta * pp[k].w);
        p4[e] = pn;
      }
      // row dot over the RW consecutive threads of a row (whole rows only)
      float sd = dot4(fv[k], pn);
#pragma unroll
      for (int off = 1; off < RW; off <<= 1) sd += __shfl_xor(sd, off);
      if (e < E4 && (e % RW) == 0) sdot[(size_t)u * MP + e / RW] = sd;
    }
  }
  if (tid == 0) {
    cg[u * 4 + 0] = rn;
    cg[u * 4 + 2] = it;
    cg[u * 4 + 3] = st;
  }
}

template <int MP, int D, int KM, bool KF>
hipError_t launch_pass(const Plan& p, const KeyArgs& a, int S, int chunk, const float* dir,
                       hipStream_t s) {
  using L = KeyLds<MP, D, KM, KF>;
  const size_t lds = L::bytes();
  hipError_t e = hipFuncSetAttribute((const void*)key_pass_kernel<MP, D, KM, KF>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
  const float inv_sqrt_d = (float)(1.0 / sqrt((double)D));
  hipLaunchKernelGGL((key_pass_kernel<MP, D, KM, KF>), dim3(S, p.U), dim3(MP / 16 * 64), lds, s,
                     a.q, a.k0, a.kcur, a.vs, a.lse2, a.fixed, a.idx, a.Fm, a.W, dir, a.sdot,
                     a.cg, a.opart, a.hpart, a.kstar, a.cg_info, p.m, p.w, p.n, p.c, S, chunk,
                     p.opt.causal_window ? 1 : 0, scale_log2, inv_sqrt_d);
  return hipGetLastError();
}

template <int MP, int D, bool KF>
hipError_t launch_key_t(const Plan& p, const KeyPlan& kp, const KeyArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((key_init_kernel<MP, D>), dim3(p.U), dim3(256), 0, s, a.q, a.y, a.zt,
                     a.stats_ws, p.lam, p.m, a.Fm, a.alpha, a.r, a.p, a.sdot, a.W, a.cg);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (!KF && a.vh) {
    // the ring kernel's passes (key_ring.hip) on V* split once into hi/lo
    e = launch_key_prep(p, a, s);
    if (e != hipSuccess) return e;
    for (int it = 0; it < a.max_iter; ++it) {
      const bool early = it < kKeyRingEarlyIters;
      const int S = early ? kp.S_full : kp.S4r, chunk = early ? kp.chunk_full : kp.chunk4r;
      // one split per unit: the CG update runs inside the pass
      const bool fuse = S == 1;
      e = launch_key_ring(p, a, false, S, chunk, a.p, fuse, s);
      if (e != hipSuccess) return e;
      if (!fuse) {
        hipLaunchKernelGGL((key_cg_kernel<MP, D>), dim3(p.U), dim3(1024), 0, s, a.opart,
                           a.hpart, S, a.Fm, a.alpha, a.r, a.p, a.sdot, a.cg, a.lam_k, a.tol,
                           a.max_iter);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
      }
    }
    return launch_key_ring(p, a, true, kp.S_full, kp.chunk_full, a.alpha, false, s);
  }
  if constexpr (KF) {
    // a later alternating step: the right-hand side gains J_G (K_cur - K0)
    e = launch_pass<MP, D, kJvp, KF>(p, a, kp.S_full, kp.chunk_full, nullptr, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((key_rhs_kernel<MP, D>), dim3(p.U), dim3(1024), 0, s, a.opart, a.hpart,
                       kp.S_full, a.Fm, a.r, a.p, a.sdot, a.cg);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  for (int it = 0; it < a.max_iter; ++it) {
    // the first iterations, while every unit is still running, with the
    // fewest blocks a full GPU needs; later ones with more splits per unit,
    // which shortens an iteration once few units remain
    const bool early = it < kKeyEarlyIters;
    const int S = early ? kp.S_full : kp.S4, chunk = early ? kp.chunk_full : kp.chunk4;
    e = launch_pass<MP, D, kOp, KF>(p, a, S, chunk, a.p, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((key_cg_kernel<MP, D>), dim3(p.U), dim3(1024), 0, s, a.opart, a.hpart,
                       S, a.Fm, a.alpha, a.r, a.p, a.sdot, a.cg, a.lam_k, a.tol, a.max_iter);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return launch_pass<MP, D, kFinal, KF>(p, a, kp.S_full, kp.chunk_full, a.alpha, s);
}

template <int MP, int D>
hipError_t launch_key_kf(const Plan& p, const KeyPlan& kp, const KeyArgs& a, hipStream_t s) {
  return a.kcur ? launch_key_t<MP, D, true>(p, kp, a, s) : launch_key_t<MP, D, false>(p, kp, a, s);
}

__global__ void to_f32_kernel(const u16* __restrict__ src, float* __restrict__ dst, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    dst[i] = bf16_to_f32(src[i]);
}

}  // namespace

hipError_t launch_to_f32(const uint16_t* src, float* dst, size_t n, hipStream_t s) {
  const size_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(to_f32_kernel, dim3((unsigned)(blocks < 65535 ? blocks : 65535)), dim3(256),
                     0, s, src, dst, n);
  return hipGetLastError();
}

bool key_supported(const Plan& p) {
  return stream_supported(p) && merge_fast_supported(p) && p.mp <= 128 &&
         (p.d == 64 || p.d == 128);
}

hipError_t launch_key(const Plan& p, const KeyPlan& kp, const KeyArgs& a, hipStream_t s) {
  if (p.d == 128) {
    switch (p.mp) {
      case 32: return launch_key_kf<32, 128>(p, kp, a, s);
      case 64: return launch_key_kf<64, 128>(p, kp, a, s);
      case 128: return launch_key_kf<128, 128>(p, kp, a, s);
    }
  } else {
    switch (p.mp) {
      case 32: return launch_key_kf<32, 64>(p, kp, a, s);
      case 64: return launch_key_kf<64, 64>(p, kp, a, s);
      case 128: return launch_key_kf<128, 64>(p, kp, a, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace grkv
