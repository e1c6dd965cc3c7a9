// Value step, recomputed for the units whose retained attention mass the
// fast retained pass cannot resolve (Eq. 8; Algorithm 1, value step; App. D.1,
// fixed tokens App. D.3).
//
// The fast retained pass forms P = 2^(t - LSE_full + bias) against the
// full-cache log-sum-exp, and the solve normalises by the retained row mass.
// When every retained key of some window row lies far below the row's best
// evicted key (retained mass under 2^-108 of the full-cache mass), those P
// values underflow, and the solve marks the unit GRKV_UNIT_RANGE.  This kernel
// then runs the whole value step of such a unit once more, against the
// retained set's own row maximum instead of the full-cache log-sum-exp:
//   M_r   = max over the retained keys row r sees of t_rj (log2 domain),
//   P'_rj = 2^(t_rj - M_r)          (the largest entry of a row is exactly 1),
//   mu_r  = sum_j P'_rj,  X = diag(1/mu) P',  retained LSE = M + log2(mu),
//   N = X_G X_G^T + lambda I,  R = Y - X V0,  N = L L^T,  Z = N^-1 R,
// and writes Z^T (fp32 and bf16 hi/lo), the retained LSE, R, N and the stats
// exactly where the solve writes them, so the update kernel that follows
// forms V* = V0 + X_G^T Z as for every other unit.
//
// Run by the solve kernel's first block of a marked unit, after that block's
// own solve (the other blocks of the unit return early), so a call without
// marked units pays nothing for it.  One block of 1024 threads; the LDS
// scratch (FixLds<MP, D>::floats) is the solve's own, reused.  The
// arithmetic is plain fp32 on the vector ALUs (products of bf16 inputs are
// exact in fp32), the Cholesky factorisation a right-looking column sweep in
// LDS: this path trades speed for range.
#pragma once

#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {

constexpr int kFixThreads = 1024;
constexpr int kFixChunk = 32;   // retained keys per step

template <int MP, int D>
struct FixLds {
  static constexpr int TPR = kFixThreads / MP;     // threads per window row
  static constexpr int JPT = kFixChunk / TPR;      // keys of a step per thread
  static constexpr int QS = D + 1;                 // padded row strides (floats)
  static constexpr int KS = D + 1;
  static constexpr int PS = kFixChunk + 1;
  static constexpr int AS = MP + 1;
  static constexpr int BS = D + 1;
  // streaming steps: Q, a step's K0 and V0 rows and its probabilities
  static constexpr size_t q_off = 0;
  static constexpr size_t k_off = q_off + (size_t)MP * QS;
  static constexpr size_t v_off = k_off + (size_t)kFixChunk * KS;
  static constexpr size_t p_off = v_off + (size_t)kFixChunk * KS;
  static constexpr size_t stream_floats = p_off + (size_t)MP * PS;
  // factorisation: N (lower triangle) and the right-hand sides
  static constexpr size_t a_off = 0;
  static constexpr size_t b_off = a_off + (size_t)MP * AS;
  static constexpr size_t solve_floats = b_off + (size_t)MP * BS;
  static constexpr size_t floats = stream_floats > solve_floats ? stream_floats : solve_floats;
  static constexpr size_t bytes = floats * sizeof(float);
};

// The value step of unit u (GRKV_UNIT_RANGE) against the retained row maxima,
// by the whole calling block (kFixThreads threads); fsm: FixLds<MP, D>::floats
// of LDS that no other code of the block uses meanwhile.
template <int MP, int D>
__device__ __forceinline__ void range_fix_unit(
    float* fsm, int u, const u16* q, const u16* k0, const u16* V, const int32_t* idx,
    const uint8_t* fixed, const float* y, int64_t n, int m, int w, int c, int causal,
    float scale_log2, float lam, float* lse2_log2, float* resid, float* gram, float* z, u16* zhi,
    u16* zlo, float* stats_ws, float* stats_user, const RagUnit* rag, int csplit, double* zpart) {
  using L = FixLds<MP, D>;
  constexpr int TPR = L::TPR, JPT = L::JPT;
  constexpr int NXV = D / TPR;    // columns of X V0 per thread
  constexpr int NN = MP / TPR;    // columns of N per thread
  static_assert(kFixThreads % MP == 0 && kFixChunk % TPR == 0, "thread mapping");
  static_assert(D % TPR == 0 && MP % TPR == 0, "thread mapping");
  __shared__ float rowmax[MP], rowinv[MP];
  __shared__ int32_t kpos[kFixChunk];
  __shared__ float kfree[kFixChunk];
  __shared__ double red[3][kFixThreads / 64];
  __shared__ int fail;

  const int tid = threadIdx.x;
  size_t slot0 = (size_t)u * c;
  if (rag) {
    slot0 = (size_t)rag[u].off;
    c = rag[u].c;
  }
  const int r = tid / TPR, sub = tid % TPR;   // window row and its sub-thread
  const bool live = r < m;
  const int64_t pos_r = n - w + (live ? r % w : 0);
  float* qs = fsm + L::q_off;
  float* ks = fsm + L::k_off;
  float* vs = fsm + L::v_off;
  float* ps = fsm + L::p_off;

  const u16* qu = q + (size_t)u * m * D;
  for (int e = tid; e < MP * D; e += kFixThreads) {
    const int rr = e / D, cc = e % D;
    qs[rr * L::QS + cc] = rr < m ? bf16_to_f32(qu[(size_t)rr * D + cc]) : 0.f;
  }
  if (tid == 0) fail = 0;

  // stage the K0 rows (and, with V, the V0 rows) of retained slots t0 .. t0+31
  auto stage = [&](int t0, bool with_v) {
    for (int e = tid; e < kFixChunk * D; e += kFixThreads) {
      const int jj = e / D, cc = e % D, t = t0 + jj;
      float kv = 0.f, vv = 0.f;
      if (t < c) {
        kv = bf16_to_f32(k0[(slot0 + t) * D + cc]);
        if (with_v) {
          const int64_t src = idx[slot0 + t];
          vv = bf16_to_f32(V[((size_t)u * n + src) * D + cc]);
        }
      }
      ks[jj * L::KS + cc] = kv;
      if (with_v) vs[jj * L::KS + cc] = vv;
    }
    if (tid < kFixChunk) {
      const int t = t0 + tid;
      kpos[tid] = t < c ? idx[slot0 + t] : 0;
      kfree[tid] = (t < c && !fixed[slot0 + t]) ? 1.f : 0.f;
    }
  };
  // log2-domain logit of row r and staged key jj, or -inf when row r does not
  // see that key (causal rule, past the retained set, padding row)
  auto logit = [&](int jj, int t0) {
    constexpr float NEG_INF = -__builtin_huge_valf();
    if (!live || t0 + jj >= c || (causal && (int64_t)kpos[jj] > pos_r)) return NEG_INF;
    float acc = 0.f;
#pragma unroll 8
    for (int e = 0; e < D; ++e) acc = fmaf(qs[r * L::QS + e], ks[jj * L::KS + e], acc);
    return acc * scale_log2;
  };

  // 1. row maxima of the retained logits
  float mx = -__builtin_huge_valf();
  for (int t0 = 0; t0 < c; t0 += kFixChunk) {
    __syncthreads();
    stage(t0, false);
    __syncthreads();
#pragma unroll
    for (int k = 0; k < JPT; ++k) mx = fmaxf(mx, logit(sub + TPR * k, t0));
  }
#pragma unroll
  for (int off = TPR / 2; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  if (sub == 0) rowmax[r] = live ? mx : 0.f;
  __syncthreads();

  // 2. P' = 2^(t - M), its row sums, X V0 and the Gram sums of the free columns
  const float mr = rowmax[r];
  float mass = 0.f;
  float xv[NXV], nn[NN];
#pragma unroll
  for (int k = 0; k < NXV; ++k) xv[k] = 0.f;
#pragma unroll
  for (int k = 0; k < NN; ++k) nn[k] = 0.f;
  for (int t0 = 0; t0 < c; t0 += kFixChunk) {
    __syncthreads();
    stage(t0, true);
    __syncthreads();
#pragma unroll
    for (int k = 0; k < JPT; ++k) {
      const int jj = sub + TPR * k;
      const float t = logit(jj, t0);
      const float p = t == -__builtin_huge_valf() ? 0.f : exp2f(t - mr);
      ps[r * L::PS + jj] = p;
      mass += p;
    }
    __syncthreads();
    for (int jj = 0; jj < kFixChunk; ++jj) {
      const float pr = ps[r * L::PS + jj];
      const float pg = pr * kfree[jj];
#pragma unroll
      for (int k = 0; k < NXV; ++k) xv[k] = fmaf(pr, vs[jj * L::KS + sub * NXV + k], xv[k]);
#pragma unroll
      for (int k = 0; k < NN; ++k) nn[k] = fmaf(pg, ps[(sub * NN + k) * L::PS + jj], nn[k]);
    }
  }
#pragma unroll
  for (int off = TPR / 2; off > 0; off >>= 1) mass += __shfl_xor(mass, off);
  if (sub == 0) {
    rowinv[r] = live ? 1.f / mass : 0.f;   // mass >= 1: the row's largest term is 2^0
    if (live) lse2_log2[(size_t)u * MP + r] = mr + __log2f(mass);
  }
  __syncthreads();

  // 3. N = D P'_G P'_G^T D + lambda I and R = Y - D P' V0 (padding rows and
  // columns of N are identity, padding rows of R zero)
  float* A = fsm + L::a_off;
  float* B = fsm + L::b_off;
  double sy = 0.0, sr = 0.0, sz = 0.0;
  {
    const float ir = rowinv[r];
    float* gu = gram + (size_t)u * MP * MP;
#pragma unroll
    for (int k = 0; k < NN; ++k) {
      const int s = sub * NN + k;
      float v = (live && s < m) ? ir * rowinv[s] * nn[k] : 0.f;
      if (r == s) v += live ? lam : 1.f;
      A[r * L::AS + s] = v;
      gu[(size_t)r * MP + s] = v;
    }
    const float* yu = y + (size_t)u * MP * D;
    float* ru = resid + (size_t)u * MP * D;
#pragma unroll
    for (int k = 0; k < NXV; ++k) {
      const int dd = sub * NXV + k;
      const float yv = live ? yu[(size_t)r * D + dd] : 0.f;
      const float rv = live ? yv - ir * xv[k] : 0.f;
      B[r * L::BS + dd] = rv;
      ru[(size_t)r * D + dd] = rv;
      sy += (double)yv * yv;
      sr += (double)rv * rv;
    }
  }
  __syncthreads();

  // 4. N = L L^T, column by column
  for (int k = 0; k < MP; ++k) {
    if (tid == 0) {
      const float dk = A[k * L::AS + k];
      if (!(dk > 0.f && dk < __builtin_huge_valf())) fail = 1;
      A[k * L::AS + k] = sqrtf(dk);
    }
    __syncthreads();
    if (fail) break;   // read after the barrier: block-uniform
    const float lkk = A[k * L::AS + k];
    for (int i = k + 1 + tid; i < MP; i += kFixThreads) A[i * L::AS + k] /= lkk;
    __syncthreads();
    const int T = MP - k - 1;
    for (int e = tid; e < T * T; e += kFixThreads) {
      const int i = k + 1 + e / T, j = k + 1 + e % T;
      if (j <= i) A[i * L::AS + j] = fmaf(-A[i * L::AS + k], A[j * L::AS + k], A[i * L::AS + j]);
    }
    __syncthreads();
  }
  const bool ok = fail == 0;

  // 5. forward and backward substitution, one right-hand-side column per thread
  if (ok && tid < D) {
    const int dd = tid;
    for (int i = 0; i < MP; ++i) {
      float s = B[i * L::BS + dd];
      for (int k = 0; k < i; ++k) s = fmaf(-A[i * L::AS + k], B[k * L::BS + dd], s);
      B[i * L::BS + dd] = s / A[i * L::AS + i];
    }
    for (int i = MP - 1; i >= 0; --i) {
      float s = B[i * L::BS + dd];
      for (int k = i + 1; k < MP; ++k) s = fmaf(-A[k * L::AS + i], B[k * L::BS + dd], s);
      B[i * L::BS + dd] = s / A[i * L::AS + i];
    }
  }
  __syncthreads();

  // 6. Z^T out (zero for a singular system), fp32 and as a bf16 hi/lo pair
  for (int e = tid; e < D * MP; e += kFixThreads) {
    const int dd = e / MP, rr = e % MP;
    const float zv = ok && rr < m ? B[rr * L::BS + dd] : 0.f;
    const size_t o = ((size_t)u * D + dd) * MP + rr;
    z[o] = zv;
    const __bf16 h = (__bf16)zv;
    zhi[o] = __builtin_bit_cast(u16, h);
    zlo[o] = __builtin_bit_cast(u16, (__bf16)(zv - (float)h));
    sz += (double)zv * zv;
  }
  const int lane = tid & 63, wave = tid >> 6;
  for (int off = 32; off > 0; off >>= 1) {
    sy += __shfl_xor(sy, off);
    sr += __shfl_xor(sr, off);
    sz += __shfl_xor(sz, off);
  }
  if (lane == 0) { red[0][wave] = sy; red[1][wave] = sr; red[2][wave] = sz; }
  __syncthreads();
  if (tid == 0) {
    double Y2 = 0, R2 = 0, Z2 = 0;
    for (int k = 0; k < kFixThreads / 64; ++k) { Y2 += red[0][k]; R2 += red[1][k]; Z2 += red[2][k]; }
    const double dn = Y2 > 0 ? Y2 : 1.0;
    const double dbefore = R2 / dn;
    const double dafter = ok ? (double)lam * lam * Z2 / dn : dbefore;
    const float st[4] = {(float)Y2, (float)dbefore, (float)dafter,
                         ok ? (float)GRKV_UNIT_OK : (float)GRKV_UNIT_SINGULAR};
    for (int k = 0; k < 4; ++k) {
      stats_ws[u * 4 + k] = st[k];
      if (stats_user) stats_user[u * 4 + k] = st[k];
    }
    // the update forms D after again from the solve blocks' shares of ||Z||^2
    if (csplit > 1) {
      for (int k = 0; k < csplit; ++k) zpart[(size_t)u * kZParts + k] = k == 0 ? Z2 : 0.0;
      zpart[(size_t)u * kZParts + kZParts - 1] = Y2;
    }
  }
}

}  // namespace grkv
