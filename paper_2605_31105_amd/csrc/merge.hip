// Value step of the ridge merge in its Woodbury dual form (Eq. 8; Algorithm 1,
// value step; App. D.1, fixed tokens App. D.3):
//   N = X_G X_G^T + lambda I_m   (gram: partial sums over column splits)
//   Z = N^-1 R                   (solve: blocked Cholesky on fp32 MFMA)
//   V*_G = V0_G + X_G^T Z        (update: fixed columns keep V0)
// On this fast path the Gram partials come from the retained-cache pass
// (stream.hip); the gram kernel here serves the generic path.
// X_G is X with the fixed columns zeroed.  The fp32 operands of the two
// products go through the bf16 MFMA as hi+lo pairs (three products per tile),
// which keeps about 16 significant bits per term; accumulation is fp32.
#include <type_traits>

#include "grkv_device.h"
#include "grkv_internal.h"
#include "range_fix.h"

namespace grkv {
namespace {

// ------------------------------------------------------------------ gram ----
// One block per (unit, column split).  Each 32-column slab of X_G (all mp rows)
// is loaded with 16-byte loads, masked, split into bf16 hi/lo and staged in LDS
// as [mp][32] (+8 pad) rows; every wave then forms its 32 rows of N against
// all mp rows.  The next slab's loads are in flight during the MFMAs.
template <int WAVES>
__global__ __launch_bounds__(WAVES * 64) void gram_kernel(const float* x, const uint8_t* fixed,
                                                          float* npart, int c, int S3, int chunk3) {
  constexpr int MP = WAVES * 32;
  constexpr int NT = MP / 16;              // 16-row tiles of N
  constexpr int RS = 40;                   // LDS row stride in bf16 (32 + 8 pad)
  constexpr int NTH = WAVES * 64;
  constexpr int F4 = MP * 32 / 4 / NTH;    // float4 loads per thread per slab
  __shared__ __attribute__((aligned(16))) u16 hi[MP * RS];
  __shared__ __attribute__((aligned(16))) u16 lo[MP * RS];

  const int s = blockIdx.x, u = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g = lane >> 4;
  const int t0 = s * chunk3, t1 = min(t0 + chunk3, c);
  const float* xu = x + (size_t)u * MP * c;
  const uint8_t* fu = fixed + (size_t)u * c;
  const bool vec = (c & 3) == 0;

  f32x4 acc[2][NT];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int bt = 0; bt < NT; ++bt) acc[rt][bt] = zero4();

  float4 rg[F4];
  uint32_t fg[F4];   // the fixed flags of rg's four slots, one per byte
  auto load = [&](int tk) {
#pragma unroll
    for (int i = 0; i < F4; ++i) {
      const int e = (tid + i * NTH) * 4;       // element in the [MP][32] slab
      const int r = e / 32, cc = e % 32, t = tk + cc;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      const float* src = xu + (size_t)r * c + t;
      if (vec && t + 3 < t1) {
        v = *reinterpret_cast<const float4*>(src);
      } else {
        float tmp[4] = {0.f, 0.f, 0.f, 0.f};
        for (int q = 0; q < 4; ++q)
          if (t + q < t1) tmp[q] = src[q];
        v = make_float4(tmp[0], tmp[1], tmp[2], tmp[3]);
      }
      rg[i] = v;
      // flags of slots past t1 read slot c - 1 (in bounds; those slots are
      // masked by t1): loads without branches, in flight with the slab's
      uint32_t f = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) f |= (uint32_t)fu[min(t + q, c - 1)] << (8 * q);
      fg[i] = f;
    }
  };
  if (t0 < t1) load(t0);
  for (int tk = t0; tk < t1; tk += 32) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < F4; ++i) {
      const int e = (tid + i * NTH) * 4;
      const int r = e / 32, cc = e % 32, t = tk + cc;
      float v[4] = {rg[i].x, rg[i].y, rg[i].z, rg[i].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float xv = (t + q < t1 && ((fg[i] >> (8 * q)) & 0xffu) == 0) ? v[q] : 0.f;
        const __bf16 h = (__bf16)xv;
        const __bf16 l = (__bf16)(xv - (float)h);
        hi[r * RS + cc + q] = __builtin_bit_cast(u16, h);
        lo[r * RS + cc + q] = __builtin_bit_cast(u16, l);
      }
    }
    __syncthreads();
    if (tk + 32 < t1) load(tk + 32);
    bf16x8 ah[2], al[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const int r = wave * 32 + rt * 16 + l16;
      ah[rt] = as_bf16x8(*reinterpret_cast<const uint4*>(&hi[r * RS + 8 * g]));
      al[rt] = as_bf16x8(*reinterpret_cast<const uint4*>(&lo[r * RS + 8 * g]));
    }
#pragma unroll
    for (int bt = 0; bt < NT; ++bt) {
      const int r = bt * 16 + l16;
      const bf16x8 bh = as_bf16x8(*reinterpret_cast<const uint4*>(&hi[r * RS + 8 * g]));
      const bf16x8 bl = as_bf16x8(*reinterpret_cast<const uint4*>(&lo[r * RS + 8 * g]));
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        acc[rt][bt] = mfma_bf16(ah[rt], bh, acc[rt][bt]);
        acc[rt][bt] = mfma_bf16(ah[rt], bl, acc[rt][bt]);
        acc[rt][bt] = mfma_bf16(al[rt], bh, acc[rt][bt]);
      }
    }
  }
  float* out = npart + ((size_t)u * S3 + s) * MP * MP;
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int bt = 0; bt < NT; ++bt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = wave * 32 + rt * 16 + 4 * g + i;
        out[(size_t)row * MP + bt * 16 + l16] = acc[rt][bt][i];
      }
}

// ----------------------------------------------------------------- solve ----
// One block per unit.  The split partials are combined here, in a fixed order:
// Y = sum of the full-cache partials, R = Y - (sum of the retained X V0
// partials), N = (sum of the Gram partials) + lambda I (padding rows and
// columns of N become identity rows, padding rows of R zero).  N Z = R is then
// solved by a blocked Cholesky factorisation N = L L^T over 16-wide panels:
//  * factor: for each panel p one wave factors the diagonal block and inverts
//    its factor (row layout, one row per lane of a 16-lane DPP row), the panel
//    below becomes L_ip = A_ip L_pp^-T and the trailing lower blocks take
//    A_ij -= L_ip L_jp^T; the update of the next diagonal block runs first, on
//    the wave that factors it, while the other waves finish the rest;
//  * solve: each wave then owns 16 columns of R in registers and runs the
//    forward (W_p = L_pp^-1 (R_p - sum L_pq W_q)) and backward
//    (Z_p = L_pp^-T (W_p - sum L_qp^T Z_q)) substitutions without barriers.
// Every product is an fp32 MFMA (16x16x4), so the solve stays in fp32.
constexpr int kSolveWaves = 16;

// Broadcast lane J of each 16-lane row to the whole row (DPP row_newbcast).
template <int J>
__device__ __forceinline__ float row_bcast(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x150 + J, 0xF, 0xF, true));
}

template <int J>
__device__ __forceinline__ float row_bcast_rt(int j, float v) {
  if constexpr (J < 16) {
    if (j == J) return row_bcast<J>(v);
    return row_bcast_rt<J + 1>(j, v);
  } else {
    return 0.f;
  }
}

// Factor the 16x16 SPD block at `blk` (LDS, row stride AS) as L L^T and write
// L^-1 (lower triangular, zero above) to `inv` (row stride 20).  Called by a
// whole wave: every 16-lane row factors the block (lane i holds row i), then
// each forms and stores four of the sixteen columns of L^-1.  Returns false
// when a pivot is not positive and finite.
template <int AS>
__device__ __forceinline__ bool factor_diag(const float* blk, float* inv, int lane) {
  const int i = lane & 15;
  float a[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 v = *reinterpret_cast<const float4*>(blk + i * AS + 4 * q);
    a[4 * q] = v.x; a[4 * q + 1] = v.y; a[4 * q + 2] = v.z; a[4 * q + 3] = v.w;
  }
  bool ok = true;
  float invd[16];
  // right-looking: column k is scaled, then the trailing lower part updated;
  // lane i's entries right of its diagonal carry values never read back.
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const float dk = row_bcast_rt<0>(k, a[k]);
    ok = ok && dk > 0.f && dk < __builtin_huge_valf();
    const float r = __builtin_amdgcn_rsqf(dk);   // 1 / L_kk
    invd[k] = r;
    a[k] = (i == k) ? dk * r : a[k] * r;
#pragma unroll
    for (int j = k + 1; j < 16; ++j) a[j] = fmaf(-a[k], row_bcast_rt<0>(j, a[k]), a[j]);
  }
  // L = D M with M unit lower triangular (M_ik = L_ik / L_ii); M^-1 by forward
  // substitution over rows, then L^-1 = M^-1 D^-1 scales column j by 1 / L_jj.
  float dii = 0.f;
#pragma unroll
  for (int k = 0; k < 16; ++k) dii = (i == k) ? invd[k] : dii;
  // Each 16-lane group g of the wave forms columns 4g .. 4g+3 of M^-1 (all
  // groups hold the same factor).  Row k of M^-1 is zero right of its
  // diagonal, so the update of a column j > k adds zero and needs no
  // predicate.
  const int g4 = 4 * (lane >> 4);
  float x[4];
#pragma unroll
  for (int cc = 0; cc < 4; ++cc) x[cc] = (g4 + cc == i) ? 1.f : 0.f;
#pragma unroll
  for (int k = 0; k < 15; ++k) {
    const float mik = (i > k) ? a[k] * dii : 0.f;   // M_ik for the rows below k
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) x[cc] = fmaf(-mik, row_bcast_rt<0>(k, x[cc]), x[cc]);
  }
  float sc[4] = {0.f, 0.f, 0.f, 0.f};   // 1 / L_jj of this group's columns
#pragma unroll
  for (int j = 0; j < 16; ++j)
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) sc[cc] = (g4 + cc == j) ? invd[j] : sc[cc];
  *reinterpret_cast<float4*>(inv + i * 20 + g4) =
      make_float4(x[0] * sc[0], x[1] * sc[1], x[2] * sc[2], x[3] * sc[3]);
  return ok;
}

template <int MP, int D>
__global__ __launch_bounds__(kSolveWaves * 64) void solve_kernel(
    const float* ypart, int S1, const float* xvpart, int S2, const float* npart, int S3,
    const float* mpart, const float* lse1_log2, float lse_bias, float* lse2_log2,
    float* y, float* resid, float* gram, float* z, u16* zhi, u16* zlo, float* stats_ws,
    float* stats_user, int m, float lam, const RagUnit* rag, int csplit, double* zpart,
    const u16* q, const u16* k0, const u16* V, const int32_t* idx, const uint8_t* fixed,
    int64_t n, int w, int c, int causal, float scale_log2) {
  constexpr int NP = MP / 16;   // panels
  constexpr int NC = D / 16;    // 16-column tiles of the right-hand side
  constexpr int AS = MP + 4;    // LDS row strides (floats); 16-byte aligned rows
  constexpr int BS = D + 4;
  constexpr int LS = 20;
  constexpr int NTH = kSolveWaves * 64;
  // A (N, row stride AS) then B (right-hand sides, row stride BS); a unit
  // marked GRKV_UNIT_RANGE reuses the same LDS for the range fix
  constexpr size_t kAB = (size_t)MP * AS + (size_t)MP * BS;
  constexpr size_t kSolveLds = kAB > FixLds<MP, D>::floats ? kAB : FixLds<MP, D>::floats;
  static_assert(kSolveWaves * 64 == kFixThreads, "the range fix runs on the solve's block");
  __shared__ __attribute__((aligned(16))) float AB[kSolveLds];
  float* const A = AB;
  float* const B = AB + MP * AS;
  __shared__ __attribute__((aligned(16))) float Li[NP * 16 * LS];
  __shared__ double red[3][kSolveWaves];
  __shared__ float inv_mass[MP];
  __shared__ int fail, range_fail;

  const int u = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g = lane >> 4;
  // With csplit > 1 the csplit blocks of a unit each factor N and solve
  // their share of the right-hand-side columns; block 0 writes y, resid,
  // gram and the stats, each block the ||Z||^2 of its columns to zpart (the
  // update forms D after from them).
  const int cblk = blockIdx.y;
  const bool lead = cblk == 0;
  // this unit's retained-pass partials: splits sp0 .. sp0 + S2 - 1 (with
  // ragged budgets a unit's own split count, indexed by flat block)
  size_t sp0 = (size_t)u * S2, sp3 = (size_t)u * S3;
  if (rag) {
    const RagUnit ru = rag[u];
    sp0 = sp3 = (size_t)ru.s0;
    S2 = S3 = ru.ns;
  }
  if (tid == 0) fail = range_fail = 0;
  __syncthreads();

  // 0. retained masses: the retained pass forms P against the full-cache
  // log-sum-exp (scaled by 2^lse_bias), so X = P / (row sum of P).  Its
  // log-sum-exp (log2 domain) goes to lse2_log2 for the update.  A row whose
  // retained mass is below 2^-60 after the scaling is outside the range this
  // path resolves: the unit reports GRKV_UNIT_RANGE.
  for (int r = tid; r < MP; r += kSolveWaves * 64) {
    float inv = 1.f;
    if (mpart) {
      // the full-cache LSE and the first four row masses loaded together
      const float l1 = lse1_log2[(size_t)u * MP + r];
      float ms = 0.f;
      for (int s0 = 0; s0 < S2; s0 += 4) {
        float mv[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) mv[k] = mpart[(sp0 + min(s0 + k, S2 - 1)) * MP + r];
#pragma unroll
        for (int k = 0; k < 4; ++k)   // in split order
          if (s0 + k < S2) ms += mv[k];
      }
      inv = 0.f;
      if (r < m) {
        if (ms >= 0x1p-60f && ms < __builtin_huge_valf()) {
          inv = 1.f / ms;
          lse2_log2[(size_t)u * MP + r] = l1 - lse_bias + __log2f(ms);
        } else {
          range_fail = 1;
          lse2_log2[(size_t)u * MP + r] = 0.f;
        }
      }
    }
    inv_mass[r] = inv;
  }
  __syncthreads();
  // a unit marked GRKV_UNIT_RANGE is solved again by its first block (at the
  // end of this kernel), which writes every column of Z^T: the other blocks
  // of the unit have nothing to add
  if (range_fail && !lead) return;   // (LDS flag after the barrier: block-uniform)

  // 1. combine the partials; every thread issues the loads of two elements
  // and four splits at a time before it sums them (in split order), which
  // keeps them in flight together
  double sy = 0.0, sr = 0.0, sz = 0.0;
  auto add4 = [](float4& a, const float4 b) { a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w; };
  // acc[h] += sum over s < S of p[s * stride + e[h]], h = 0, 1, in order of s
  auto sum_parts = [&](const float4* __restrict__ p, size_t stride, int S, const int (&e)[2],
                       float4 (&acc)[2]) {
    int s = 0;
    for (; s + 4 <= S; s += 4) {
      float4 v[4][2];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h) v[i][h] = p[(size_t)(s + i) * stride + e[h]];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h) add4(acc[h], v[i][h]);
    }
    for (; s < S; ++s)
#pragma unroll
      for (int h = 0; h < 2; ++h) add4(acc[h], p[(size_t)s * stride + e[h]]);
  };
  // R = Y - X V0 (scaled by the inverse retained masses) and Y for element
  // e of the [MP][D] arrays (both sums given)
  auto put_r = [&](int e, float4 yy, const float4 xv) {
    const int r = e / (D / 4), c4 = (e % (D / 4)) * 4;
    const float im = inv_mass[r];
    float4 rv = make_float4(yy.x - im * xv.x, yy.y - im * xv.y, yy.z - im * xv.z, yy.w - im * xv.w);
    if (r >= m) yy = rv = make_float4(0.f, 0.f, 0.f, 0.f);
    if (lead) {
      reinterpret_cast<float4*>(y)[(size_t)u * (MP * D / 4) + e] = yy;
      reinterpret_cast<float4*>(resid)[(size_t)u * (MP * D / 4) + e] = rv;
    }
    *reinterpret_cast<float4*>(B + r * BS + c4) = rv;
    sy += (double)yy.x * yy.x + (double)yy.y * yy.y + (double)yy.z * yy.z + (double)yy.w * yy.w;
    sr += (double)rv.x * rv.x + (double)rv.y * rv.y + (double)rv.z * rv.z + (double)rv.w * rv.w;
  };
  // N = Gram sum scaled by the inverse masses, + lambda I (padding: identity)
  auto put_n = [&](int e, const float4 v) {
    const int r = e / (MP / 4), c4 = (e % (MP / 4)) * 4;
    float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int col = c4 + k;
      vv[k] *= inv_mass[r] * inv_mass[col];
      if (r >= m || col >= m) vv[k] = 0.f;
      if (r == col) vv[k] += r < m ? lam : 1.f;
    }
    const float4 o = make_float4(vv[0], vv[1], vv[2], vv[3]);
    if (lead) reinterpret_cast<float4*>(gram)[(size_t)u * (MP * MP / 4) + e] = o;
    *reinterpret_cast<float4*>(A + r * AS + c4) = o;
  };
  // the usual shapes (at most two retained splits, at most four full-cache
  // splits): every load of two elements of Y, X V0 and N in flight together.
  // C1, C2, C3 splits are loaded (indices past S1, S2, S3 read the last
  // split again, in bounds, and are not summed): without branches around the
  // loads; the common split counts get their exact load counts.
  auto combine_small = [&](auto c1, auto c2, auto c3) {
    constexpr int C1 = decltype(c1)::value, C2 = decltype(c2)::value, C3 = decltype(c3)::value;
    constexpr int E = MP * D / 4;
    const float4* __restrict__ yp = reinterpret_cast<const float4*>(ypart) + (size_t)u * S1 * E;
    const float4* __restrict__ xp = reinterpret_cast<const float4*>(xvpart) + sp0 * E;
    const float4* __restrict__ np = reinterpret_cast<const float4*>(npart) + sp3 * E;
    for (int e0 = tid; e0 < E; e0 += 2 * NTH) {
      const int ee[2] = {e0, min(e0 + NTH, E - 1)};
      float4 yv[C1][2], xv[C2][2], nv[C3][2];
#pragma unroll
      for (int sp = 0; sp < C1; ++sp)
#pragma unroll
        for (int h = 0; h < 2; ++h) yv[sp][h] = yp[(size_t)min(sp, S1 - 1) * E + ee[h]];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int sp = 0; sp < C2; ++sp) xv[sp][h] = xp[(size_t)min(sp, S2 - 1) * E + ee[h]];
#pragma unroll
        for (int sp = 0; sp < C3; ++sp) nv[sp][h] = np[(size_t)min(sp, S3 - 1) * E + ee[h]];
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int e = e0 + h * NTH;
        if (e >= E) break;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f), xa = acc, na = acc;
#pragma unroll
        for (int sp = 0; sp < C1; ++sp)   // in split order
          if (sp < S1) add4(acc, yv[sp][h]);
#pragma unroll
        for (int sp = 0; sp < C2; ++sp)
          if (sp < S2) add4(xa, xv[sp][h]);
#pragma unroll
        for (int sp = 0; sp < C3; ++sp)
          if (sp < S3) add4(na, nv[sp][h]);
        put_r(e, acc, xa);
        put_n(e, na);
      }
    }
  };
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I4 = std::integral_constant<int, 4>;
  if (MP == D && S1 == 4 && S2 == 1 && S3 == 1) {
    combine_small(I4{}, I1{}, I1{});   // many units: four full-cache splits
  } else if (MP == D && S1 == 1 && S2 == 1 && S3 == 1) {
    combine_small(I1{}, I1{}, I1{});   // few units: partials summed beforehand
  } else if (MP == D && S1 <= 4 && S2 <= 2 && S3 <= 2) {
    combine_small(I4{}, I2{}, I2{});
  } else {
    {
      constexpr int E = MP * D / 4;
      const float4* __restrict__ yp = reinterpret_cast<const float4*>(ypart) + (size_t)u * S1 * E;
      const float4* __restrict__ xp = reinterpret_cast<const float4*>(xvpart) + sp0 * E;
      for (int e0 = tid; e0 < E; e0 += 2 * NTH) {
        float4 yv[2], xv[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) yv[h] = xv[h] = make_float4(0.f, 0.f, 0.f, 0.f);
        const int e1 = min(e0 + NTH, E - 1);   // the second element, clamped (stored only if < E)
        const int ee[2] = {e0, e1};
        sum_parts(yp, E, S1, ee, yv);
        sum_parts(xp, E, S2, ee, xv);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int e = e0 + h * NTH;
          if (e >= E) break;
          put_r(e, yv[h], xv[h]);
        }
      }
    }
    {
      constexpr int E = MP * MP / 4;
      const float4* __restrict__ np = reinterpret_cast<const float4*>(npart) + sp3 * E;
      for (int e2 = tid; e2 < E; e2 += 2 * NTH) {
        float4 v2[2] = {make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
        const int ee[2] = {e2, min(e2 + NTH, E - 1)};
        sum_parts(np, E, S3, ee, v2);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int e = e2 + h * NTH;
          if (e >= E) break;
          put_n(e, v2[h]);
        }
      }
    }
  }
  __syncthreads();

  // 2. factor N = L L^T in place (lower blocks), L_pp^-1 into Li
  // lower-triangle tile t -> (ii, jj), jj <= ii < T
  auto tri = [](int t, int& ii, int& jj) {
    ii = 0;
    while ((ii + 1) * (ii + 2) / 2 <= t) ++ii;
    jj = t - ii * (ii + 1) / 2;
  };
  bool ok_local = true;
  for (int p = 0; p < NP; ++p) {
    const int p0 = p * 16;
    if (p > 0) {
      // trailing update from panel q = p - 1 over blocks (ib, jb), p <= jb <= ib;
      // tile 0 is the diagonal block (p, p), taken by wave 0
      const int q0 = p0 - 16, T = NP - p, TA = T * (T + 1) / 2;
      for (int t = wave; t < (wave == 0 ? 1 : TA); t += kSolveWaves - 1) {
        int ii, jj;
        tri(t, ii, jj);
        const int i0 = (p + ii) * 16, j0 = (p + jj) * 16;
        const float4 af = *reinterpret_cast<const float4*>(A + (i0 + l16) * AS + q0 + 4 * g);
        const float4 bf = *reinterpret_cast<const float4*>(A + (j0 + l16) * AS + q0 + 4 * g);
        f32x4 acc;
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = A[(i0 + 4 * g + i) * AS + j0 + l16];
        acc = mfma_f32(-af.x, bf.x, acc);
        acc = mfma_f32(-af.y, bf.y, acc);
        acc = mfma_f32(-af.z, bf.z, acc);
        acc = mfma_f32(-af.w, bf.w, acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) A[(i0 + 4 * g + i) * AS + j0 + l16] = acc[i];
      }
    }
    if (wave == 0) ok_local = factor_diag<AS>(A + p0 * AS + p0, Li + p * 16 * LS, lane) && ok_local;
    __syncthreads();
    // panel: L_ip = A_ip L_pp^-T for the blocks below the diagonal
    for (int t = wave; t < NP - 1 - p; t += kSolveWaves) {
      const int i0 = (p + 1 + t) * 16;
      const float4 af = *reinterpret_cast<const float4*>(A + (i0 + l16) * AS + p0 + 4 * g);
      const float4 bf = *reinterpret_cast<const float4*>(Li + (p * 16 + l16) * LS + 4 * g);
      f32x4 acc = zero4();
      acc = mfma_f32(af.x, bf.x, acc);
      acc = mfma_f32(af.y, bf.y, acc);
      acc = mfma_f32(af.z, bf.z, acc);
      acc = mfma_f32(af.w, bf.w, acc);
#pragma unroll
      for (int i = 0; i < 4; ++i) A[(i0 + 4 * g + i) * AS + p0 + l16] = acc[i];
    }
    __syncthreads();
  }
  if (wave == 0 && lane == 0 && !ok_local) fail = 1;
  __syncthreads();
  const bool ok = fail == 0 && range_fail == 0;

  // 3. forward and backward substitution, 16 right-hand-side columns per wave;
  // tile rows 16t + 4g + i, column c0 + l16 live in r[t][i]
  const int tpb = NC / csplit;   // column tiles of this block
  for (int ct = wave; ct < tpb; ct += kSolveWaves) {
    const int c0 = (cblk * tpb + ct) * 16;
    f32x4 r[NP];
#pragma unroll
    for (int t = 0; t < NP; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) r[t][i] = B[(16 * t + 4 * g + i) * BS + c0 + l16];
    // forward: W_p = L_pp^-1 R_p, then R_i -= L_ip W_p for i > p
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const float4 lf = *reinterpret_cast<const float4*>(Li + (p * 16 + l16) * LS + 4 * g);
      f32x4 w = zero4();
      w = mfma_f32(lf.x, r[p][0], w);
      w = mfma_f32(lf.y, r[p][1], w);
      w = mfma_f32(lf.z, r[p][2], w);
      w = mfma_f32(lf.w, r[p][3], w);
      r[p] = w;
      // the updates of the tiles below are independent chains: issued
      // interleaved (k outer) so that the matrix unit is not left waiting on
      // one chain; each tile still sums k = 0..3 in order
      float4 af[NP];
#pragma unroll
      for (int t = p + 1; t < NP; ++t)
        af[t] = *reinterpret_cast<const float4*>(A + (16 * t + l16) * AS + 16 * p + 4 * g);
#pragma unroll
      for (int t = p + 1; t < NP; ++t) r[t] = mfma_f32(-af[t].x, w[0], r[t]);
#pragma unroll
      for (int t = p + 1; t < NP; ++t) r[t] = mfma_f32(-af[t].y, w[1], r[t]);
#pragma unroll
      for (int t = p + 1; t < NP; ++t) r[t] = mfma_f32(-af[t].z, w[2], r[t]);
#pragma unroll
      for (int t = p + 1; t < NP; ++t) r[t] = mfma_f32(-af[t].w, w[3], r[t]);
    }
    // backward: Z_p = L_pp^-T W_p, then W_i -= L_pi^T Z_p for i < p
#pragma unroll
    for (int p = NP - 1; p >= 0; --p) {
      f32x4 zt = zero4();
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        zt = mfma_f32(Li[(p * 16 + 4 * g + kb) * LS + l16], r[p][kb], zt);
      r[p] = zt;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int t = 0; t < p; ++t)
          r[t] = mfma_f32(-A[(16 * p + 4 * g + kb) * AS + 16 * t + l16], zt[kb], r[t]);
    }
    // Z^T out: row dd = c0 + l16, entries 16t + 4g .. +3
    const int dd = c0 + l16;
    float* zr = z + ((size_t)u * D + dd) * MP;
    u16* hr = zhi + ((size_t)u * D + dd) * MP;
    u16* lr = zlo + ((size_t)u * D + dd) * MP;
#pragma unroll
    for (int t = 0; t < NP; ++t) {
      float zv[4];
      u16 hv[4], lv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * t + 4 * g + i;
        zv[i] = ok && row < m ? r[t][i] : 0.f;
        const __bf16 h = (__bf16)zv[i];
        hv[i] = __builtin_bit_cast(u16, h);
        lv[i] = __builtin_bit_cast(u16, (__bf16)(zv[i] - (float)h));
        sz += (double)zv[i] * zv[i];
      }
      *reinterpret_cast<float4*>(zr + 16 * t + 4 * g) = make_float4(zv[0], zv[1], zv[2], zv[3]);
      *reinterpret_cast<uint2*>(hr + 16 * t + 4 * g) =
          make_uint2(hv[0] | ((uint32_t)hv[1] << 16), hv[2] | ((uint32_t)hv[3] << 16));
      *reinterpret_cast<uint2*>(lr + 16 * t + 4 * g) =
          make_uint2(lv[0] | ((uint32_t)lv[1] << 16), lv[2] | ((uint32_t)lv[3] << 16));
    }
  }

  // 4. stats: ||Y||^2, D before = ||R||^2 / ||Y||^2, D after = lambda^2 ||Z||^2 / ||Y||^2
  for (int off = 32; off > 0; off >>= 1) {
    sy += __shfl_xor(sy, off);
    sr += __shfl_xor(sr, off);
    sz += __shfl_xor(sz, off);
  }
  if (lane == 0) { red[0][wave] = sy; red[1][wave] = sr; red[2][wave] = sz; }
  __syncthreads();
  if (tid == 0) {
    double Y2 = 0, R2 = 0, Z2 = 0;
    for (int k = 0; k < kSolveWaves; ++k) { Y2 += red[0][k]; R2 += red[1][k]; Z2 += red[2][k]; }
    const double dn = Y2 > 0 ? Y2 : 1.0;
    const double dbefore = R2 / dn;
    const double dafter = ok ? (double)lam * lam * Z2 / dn : dbefore;
    const float st[4] = {(float)Y2, (float)dbefore, (float)dafter,
                         range_fail ? (float)GRKV_UNIT_RANGE : ok ? 0.f : (float)GRKV_UNIT_SINGULAR};
    if (csplit > 1) {
      zpart[(size_t)u * kZParts + cblk] = Z2;
      if (lead) zpart[(size_t)u * kZParts + kZParts - 1] = Y2;
    }
    for (int k = 0; k < 4; ++k) {
      if (!lead || (csplit > 1 && k == 2)) continue;   // D after: formed by the update
      stats_ws[u * 4 + k] = st[k];
      if (stats_user) stats_user[u * 4 + k] = st[k];
    }
  }
  if (range_fail) {   // only the unit's first block gets here (block-uniform)
    __syncthreads();   // every write above is done, A and B are free
    range_fix_unit<MP, D>(AB, u, q, k0, V, idx, fixed, y, n, m, w, c, causal, scale_log2, lam,
                          lse2_log2, resid, gram, z, zhi, zlo, stats_ws, stats_user, rag, csplit,
                          zpart);
  }
}

// ---------------------------------------------------------------- update ----
// v_out = V0 + X_G^T Z over a range of retained slots per block (fixed slots,
// and every slot of a unit whose system was singular, get V0).  X is
// recomputed from the window queries, K0 and the retained-set log-sum-exp
// rather than stored: S = Q K0^T on the MFMA leaves each lane holding eight
// rows (two groups of four) of one slot's column, which is exactly the A
// operand of X_G^T Z with the rows as the contraction index.  Z^T arrives as
// bf16 hi/lo from the solve; Q, Z^T, -LSE and the block's fixed flags are
// staged in LDS once per block.  A wave works on two 16-slot tiles at a time,
// so every Q and Z^T fragment read from LDS feeds two MFMAs; it loads the K0
// rows of its next pair of tiles and the V0 rows of the current one before
// computing.  The rows of Z^T are staged in the order (dd mod DT) * 16 + dd / DT
// (DT = D / 16 output tiles), which hands each lane DT consecutive output
// columns: V0 and v_out move in 16-byte pieces.
constexpr int kUpdWaves = 8;        // waves per update block
constexpr int kUpdMaxSlots = 4096;  // retained slots per update block at most

template <int MP, int D>
__host__ __device__ constexpr size_t update_lds_bytes(int spb) {
  return ((size_t)MP * (D + 8) + 2 * (size_t)D * (MP + 8)) * sizeof(u16) + MP * sizeof(float) +
         (size_t)spb * sizeof(int32_t) + (size_t)spb;
}

template <int MP, int D>
__global__ __launch_bounds__(kUpdWaves * 64) void update_kernel(
    const u16* q, const u16* k0, const float* lse_log2, const uint8_t* fixed, const u16* zhi,
    const u16* zlo, const float* stats_ws, const u16* V, const int32_t* idx, int64_t n,
    float* v_out, int m, int w, int c, int spb, int causal, float scale_log2, const RagUnit* rag,
    const int32_t* upd_unit, const int32_t* upd_order, const double* zpart, int csplit, float lam,
    float* stats_ws_w, float* stats_user) {
  constexpr int QS = D + 8;    // LDS row stride (bf16) of Q rows
  constexpr int ZS = MP + 8;   // LDS row stride (bf16) of Z^T rows
  constexpr int DT = D / 16;   // output tiles per slot row
  constexpr int NTH = kUpdWaves * 64;
  constexpr float NEG_INF = -__builtin_huge_valf();
  extern __shared__ __attribute__((aligned(16))) u16 sm[];
  u16* qs = sm;                                            // [MP][QS]
  u16* zh = qs + MP * QS;                                  // [D][ZS]
  u16* zl = zh + D * ZS;                                   // [D][ZS]
  float* nls = reinterpret_cast<float*>(zl + D * ZS);      // [MP] -LSE (log2 domain)
  int32_t* ps = reinterpret_cast<int32_t*>(nls + MP);      // [spb] source rows of the slots
  uint8_t* fl = reinterpret_cast<uint8_t*>(ps + spb);      // [spb] fixed flags
  // unit, block within the unit and first slot (ragged budgets: a flat grid
  // of update blocks, each unit's slots packed from its own offset)
  int u = blockIdx.y, blk = blockIdx.x;
  size_t slot0 = (size_t)blockIdx.y * c;
  if (rag) {
    const int f = upd_order[blockIdx.x];
    u = upd_unit[f];
    const RagUnit ru = rag[u];
    blk = f - ru.ub0;
    c = ru.c;
    slot0 = (size_t)ru.off;
  }
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g = lane >> 4;
  const bool singular = stats_ws[u * 4 + 3] != 0.f;
  if (csplit > 1 && blk == 0 && tid == 0) {
    // D after = lambda^2 ||Z||^2 / ||Y||^2 from the solve blocks' column
    // shares, summed in block order
    double Z2 = 0.0;
    for (int k = 0; k < csplit; ++k) Z2 += zpart[(size_t)u * kZParts + k];
    const double Y2 = zpart[(size_t)u * kZParts + kZParts - 1], dn = Y2 > 0 ? Y2 : 1.0;
    const float dafter = singular ? stats_ws[u * 4 + 1] : (float)((double)lam * lam * Z2 / dn);
    stats_ws_w[u * 4 + 2] = dafter;
    if (stats_user) stats_user[u * 4 + 2] = dafter;
  }
  const int win0 = c - w;   // first window slot of the retained set
  const int s0 = blk * spb;
  const int s1 = min(c, s0 + spb);

  // Staging: every thread issues all of its loads (Q rows, Z^T hi/lo, -LSE,
  // the slots' source rows and fixed flags) before its first LDS store, so
  // that they are in flight together.  Q rows past m read row m - 1 (in
  // bounds) and are stored as zeros.
  constexpr int QE = MP * (D / 8), QB = (QE + NTH - 1) / NTH;
  constexpr int ZE = D * (MP / 8), ZB = (ZE + NTH - 1) / NTH;
  constexpr int TB = (kUpdMaxSlots + NTH - 1) / NTH;
  const int ns = s1 - s0;
  uint4 qv[QB], zvh[ZB], zvl[ZB];
  float lv = 0.f;
  int64_t iv[TB];
  uint8_t fv[TB];
  const u16* qu = q + (size_t)u * m * D;
  const u16* zhu = zhi + (size_t)u * D * MP;
  const u16* zlu = zlo + (size_t)u * D * MP;
  if (!singular) {
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      const int e = tid + b * NTH;
      if (QE % NTH == 0 || e < QE) {
        const int r = e / (D / 8), ch = e % (D / 8);
        qv[b] = *reinterpret_cast<const uint4*>(qu + (size_t)min(r, m - 1) * D + ch * 8);
      }
    }
#pragma unroll
    for (int b = 0; b < ZB; ++b) {
      const int e = tid + b * NTH;
      if (ZE % NTH == 0 || e < ZE) {
        const int dd = e / (MP / 8), r0 = 8 * (e % (MP / 8));
        zvh[b] = *reinterpret_cast<const uint4*>(zhu + (size_t)dd * MP + r0);
        zvl[b] = *reinterpret_cast<const uint4*>(zlu + (size_t)dd * MP + r0);
      }
    }
    if (tid < MP) lv = lse_log2[(size_t)u * MP + tid];
  }
#pragma unroll
  for (int b = 0; b < TB; ++b) {   // (slots past ns read slot ns - 1: no branch)
    const int t = min(tid + b * NTH, ns - 1);
    fv[b] = fixed[slot0 + s0 + t];
    iv[b] = idx[slot0 + s0 + t];
  }
  if (!singular) {
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      const int e = tid + b * NTH;
      if (QE % NTH == 0 || e < QE) {
        const int r = e / (D / 8), ch = e % (D / 8);
        *reinterpret_cast<uint4*>(qs + r * QS + ch * 8) = r < m ? qv[b] : make_uint4(0, 0, 0, 0);
      }
    }
    // Z^T row dd goes to LDS row (dd mod DT) * 16 + dd / DT; within a row, Z
    // row r = 32rp + 16h + 4g + i sits at 32rp + 8g + 4h + i, the order in
    // which a lane of group g holds its eight X values (one 16-byte read)
#pragma unroll
    for (int b = 0; b < ZB; ++b) {
      const int e = tid + b * NTH;
      if (ZE % NTH == 0 || e < ZE) {
        const int dd = e / (MP / 8), r0 = 8 * (e % (MP / 8));
        const int row = (dd % DT) * 16 + dd / DT;
        const int rp = r0 >> 5, h = (r0 >> 4) & 1, g0 = (r0 >> 2) & 3;   // rows r0..r0+7: groups g0, g0+1
        const int p0 = row * ZS + 32 * rp + 8 * g0 + 4 * h, p1 = p0 + 8;
        *reinterpret_cast<uint2*>(zh + p0) = make_uint2(zvh[b].x, zvh[b].y);
        *reinterpret_cast<uint2*>(zh + p1) = make_uint2(zvh[b].z, zvh[b].w);
        *reinterpret_cast<uint2*>(zl + p0) = make_uint2(zvl[b].x, zvl[b].y);
        *reinterpret_cast<uint2*>(zl + p1) = make_uint2(zvl[b].z, zvl[b].w);
      }
    }
    // padding rows get -inf, hence probability zero
    if (tid < MP) nls[tid] = tid < m ? -lv : NEG_INF;
  }
#pragma unroll
  for (int b = 0; b < TB; ++b) {
    const int t = tid + b * NTH;
    if (t < ns) {
      fl[t] = fv[b];
      const int64_t r = iv[b];
      ps[t] = (int32_t)(r < 0 ? 0 : r >= n ? n - 1 : r);   // in range by construction
    }
  }
  __syncthreads();

  auto load_k = [&](int tb, uint4 (&kb)[2][D / 32]) {
#pragma unroll
    for (int T = 0; T < 2; ++T) {
      const int t = tb + 16 * T + l16;
      const u16* kr = k0 + (slot0 + (t < s1 ? t : s1 - 1)) * D;
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) kb[T][ks] = *reinterpret_cast<const uint4*>(kr + ks * 32 + 8 * g);
    }
  };
  uint4 kb[2][D / 32];
  int tb = s0 + 32 * wave;
  for (; tb < s1; tb += 32 * kUpdWaves) {
    // this pair's K0 rows (the other waves of the block hide their latency)
    if (!singular) load_k(tb, kb);
    // V0 rows of this pair (slot tb + 16T + 4g + i, columns l16 * DT ..),
    // loaded now so that they arrive during the products
    uint32_t v0r[2][4][DT / 2];
#pragma unroll
    for (int T = 0; T < 2; ++T)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ts = min(tb + 16 * T + 4 * g + i, s1 - 1);
        const u16* src = V + ((size_t)u * n + ps[ts - s0]) * D + l16 * DT;
        if constexpr (DT == 8) {
          const uint4 r4 = *reinterpret_cast<const uint4*>(src);
          v0r[T][i][0] = r4.x; v0r[T][i][1] = r4.y; v0r[T][i][2] = r4.z; v0r[T][i][3] = r4.w;
        } else {
          const uint2 r2 = *reinterpret_cast<const uint2*>(src);
          v0r[T][i][0] = r2.x; v0r[T][i][1] = r2.y;
        }
      }
    f32x4 acc[2][DT];
#pragma unroll
    for (int T = 0; T < 2; ++T)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) acc[T][dt] = zero4();
    if (!singular) {
      float cm[2];   // 0 for a free slot, -inf for a fixed or missing one
      int tw[2];     // window index of the slot (< 0 outside the window)
#pragma unroll
      for (int T = 0; T < 2; ++T) {
        const int t = tb + 16 * T + l16;   // the slot whose column this lane holds
        cm[T] = (t < s1 && !fl[t - s0]) ? 0.f : NEG_INF;
        tw[T] = t - win0;
      }
      // X_G^T Z for this pair of tiles; WIN adds the causal rule of the window
      // slots, which only the last tiles of the retained set contain
      auto pair_product = [&](auto win_tag) {
        constexpr bool WIN = decltype(win_tag)::value;
#pragma unroll
        for (int rp = 0; rp < MP / 32; ++rp) {
          bf16x8 ah[2], al[2];
          float x8[2][8];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int rt = 2 * rp + h;
            f32x4 st[2] = {zero4(), zero4()};
#pragma unroll
            for (int ks = 0; ks < D / 32; ++ks) {
              const bf16x8 qa = as_bf16x8(*reinterpret_cast<const uint4*>(qs + (rt * 16 + l16) * QS + ks * 32 + 8 * g));
              st[0] = mfma_bf16(qa, as_bf16x8(kb[0][ks]), st[0]);
              st[1] = mfma_bf16(qa, as_bf16x8(kb[1][ks]), st[1]);
            }
            const float4 nv = *reinterpret_cast<const float4*>(nls + rt * 16 + 4 * g);
            const float nl[4] = {nv.x, nv.y, nv.z, nv.w};
            // st[T][i] = q_row . k_t for row = 16rt + 4g + i
#pragma unroll
            for (int T = 0; T < 2; ++T)
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                float arg = fmaf(st[T][i], scale_log2, nl[i]) + cm[T];
                if constexpr (WIN) {
                  if (tw[T] > (rt * 16 + 4 * g + i) % w) arg = NEG_INF;
                }
                x8[T][4 * h + i] = __builtin_amdgcn_exp2f(arg);
              }
          }
#pragma unroll
          for (int T = 0; T < 2; ++T) split8(x8[T], ah[T], al[T]);
          // the eight rows {32rp + 4g + i, 32rp + 16 + 4g + i} of a lane form
          // its A operand; Z^T rows in the permuted order above, output
          // column l16 * DT + dt
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const int zo = (dt * 16 + l16) * ZS + 32 * rp + 8 * g;
            const bf16x8 bh = as_bf16x8(*reinterpret_cast<const uint4*>(zh + zo));
            const bf16x8 bl = as_bf16x8(*reinterpret_cast<const uint4*>(zl + zo));
#pragma unroll
            for (int T = 0; T < 2; ++T) {
              acc[T][dt] = mfma_bf16(ah[T], bh, acc[T][dt]);
              acc[T][dt] = mfma_bf16(ah[T], bl, acc[T][dt]);
              acc[T][dt] = mfma_bf16(al[T], bh, acc[T][dt]);
            }
          }
        }
      };
      if (causal && tb + 31 >= win0)   // wave-uniform
        pair_product(std::true_type{});
      else
        pair_product(std::false_type{});
    }
    // lane holds dV[slot = tb + 16T + 4g + i][dd = l16 * DT + dt]
#pragma unroll
    for (int T = 0; T < 2; ++T)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ts = tb + 16 * T + 4 * g + i;
        if (ts >= s1) continue;
        const bool upd = !singular && !fl[ts - s0];
        float v[DT];
#pragma unroll
        for (int k = 0; k < DT / 2; ++k) {
          v[2 * k] = __uint_as_float(v0r[T][i][k] << 16);
          v[2 * k + 1] = __uint_as_float(v0r[T][i][k] & 0xffff0000u);
        }
        if (upd) {
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) v[dt] += acc[T][dt][i];
        }
        float* dst = v_out + (slot0 + ts) * D + l16 * DT;
#pragma unroll
        for (int k = 0; k < DT / 4; ++k)
          *reinterpret_cast<float4*>(dst + 4 * k) = make_float4(v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]);
      }
  }
}

template <int WAVES>
hipError_t launch_gram_w(const Plan& p, const float* x, const uint8_t* fixed, float* npart,
                         hipStream_t s) {
  hipLaunchKernelGGL(gram_kernel<WAVES>, dim3(p.S3, p.U), dim3(WAVES * 64), 0, s, x, fixed, npart,
                     p.c, p.S3, p.chunk3);
  return hipGetLastError();
}

template <int MP, int D>
hipError_t launch_solve_t(const Plan& p, const float* ypart, int S1, int S2, const float* xvpart,
                          const float* npart, const float* mpart, const float* lse1_log2,
                          float lse_bias, float* lse2_log2, float* y, float* resid, float* gram,
                          float* z, u16* zhi, u16* zlo, float* stats_ws, float* stats_user,
                          double* zpart, const void* q, const void* k0, const void* V,
                          const int32_t* idx, const uint8_t* fixed, hipStream_t s) {
  const int csplit = p.rag ? 1 : p.csplit;
  if (csplit < 1 || csplit > kZParts - 1 || (D / 16) % csplit != 0) return hipErrorInvalidValue;
  // the range fix (with mpart) reads q_obs, K0, V and the retained set
  if (mpart && (!q || !k0 || !V || !idx || !fixed)) return hipErrorInvalidValue;
  const float scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  hipLaunchKernelGGL((solve_kernel<MP, D>), dim3(p.U, csplit), dim3(kSolveWaves * 64), 0, s,
                     ypart, S1, xvpart, S2, npart, S2, mpart, lse1_log2, lse_bias, lse2_log2, y,
                     resid, gram, z, zhi, zlo, stats_ws, stats_user, p.m, p.lam, p.rag, csplit,
                     zpart, (const u16*)q, (const u16*)k0, (const u16*)V, idx, fixed, p.n, p.w,
                     p.c, p.opt.causal_window ? 1 : 0, scale_log2);
  return hipGetLastError();
}

template <int MP, int D>
hipError_t launch_update_t(const Plan& p, const void* q, const void* k0, const float* lse_log2,
                           const uint8_t* fixed, const u16* zhi, const u16* zlo,
                           const float* stats_ws, const u16* V, const int32_t* idx,
                           float* v_out, const double* zpart, float* stats_ws_w,
                           float* stats_user, hipStream_t s) {
  int spb = p.rag ? p.upd_spb : update_slots_per_block(p, p.c);
  if (spb < 32 || spb > kUpdMaxSlots ||
      (p.rag && (!p.rag_upd_unit || !p.rag_upd_order || p.rag_upd_blocks < 1)))
    return hipErrorInvalidValue;
  const int bpu = (p.c + spb - 1) / spb;
  const size_t lds = update_lds_bytes<MP, D>(spb);
  hipError_t e = hipFuncSetAttribute((const void*)update_kernel<MP, D>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const float scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  const dim3 grid = p.rag ? dim3(p.rag_upd_blocks, 1) : dim3(bpu, p.U);
  hipLaunchKernelGGL((update_kernel<MP, D>), grid, dim3(kUpdWaves * 64), lds, s,
                     (const u16*)q, (const u16*)k0, lse_log2, fixed, zhi, zlo, stats_ws, V, idx,
                     p.n, v_out, p.m, p.w, p.c, spb, p.opt.causal_window ? 1 : 0, scale_log2,
                     p.rag, p.rag_upd_unit, p.rag_upd_order, zpart, p.rag ? 1 : p.csplit, p.lam,
                     stats_ws_w, stats_user);
  return hipGetLastError();
}

}  // namespace

int update_slots_per_block(const Plan& p, int c) {
  // about one block per compute unit: split a unit's slots over several
  // blocks only when there are fewer units than that, down to 128 slots per
  // block (half of the waves' 32-slot pairs: a one-layer call at c = 2048
  // measured 156 us per call with 128 or 64 slots per block, 158 with 256)
  const int least_slots = 16 * kUpdWaves;
  int bpu = (256 + p.U - 1) / p.U;
  const int most = (c + least_slots - 1) / least_slots;
  if (bpu > most) bpu = most;
  const int least = (c + kUpdMaxSlots - 1) / kUpdMaxSlots;
  if (bpu < least) bpu = least;
  if (bpu < 1) bpu = 1;
  int spb = (c + bpu - 1) / bpu;
  return (spb + 31) / 32 * 32;
}

bool merge_fast_supported(const Plan& p) {
  return p.dtype == GRKV_BF16 && p.mp <= 128 && (p.d == 64 || p.d == 128);
}

hipError_t launch_gram(const Plan& p, const float* x, const uint8_t* fixed, float* npart,
                       hipStream_t s) {
  switch (p.waves) {
    case 1: return launch_gram_w<1>(p, x, fixed, npart, s);
    case 2: return launch_gram_w<2>(p, x, fixed, npart, s);
    case 4: return launch_gram_w<4>(p, x, fixed, npart, s);
    case 8: return launch_gram_w<8>(p, x, fixed, npart, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_solve(const Plan& p, const float* ypart, int S1, int S2, const float* xvpart,
                        const float* npart,
                        const float* mpart, const float* lse1_log2, float lse_bias,
                        float* lse2_log2, float* y, float* resid, float* gram, float* z, u16* zhi,
                        u16* zlo, float* stats_ws, float* stats_user, double* zpart,
                        const void* q, const void* k0, const void* V, const int32_t* idx,
                        const uint8_t* fixed, hipStream_t s) {
#define GRKV_SOLVE(MPV, DV)                                                                   \
  if (p.mp == MPV && p.d == DV)                                                               \
    return launch_solve_t<MPV, DV>(p, ypart, S1, S2, xvpart, npart, mpart, lse1_log2, lse_bias, \
                                   lse2_log2, y, resid, gram, z, zhi, zlo, stats_ws,            \
                                   stats_user, zpart, q, k0, V, idx, fixed, s);
  GRKV_SOLVE(32, 64) GRKV_SOLVE(32, 128) GRKV_SOLVE(64, 64) GRKV_SOLVE(64, 128)
  GRKV_SOLVE(128, 64) GRKV_SOLVE(128, 128)
#undef GRKV_SOLVE
  return hipErrorInvalidValue;
}

hipError_t launch_update(const Plan& p, const void* q, const void* k0, const float* lse_log2,
                         const uint8_t* fixed, const u16* zhi, const u16* zlo,
                         const float* stats_ws, const void* V, const int32_t* idx, float* v_out,
                         const double* zpart, float* stats_user, hipStream_t s) {
#define GRKV_UPD(MPV, DV)                                                                     \
  if (p.mp == MPV && p.d == DV)                                                               \
    return launch_update_t<MPV, DV>(p, q, k0, lse_log2, fixed, zhi, zlo, stats_ws,             \
                                    (const u16*)V, idx, v_out, zpart,                          \
                                    const_cast<float*>(stats_ws), stats_user, s);
  GRKV_UPD(32, 64) GRKV_UPD(32, 128) GRKV_UPD(64, 64) GRKV_UPD(64, 128)
  GRKV_UPD(128, 64) GRKV_UPD(128, 128)
#undef GRKV_UPD
  return hipErrorInvalidValue;
}

}  // namespace grkv
