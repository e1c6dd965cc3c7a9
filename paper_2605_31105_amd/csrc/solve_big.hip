// Solve of the value step (Eq. 8; App. D.1) for 256 stacked window rows
// (G * w in (128, 256]), where N = X_G X_G^T + lambda I is 256 x 256:
// too large for the row-major LDS layout of the m <= 128 solve, too slow for
// a column-by-column factorisation.
//
// One block of 8 waves per unit.  N's lower triangle is held in LDS as
// 136 16 x 16 blocks (139 KB), block (I, J), J <= I, at index I(I+1)/2 + J,
// each row-major with its four 16-byte chunks of row r rotated by r mod 4 so
// that a wave's float4 reads of one chunk column fall on distinct banks.
// The factorisation N = L L^T is the blocked right-looking one of the m <= 128
// solve: for every 16-wide panel one wave factors the diagonal block and
// inverts its factor, the blocks below become L_ip = A_ip L_pp^-T, and the
// trailing lower blocks take A_ij -= L_ip L_jp^T, all on fp32 MFMA (16x16x4).
// The right-hand sides R are read from global memory straight into registers
// (16 columns per wave) for the forward and backward substitutions.
//
// Inputs are the generic value step's: the Gram partials npart [U][S3][mp][mp]
// of the stored X (the caller sums them over all units with one wide launch
// first and passes that sum, S3 = 1: read by one block per unit, 2 MB of
// partials take longer than the factorisation), and Y and R = Y - X V0
// combined [U][mp][D].  Outputs: the full N (gram), Z^T (z [U][D][mp]) and
// the stats, as the generic solve.
#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

constexpr int kBigMP = 256;
constexpr int kBigWaves = 8;
constexpr int kBigNP = kBigMP / 16;                        // panels
constexpr int kBigBlocks = kBigNP * (kBigNP + 1) / 2;      // lower 16 x 16 blocks
constexpr int kBigLS = 20;                                 // row stride of the inverted diagonal factors
constexpr int kBigBatch = 8;                               // N elements loaded together per thread

__device__ __forceinline__ int blk_index(int I, int J) { return I * (I + 1) / 2 + J; }

// Float offset of element (r, c) (0 <= r, c < 16) inside a block.
__device__ __forceinline__ int blk_off(int r, int c) {
  return r * 16 + ((((c >> 2) ^ (r & 3)) << 2) | (c & 3));
}
// Float offset of chunk q (columns 4q .. 4q+3) of row r inside a block.
__device__ __forceinline__ int blk_chunk(int r, int q) { return r * 16 + ((q ^ (r & 3)) << 2); }

template <int J>
__device__ __forceinline__ float bcast_row(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x150 + J, 0xF, 0xF, true));
}
template <int J>
__device__ __forceinline__ float bcast_row_rt(int j, float v) {
  if constexpr (J < 16) {
    if (j == J) return bcast_row<J>(v);
    return bcast_row_rt<J + 1>(j, v);
  } else {
    return 0.f;
  }
}

// L L^T of the SPD diagonal block `blk`; L^-1 (lower, zero above) to `inv`
// (row stride kBigLS).  Called by a whole wave: every 16-lane row factors the
// block (lane i holds row i), then each forms and stores four of the sixteen
// columns of L^-1.  False when a pivot is not positive and finite.
__device__ __forceinline__ bool factor_diag_blk(const float* blk, float* inv, int lane) {
  const int i = lane & 15;
  float a[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 v = *reinterpret_cast<const float4*>(blk + blk_chunk(i, q));
    a[4 * q] = v.x; a[4 * q + 1] = v.y; a[4 * q + 2] = v.z; a[4 * q + 3] = v.w;
  }
  bool ok = true;
  float invd[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const float dk = bcast_row_rt<0>(k, a[k]);
    ok = ok && dk > 0.f && dk < __builtin_huge_valf();
    const float r = __builtin_amdgcn_rsqf(dk);   // 1 / L_kk
    invd[k] = r;
    a[k] = (i == k) ? dk * r : a[k] * r;
#pragma unroll
    for (int j = k + 1; j < 16; ++j) a[j] = fmaf(-a[k], bcast_row_rt<0>(j, a[k]), a[j]);
  }
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
    const float mik = (i > k) ? a[k] * dii : 0.f;
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) x[cc] = fmaf(-mik, bcast_row_rt<0>(k, x[cc]), x[cc]);
  }
  float sc[4] = {0.f, 0.f, 0.f, 0.f};   // 1 / L_jj of this group's columns
#pragma unroll
  for (int j = 0; j < 16; ++j)
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) sc[cc] = (g4 + cc == j) ? invd[j] : sc[cc];
  *reinterpret_cast<float4*>(inv + i * kBigLS + g4) =
      make_float4(x[0] * sc[0], x[1] * sc[1], x[2] * sc[2], x[3] * sc[3]);
  return ok;
}

template <int D>
__global__ __launch_bounds__(kBigWaves * 64) void solve_big_kernel(
    const float* npart, int S3, const float* y, const float* resid, float* gram, float* z,
    float* stats_ws, float* stats_user, int m, float lam) {
  constexpr int MP = kBigMP, NP = kBigNP, NC = D / 16, NTH = kBigWaves * 64;
  __shared__ __attribute__((aligned(16))) float A[kBigBlocks * 256];
  __shared__ __attribute__((aligned(16))) float Li[NP * 16 * kBigLS];
  __shared__ double red[3][kBigWaves];
  __shared__ int fail;

  const int u = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g = lane >> 4;
  if (tid == 0) fail = 0;

  // 1. N = sum of the Gram partials + lambda I (padding rows and columns:
  // identity), to LDS (lower blocks) and to gram (all of it).  A thread
  // issues the loads of kBigBatch elements before it uses them (with one
  // partial, the usual case, they are all in flight together).
  {
    constexpr int E = MP * MP / 4;
    static_assert(E % (kBigBatch * NTH) == 0, "whole batches");
    const float4* np = reinterpret_cast<const float4*>(npart) + (size_t)u * S3 * E;
    float4* go = reinterpret_cast<float4*>(gram) + (size_t)u * E;
    for (int e0 = tid; e0 < E; e0 += kBigBatch * NTH) {
      float4 vb[kBigBatch];
#pragma unroll
      for (int b = 0; b < kBigBatch; ++b) vb[b] = np[e0 + b * NTH];
      for (int s = 1; s < S3; ++s)   // in split order
#pragma unroll
        for (int b = 0; b < kBigBatch; ++b) {
          const float4 t = np[(size_t)s * E + e0 + b * NTH];
          vb[b].x += t.x; vb[b].y += t.y; vb[b].z += t.z; vb[b].w += t.w;
        }
#pragma unroll
      for (int b = 0; b < kBigBatch; ++b) {
        const int e = e0 + b * NTH;
        const int r = e / (MP / 4), c0 = (e % (MP / 4)) * 4;
        float vv[4] = {vb[b].x, vb[b].y, vb[b].z, vb[b].w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int c = c0 + k;
          if (r >= m || c >= m) vv[k] = 0.f;
          if (r == c) vv[k] += r < m ? lam : 1.f;
        }
        go[e] = make_float4(vv[0], vv[1], vv[2], vv[3]);
        const int I = r >> 4, J = c0 >> 4;
        if (J <= I)
          *reinterpret_cast<float4*>(A + blk_index(I, J) * 256 + blk_chunk(r & 15, (c0 & 15) >> 2)) =
              make_float4(vv[0], vv[1], vv[2], vv[3]);
      }
    }
  }
  __syncthreads();

  // 2. N = L L^T in place (lower blocks); L_pp^-1 into Li
  auto tri = [](int t, int& ii, int& jj) {
    ii = 0;
    while ((ii + 1) * (ii + 2) / 2 <= t) ++ii;
    jj = t - ii * (ii + 1) / 2;
  };
  bool ok_local = true;
  for (int p = 0; p < NP; ++p) {
    if (p > 0) {
      // trailing update from panel q = p - 1 over blocks (p + ii, p + jj),
      // jj <= ii; tile 0, the next diagonal block, goes to wave 0 alone
      const int q = p - 1, T = NP - p, TA = T * (T + 1) / 2;
      for (int t = wave; t < (wave == 0 ? 1 : TA); t += kBigWaves - 1) {
        int ii, jj;
        tri(t, ii, jj);
        const int I = p + ii, J = p + jj;
        const float4 af = *reinterpret_cast<const float4*>(A + blk_index(I, q) * 256 + blk_chunk(l16, g));
        const float4 bf = *reinterpret_cast<const float4*>(A + blk_index(J, q) * 256 + blk_chunk(l16, g));
        float* cb = A + blk_index(I, J) * 256;
        f32x4 acc;
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = cb[blk_off(4 * g + i, l16)];
        acc = mfma_f32(-af.x, bf.x, acc);
        acc = mfma_f32(-af.y, bf.y, acc);
        acc = mfma_f32(-af.z, bf.z, acc);
        acc = mfma_f32(-af.w, bf.w, acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) cb[blk_off(4 * g + i, l16)] = acc[i];
      }
    }
    if (wave == 0) ok_local = factor_diag_blk(A + blk_index(p, p) * 256, Li + p * 16 * kBigLS, lane) && ok_local;
    __syncthreads();
    // panel: L_ip = A_ip L_pp^-T for the blocks below the diagonal
    for (int t = wave; t < NP - 1 - p; t += kBigWaves) {
      const int I = p + 1 + t;
      float* cb = A + blk_index(I, p) * 256;
      const float4 af = *reinterpret_cast<const float4*>(cb + blk_chunk(l16, g));
      const float4 bf = *reinterpret_cast<const float4*>(Li + (p * 16 + l16) * kBigLS + 4 * g);
      f32x4 acc = zero4();
      acc = mfma_f32(af.x, bf.x, acc);
      acc = mfma_f32(af.y, bf.y, acc);
      acc = mfma_f32(af.z, bf.z, acc);
      acc = mfma_f32(af.w, bf.w, acc);
      // every lane of the wave has read the block (one MFMA operand each)
      // before any lane writes it back
#pragma unroll
      for (int i = 0; i < 4; ++i) cb[blk_off(4 * g + i, l16)] = acc[i];
    }
    __syncthreads();
  }
  if (wave == 0 && lane == 0 && !ok_local) fail = 1;
  __syncthreads();
  const bool ok = fail == 0;

  // 3. forward and backward substitution, 16 right-hand-side columns per
  // wave; tile rows 16t + 4g + i, column c0 + l16 live in r[t][i]
  double sy = 0.0, sr = 0.0, sz = 0.0;
  for (int cb = wave; cb < NC; cb += kBigWaves) {
    const int c0 = cb * 16;
    const float* ru = resid + (size_t)u * MP * D;
    const float* yu = y + (size_t)u * MP * D;
    // every row of the [MP][D] arrays is read (rows past m are in bounds)
    // and masked afterwards: loads without branches stay in flight together.
    // Row 16t + 4g + i of column c0 + l16 is the uniform row base of 16t + i
    // plus one 32-bit lane offset.
    const uint32_t lo = (uint32_t)(4 * g * D + c0 + l16);
    f32x4 r[NP];
#pragma unroll
    for (int t = 0; t < NP; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) r[t][i] = (ru + (16 * t + i) * D)[lo];
#pragma unroll
    for (int t = 0; t < NP; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool in = 16 * t + 4 * g + i < m;
        const float rv = in ? r[t][i] : 0.f;
        r[t][i] = rv;
        sr += (double)rv * rv;
      }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const float4 lf = *reinterpret_cast<const float4*>(Li + (p * 16 + l16) * kBigLS + 4 * g);
      f32x4 w = zero4();
      w = mfma_f32(lf.x, r[p][0], w);
      w = mfma_f32(lf.y, r[p][1], w);
      w = mfma_f32(lf.z, r[p][2], w);
      w = mfma_f32(lf.w, r[p][3], w);
      r[p] = w;
#pragma unroll
      for (int t = p + 1; t < NP; ++t) {
        const float4 af = *reinterpret_cast<const float4*>(A + blk_index(t, p) * 256 + blk_chunk(l16, g));
        r[t] = mfma_f32(-af.x, w[0], r[t]);
        r[t] = mfma_f32(-af.y, w[1], r[t]);
        r[t] = mfma_f32(-af.z, w[2], r[t]);
        r[t] = mfma_f32(-af.w, w[3], r[t]);
      }
    }
#pragma unroll
    for (int p = NP - 1; p >= 0; --p) {
      f32x4 zt = zero4();
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) zt = mfma_f32(Li[(p * 16 + 4 * g + kb) * kBigLS + l16], r[p][kb], zt);
      r[p] = zt;
#pragma unroll
      for (int t = 0; t < p; ++t) {
        const float* lb = A + blk_index(p, t) * 256;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) r[t] = mfma_f32(-lb[blk_off(4 * g + kb, l16)], zt[kb], r[t]);
      }
    }
    float* zr = z + ((size_t)u * D + c0 + l16) * MP;
#pragma unroll
    for (int t = 0; t < NP; ++t) {
      float zv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * t + 4 * g + i;
        zv[i] = ok && row < m ? r[t][i] : 0.f;
        sz += (double)zv[i] * zv[i];
      }
      *reinterpret_cast<float4*>(zr + 16 * t + 4 * g) = make_float4(zv[0], zv[1], zv[2], zv[3]);
    }
    // ||Y||^2 of these columns (after the substitution, whose registers are
    // free again), all 64 loads in flight before the sum
    float yv[NP][4];
#pragma unroll
    for (int t = 0; t < NP; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) yv[t][i] = (yu + (16 * t + i) * D)[lo];
#pragma unroll
    for (int t = 0; t < NP; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float yy = 16 * t + 4 * g + i < m ? yv[t][i] : 0.f;
        sy += (double)yy * yy;
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
    for (int k = 0; k < kBigWaves; ++k) { Y2 += red[0][k]; R2 += red[1][k]; Z2 += red[2][k]; }
    const double dn = Y2 > 0 ? Y2 : 1.0;
    const double dbefore = R2 / dn;
    const double dafter = ok ? (double)lam * lam * Z2 / dn : dbefore;
    const float st[4] = {(float)Y2, (float)dbefore, (float)dafter,
                         ok ? (float)GRKV_UNIT_OK : (float)GRKV_UNIT_SINGULAR};
    for (int k = 0; k < 4; ++k) {
      stats_ws[u * 4 + k] = st[k];
      if (stats_user) stats_user[u * 4 + k] = st[k];
    }
  }
}

}  // namespace

bool solve_big_supported(const Plan& p) { return p.mp == kBigMP && (p.d == 64 || p.d == 128); }

hipError_t launch_solve_big(const Plan& p, const float* npart, int S3, const float* y,
                            const float* resid, float* gram, float* z, float* stats_ws,
                            float* stats_user, hipStream_t s) {
  if (!solve_big_supported(p) || S3 < 1) return hipErrorInvalidValue;
  if (npart == gram && S3 != 1) return hipErrorInvalidValue;
  if (p.d == 128)
    hipLaunchKernelGGL(solve_big_kernel<128>, dim3(p.U), dim3(kBigWaves * 64), 0, s, npart, S3,
                       y, resid, gram, z, stats_ws, stats_user, p.m, p.lam);
  else
    hipLaunchKernelGGL(solve_big_kernel<64>, dim3(p.U), dim3(kBigWaves * 64), 0, s, npart, S3,
                       y, resid, gram, z, stats_ws, stats_user, p.m, p.lam);
  return hipGetLastError();
}

}  // namespace grkv
