// Generic value-step kernels for shapes outside the fast path (float32
// inputs, or m > 128 rows), which store X: Cholesky of N in LDS (packed lower
// triangle, the right-hand sides in LDS when they fit and in the z buffer
// otherwise; 256 rows have a blocked solve of their own), then
// V* = V0 + X_G^T Z over every retained slot from X, Z^T and the compact V0
// copy.  update_add_kernel adds X_G^T Z into a v_out that already holds V0
// (the later alternating steps of the key-step entry point).  Same arithmetic
// contract as merge.hip.
#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

__device__ __forceinline__ int tri(int i, int j) { return i * (i + 1) / 2 + j; }

// One block per unit.  L (packed lower triangle) lives in LDS; the right-hand
// sides W are in LDS when they fit (w_in_lds) and otherwise in the z buffer.
__global__ __launch_bounds__(256) void chol_kernel(const float* npart, int S3, const float* y,
                                                  const float* resid, float* gram, float* z,
                                                  float* stats_ws, float* stats_user, int m,
                                                  int mp, int D, float lam, int w_in_lds) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  __shared__ int fail;
  __shared__ double red[3][4];
  const int u = blockIdx.x, tid = threadIdx.x;
  float* L = lds;
  const int ntri = mp * (mp + 1) / 2;
  float* zu = z + (size_t)u * D * mp;  // Z^T [D][mp]
  float* Wl = lds + ((ntri + 3) & ~3);
  // W(i, col): LDS [mp][D] or global [D][mp]
  float* Wb = w_in_lds ? Wl : zu;
  const int si = w_in_lds ? D : 1, sc = w_in_lds ? 1 : mp;

  if (tid == 0) fail = 0;
  const float* np = npart + (size_t)u * S3 * mp * mp;
  float* gu = gram + (size_t)u * mp * mp;
  for (int e = tid; e < mp * mp; e += blockDim.x) {
    int i = e / mp, j = e % mp;
    float v = 0.f;
    for (int s = 0; s < S3; ++s) v += np[(size_t)s * mp * mp + e];
    if (i == j) v += (i < m) ? lam : 1.f;
    gu[e] = v;
    if (j <= i) L[tri(i, j)] = v;
  }
  const float* ru = resid + (size_t)u * mp * D;
  for (int e = tid; e < mp * D; e += blockDim.x) {
    int i = e / D, col = e % D;
    Wb[i * si + col * sc] = ru[e];
  }
  __syncthreads();

  for (int k = 0; k < mp; ++k) {
    if (tid == 0) {
      float dkk = L[tri(k, k)];
      if (!(dkk > 0.f) || !isfinite(dkk)) { fail = 1; dkk = 1.f; }
      L[tri(k, k)] = sqrtf(dkk);
    }
    __syncthreads();
    const float inv = 1.f / L[tri(k, k)];
    for (int i = k + 1 + tid; i < mp; i += blockDim.x) L[tri(i, k)] *= inv;
    __syncthreads();
    const int rem = mp - k - 1;
    for (int e = tid; e < rem * rem; e += blockDim.x) {
      int i = k + 1 + e / rem, j = k + 1 + e % rem;
      if (j <= i) L[tri(i, j)] -= L[tri(i, k)] * L[tri(j, k)];
    }
    __syncthreads();
  }
  const bool ok = fail == 0;

  // forward (L W = R) then backward (L^T Z = W), one right-hand side per thread
  for (int col = tid; col < D; col += blockDim.x) {
    if (!ok) {
      for (int i = 0; i < mp; ++i) Wb[i * si + col * sc] = 0.f;
      continue;
    }
    for (int i = 0; i < mp; ++i) {
      float acc = Wb[i * si + col * sc];
      for (int j = 0; j < i; ++j) acc -= L[tri(i, j)] * Wb[j * si + col * sc];
      Wb[i * si + col * sc] = acc / L[tri(i, i)];
    }
    for (int i = mp - 1; i >= 0; --i) {
      float acc = Wb[i * si + col * sc];
      for (int j = i + 1; j < mp; ++j) acc -= L[tri(j, i)] * Wb[j * si + col * sc];
      Wb[i * si + col * sc] = acc / L[tri(i, i)];
    }
  }
  __syncthreads();
  if (w_in_lds)
    for (int e = tid; e < mp * D; e += blockDim.x) {
      int col = e / mp, i = e % mp;
      zu[e] = Wl[i * D + col];
    }

  // stats: ||Y||^2, ||R||^2, ||Z||^2 over the m real rows
  const float* yu = y + (size_t)u * mp * D;
  double sy = 0.0, sr = 0.0, sz = 0.0;
  for (int e = tid; e < m * D; e += blockDim.x) {
    int i = e / D, col = e % D;
    double yv = yu[e], rv = ru[e], zv = Wb[i * si + col * sc];
    sy += yv * yv;
    sr += rv * rv;
    sz += zv * zv;
  }
  for (int off = 32; off > 0; off >>= 1) {
    sy += __shfl_xor(sy, off);
    sr += __shfl_xor(sr, off);
    sz += __shfl_xor(sz, off);
  }
  if ((tid & 63) == 0) { red[0][tid >> 6] = sy; red[1][tid >> 6] = sr; red[2][tid >> 6] = sz; }
  __syncthreads();
  if (tid == 0) {
    double Y2 = 0, R2 = 0, Z2 = 0;
    for (int k = 0; k < (int)(blockDim.x >> 6); ++k) { Y2 += red[0][k]; R2 += red[1][k]; Z2 += red[2][k]; }
    double dn = Y2 > 0 ? Y2 : 1.0;
    double dbefore = R2 / dn;
    double dafter = ok ? (double)lam * lam * Z2 / dn : dbefore;
    float st[4] = {(float)Y2, (float)dbefore, (float)dafter, ok ? 0.f : (float)GRKV_UNIT_SINGULAR};
    for (int k = 0; k < 4; ++k) {
      stats_ws[u * 4 + k] = st[k];
      if (stats_user) stats_user[u * 4 + k] = st[k];
    }
  }
}

// dV = X_G^T Z for 64 retained columns per block; adds into v_out (which holds V0).
__global__ __launch_bounds__(256) void update_add_kernel(const float* x, const uint8_t* fixed,
                                                     const float* z, const float* stats_ws,
                                                     float* v_out, int c, int mp, int D) {
  extern __shared__ __attribute__((aligned(16))) float Xs[];  // [mp][68]
  constexpr int XS = 68;
  const int u = blockIdx.y, t0 = blockIdx.x * 64;
  if (stats_ws[u * 4 + 3] != 0.f) return;  // singular: keep V0
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const float* xu = x + (size_t)u * mp * c;
  const uint8_t* fu = fixed + (size_t)u * c;
  // X of the block's 64 slots to LDS, masked by the fixed flags; a thread
  // loads four elements and their flags before it stores them (slots past c
  // read slot c - 1, in bounds, and store zero).  mp is a multiple of 32, so
  // the mp x 64 elements are whole batches of 4 x 256.
  for (int e0 = tid; e0 < mp * 64; e0 += 4 * 256) {
    float xv[4];
    uint8_t fv[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int e = e0 + 256 * b, r = e / 64, t = min(t0 + e % 64, c - 1);
      xv[b] = xu[(size_t)r * c + t];
      fv[b] = fu[t];
    }
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int e = e0 + 256 * b, r = e / 64, tt = e % 64;
      Xs[r * XS + tt] = (t0 + tt < c && !fv[b]) ? xv[b] : 0.f;
    }
  }
  __syncthreads();
  const float* zu = z + (size_t)u * D * mp;
  f32x4 acc[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) acc[dt] = zero4();
  const int ndt = D / 16;
  for (int ks = 0; ks < mp / 32; ++ks) {
    float av[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) av[e] = Xs[(ks * 32 + 8 * g + e) * XS + wave * 16 + l16];
    bf16x8 ahi, alo;
    split8(av, ahi, alo);
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      if (dt >= ndt) break;
      const float* zr = zu + (size_t)(dt * 16 + l16) * mp + ks * 32 + 8 * g;
      float bv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) bv[e] = zr[e];
      bf16x8 bhi, blo;
      split8(bv, bhi, blo);
      acc[dt] = mfma_bf16(ahi, bhi, acc[dt]);
      acc[dt] = mfma_bf16(ahi, blo, acc[dt]);
      acc[dt] = mfma_bf16(alo, bhi, acc[dt]);
    }
  }
  // v_out += dV at the free slots: flags and old values loaded first (slots
  // past c read slot c - 1 and are not written)
  bool upd[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = t0 + wave * 16 + 4 * g + i;
    const uint8_t f = fu[min(t, c - 1)];
    upd[i] = t < c && !f;
  }
  float vo[8][4];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    if (dt >= ndt) break;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = min(t0 + wave * 16 + 4 * g + i, c - 1);
      vo[dt][i] = v_out[((size_t)u * c + t) * D + dt * 16 + l16];
    }
  }
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    if (dt >= ndt) break;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = t0 + wave * 16 + 4 * g + i;
      if (upd[i]) v_out[((size_t)u * c + t) * D + dt * 16 + l16] = vo[dt][i] + acc[dt][i];
    }
  }
}

// v_out = V0 + X_G^T Z for 256 retained slots per block (fixed slots, and
// every slot of a unit whose system was singular, get V0), from the stored X
// [mp][c] and Z^T.  Z^T goes to LDS once per block as bf16 hi/lo pairs, its
// row dd at (dd mod DT) * 16 + dd / DT (DT = D / 16 output tiles), which hands
// each lane DT consecutive output columns: V0 and v_out move in 16-byte
// pieces.  Each wave takes 32 slots (two 16-slot tiles); a lane reads the X
// values of its slot straight from global memory (8 rows of one column per
// MFMA step: across the 16 lanes of a row, 64 contiguous bytes), masked by the
// slot's fixed flag and split into bf16 hi/lo.  Products are three bf16 MFMAs
// (hi hi, hi lo, lo hi) with fp32 accumulation.
constexpr int kUpdGenWaves = 8;
constexpr int kUpdGenSlots = 32 * kUpdGenWaves;

template <typename T, int MP, int D>
__global__ __launch_bounds__(kUpdGenWaves * 64) void update_gen_kernel(
    const float* x, const uint8_t* fixed, const float* z, const float* stats_ws, const T* v0c,
    float* v_out, int m, int c) {
  constexpr int DT = D / 16;
  constexpr int ZS = MP + 8;   // LDS row stride (bf16) of Z^T rows
  constexpr int NTH = kUpdGenWaves * 64;
  __shared__ __attribute__((aligned(16))) u16 zh[D * ZS];
  __shared__ __attribute__((aligned(16))) u16 zl[D * ZS];
  const int u = blockIdx.y, t0 = blockIdx.x * kUpdGenSlots;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g = lane >> 4;
  const bool singular = stats_ws[u * 4 + 3] != 0.f;   // block-uniform
  const uint8_t* fu = fixed + (size_t)u * c;

  if (!singular) {
    // Z^T to bf16 hi/lo in LDS; a thread's loads of ZB elements are issued
    // before it converts them
    const float* zu = z + (size_t)u * D * MP;
    constexpr int ZE = D * (MP / 4), ZB = ZE / NTH < 8 ? ZE / NTH : 8;
    static_assert(ZB >= 1 && ZE % (ZB * NTH) == 0, "whole batches");
    for (int e0 = tid; e0 < ZE; e0 += ZB * NTH) {
      float4 zb[ZB];
#pragma unroll
      for (int b = 0; b < ZB; ++b) {
        const int e = e0 + b * NTH;
        zb[b] = *reinterpret_cast<const float4*>(zu + (size_t)(e / (MP / 4)) * MP + 4 * (e % (MP / 4)));
      }
#pragma unroll
      for (int b = 0; b < ZB; ++b) {
        const int e = e0 + b * NTH;
        const int dd = e / (MP / 4), r0 = 4 * (e % (MP / 4));
        const float4 v = zb[b];
        const float vv[4] = {v.x, v.y, v.z, v.w};
        u16 hh[4], ll[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const __bf16 h = (__bf16)vv[i];
          hh[i] = __builtin_bit_cast(u16, h);
          ll[i] = __builtin_bit_cast(u16, (__bf16)(vv[i] - (float)h));
        }
        const int row = (dd % DT) * 16 + dd / DT;
        *reinterpret_cast<uint2*>(zh + row * ZS + r0) =
            make_uint2(hh[0] | ((uint32_t)hh[1] << 16), hh[2] | ((uint32_t)hh[3] << 16));
        *reinterpret_cast<uint2*>(zl + row * ZS + r0) =
            make_uint2(ll[0] | ((uint32_t)ll[1] << 16), ll[2] | ((uint32_t)ll[3] << 16));
      }
    }
  }
  __syncthreads();

  const int tb = t0 + 32 * wave;   // this wave's first slot
  f32x4 acc[2][DT];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[tt][dt] = zero4();
  if (!singular && tb < c) {
    const float* xu = x + (size_t)u * MP * c;
    float keep[2];   // 1 for a free slot inside the retained set, else 0
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int t = tb + 16 * tt + l16;
      const uint8_t f = fu[min(t, c - 1)];   // in bounds, without a branch
      keep[tt] = (t < c && !f) ? 1.f : 0.f;
    }
#pragma unroll 1
    for (int r0 = 0; r0 < MP; r0 += 32) {
      // every row of X is read (rows past m are in bounds) and masked
      // afterwards, so the sixteen loads are in flight together
      float xl[2][8];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        const int t = min(tb + 16 * tt + l16, c - 1);
#pragma unroll
        for (int e = 0; e < 8; ++e) xl[tt][e] = xu[(size_t)(r0 + 8 * g + e) * c + t];
      }
      bf16x8 ah[2], al[2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        float xv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) xv[e] = r0 + 8 * g + e < m ? keep[tt] * xl[tt][e] : 0.f;
        split8(xv, ah[tt], al[tt]);
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int zo = (dt * 16 + l16) * ZS + r0 + 8 * g;
        const bf16x8 bh = as_bf16x8(*reinterpret_cast<const uint4*>(zh + zo));
        const bf16x8 bl = as_bf16x8(*reinterpret_cast<const uint4*>(zl + zo));
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          acc[tt][dt] = mfma_bf16(ah[tt], bh, acc[tt][dt]);
          acc[tt][dt] = mfma_bf16(ah[tt], bl, acc[tt][dt]);
          acc[tt][dt] = mfma_bf16(al[tt], bh, acc[tt][dt]);
        }
      }
    }
  }
  // lane holds dV[slot = tb + 16tt + 4g + i][dd = l16 * DT + dt]; V0 from the
  // compact copy, every slot of the block written.  The V0 rows and fixed
  // flags of all eight slots are loaded first (slots past c read slot c - 1,
  // in bounds, and are not written).
  T v0r[2][4][DT];
  uint8_t flr[2][4];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tc = min(tb + 16 * tt + 4 * g + i, c - 1);
      flr[tt][i] = fu[tc];
      const T* src = v0c + ((size_t)u * c + tc) * D + l16 * DT;
#pragma unroll
      for (int k = 0; k < DT; ++k) v0r[tt][i][k] = src[k];
    }
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = tb + 16 * tt + 4 * g + i;
      if (t >= c) continue;
      const bool upd = !singular && !flr[tt][i];
      float v[DT];
#pragma unroll
      for (int k = 0; k < DT; ++k) {
        if constexpr (sizeof(T) == 2) v[k] = bf16_to_f32(v0r[tt][i][k]);
        else v[k] = (float)v0r[tt][i][k];
      }
      if (upd) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) v[dt] += acc[tt][dt][i];
      }
      float* dst = v_out + ((size_t)u * c + t) * D + l16 * DT;
#pragma unroll
      for (int k = 0; k < DT / 4; ++k)
        *reinterpret_cast<float4*>(dst + 4 * k) = make_float4(v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]);
    }
}

template <typename T, int MP, int D>
hipError_t launch_update_gen_t(const Plan& p, const float* x, const uint8_t* fixed, const float* z,
                               const float* stats_ws, const void* v0c, float* v_out,
                               hipStream_t s) {
  const dim3 grid((p.c + kUpdGenSlots - 1) / kUpdGenSlots, p.U);
  hipLaunchKernelGGL((update_gen_kernel<T, MP, D>), grid, dim3(kUpdGenWaves * 64), 0, s, x, fixed,
                     z, stats_ws, (const T*)v0c, v_out, p.m, p.c);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_update_gen(const Plan& p, const float* x, const uint8_t* fixed, const float* z,
                             const float* stats_ws, const void* v0c, float* v_out, hipStream_t s) {
#define GRKV_UG(MPV, DV)                                                                      \
  if (p.mp == MPV && p.d == DV)                                                               \
    return p.dtype == GRKV_BF16                                                               \
               ? launch_update_gen_t<u16, MPV, DV>(p, x, fixed, z, stats_ws, v0c, v_out, s)   \
               : launch_update_gen_t<float, MPV, DV>(p, x, fixed, z, stats_ws, v0c, v_out, s);
  GRKV_UG(32, 64) GRKV_UG(32, 128) GRKV_UG(64, 64) GRKV_UG(64, 128) GRKV_UG(128, 64)
  GRKV_UG(128, 128) GRKV_UG(256, 64) GRKV_UG(256, 128)
#undef GRKV_UG
  return hipErrorInvalidValue;
}

static size_t chol_lds_bytes(int mp, int D, bool* w_in_lds) {
  size_t tri_f = ((size_t)mp * (mp + 1) / 2 + 3) & ~(size_t)3;
  size_t with_w = (tri_f + (size_t)mp * D) * sizeof(float);
  if (with_w <= 150 * 1024) { *w_in_lds = true; return with_w; }
  *w_in_lds = false;
  return tri_f * sizeof(float);
}

hipError_t launch_cholesky_solve(const Plan& p, const float* npart, const float* y,
                                 const float* resid, float* gram, float* z, float* stats_ws,
                                 float* stats_user, hipStream_t s) {
  bool w_in_lds;
  size_t lds = chol_lds_bytes(p.mp, p.d, &w_in_lds);
  hipError_t e = hipFuncSetAttribute((const void*)chol_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(chol_kernel, dim3(p.U), dim3(256), lds, s, npart, p.S3, y, resid, gram, z,
                     stats_ws, stats_user, p.m, p.mp, p.d, p.lam, w_in_lds ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_update_add(const Plan& p, const float* x, const uint8_t* fixed, const float* z,
                             const float* stats_ws, float* v_out, hipStream_t s) {
  size_t lds = (size_t)p.mp * 68 * sizeof(float);
  hipError_t e = hipFuncSetAttribute((const void*)update_add_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(update_add_kernel, dim3((p.c + 63) / 64, p.U), dim3(256), lds, s, x, fixed, z,
                     stats_ws, v_out, p.c, p.mp, p.d);
  return hipGetLastError();
}

}  // namespace grkv
