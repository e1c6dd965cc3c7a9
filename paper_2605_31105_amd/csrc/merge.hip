// Value step of the ridge merge in its Woodbury dual form (Eq. 8; Algorithm 1,
// value step; App. D.1, fixed tokens App. D.3):
//   N = X_G X_G^T + lambda I_m   (gram: partial sums over column splits)
//   Z = N^-1 R                   (solve: elimination in registers and LDS)
//   V*_G = V0_G + X_G^T Z        (update: fixed columns keep V0)
// On this fast path the Gram partials come from the retained-cache pass
// (stream.hip); the gram kernel here serves the generic path.
// X_G is X with the fixed columns zeroed.  The fp32 operands of the two
// products go through the bf16 MFMA as hi+lo pairs (three products per tile),
// which keeps about 16 significant bits per term; accumulation is fp32.
#include "grkv_device.h"
#include "grkv_internal.h"

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
        const float xv = (t + q < t1 && !fu[t + q]) ? v[q] : 0.f;
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
// One block per unit solves N Z = R for the d right-hand sides by Gaussian
// elimination without pivoting (N is symmetric positive definite for
// lambda > 0) followed by back substitution, in fp32.
// Thread (rb, j) holds rows 32rb..32rb+31 of column j of the augmented matrix
// [N | R] in registers (j < MP: N, j >= MP: right-hand side j - MP).  The
// elimination step for pivot k publishes row k in LDS; since the trailing
// block stays symmetric, the multipliers of the rows below k are that row's
// own entries, A[i][k] = A[k][i].  The finished rows of U are kept in LDS,
// transposed, for the back substitution.
template <int MP, int D>
__global__ __launch_bounds__(MP / 32 * 256) void solve_kernel(
    const float* npart, int S3, const float* y, const float* resid, float* gram, float* z,
    u16* zhi, u16* zlo, float* stats_ws, float* stats_user, int m, float lam) {
  constexpr int RB = MP / 32;
  constexpr int NC = MP + D;              // augmented columns (<= 256)
  constexpr int US = MP + 4;              // Ucol row stride
  __shared__ __attribute__((aligned(16))) float rowk[2][256];
  __shared__ __attribute__((aligned(16))) float ucol[MP * US];   // ucol[k][i] = U[i][k]
  __shared__ float zk[2][256];
  __shared__ int fail;
  __shared__ double red[3][RB * 4];

  const int u = blockIdx.x, tid = threadIdx.x;
  const int rb = tid >> 8, j = tid & 255;
  const bool active = j < NC;
  const bool rhs = j >= MP && active;
  const int r0 = rb * 32;
  float a[32];

  if (tid == 0) fail = 0;
  // load: column j < MP is row j of the symmetric N; j >= MP is column j-MP of R
  const float* np = npart + (size_t)u * S3 * MP * MP;
  const float* ru = resid + (size_t)u * MP * D;
  if (j < MP) {
#pragma unroll
    for (int ii = 0; ii < 32; ++ii) a[ii] = 0.f;
    for (int s = 0; s < S3; ++s) {
      const float4* src = reinterpret_cast<const float4*>(np + (size_t)s * MP * MP + (size_t)j * MP + r0);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        float4 v = src[q];
        a[4 * q] += v.x; a[4 * q + 1] += v.y; a[4 * q + 2] += v.z; a[4 * q + 3] += v.w;
      }
    }
#pragma unroll
    for (int ii = 0; ii < 32; ++ii)
      if (r0 + ii == j) a[ii] += (j < m) ? lam : 1.f;
    float* gu = gram + (size_t)u * MP * MP + (size_t)j * MP + r0;
#pragma unroll
    for (int ii = 0; ii < 32; ++ii) gu[ii] = a[ii];
  } else if (rhs) {
#pragma unroll
    for (int ii = 0; ii < 32; ++ii) a[ii] = ru[(size_t)(r0 + ii) * D + (j - MP)];
  } else {
#pragma unroll
    for (int ii = 0; ii < 32; ++ii) a[ii] = 0.f;
  }

  // forward elimination
  for (int pb = 0; pb < RB; ++pb) {
#pragma unroll
    for (int kk = 0; kk < 32; ++kk) {
      const int k = pb * 32 + kk;
      float* rk = rowk[kk & 1];
      if (rb == pb && active) {
        rk[j] = a[kk];
        if (j < MP) ucol[j * US + k] = a[kk];   // U[k][j], stored transposed
      }
      __syncthreads();
      const float pk = rk[k];
      if (tid == 0 && !(pk > 0.f && isfinite(pk))) fail = 1;
      if (active && rb >= pb) {
        const float f = rk[j] * __builtin_amdgcn_rcpf(pk);
        if (rb > pb) {
#pragma unroll
          for (int ii = 0; ii < 32; ++ii) a[ii] -= rk[r0 + ii] * f;
        } else {
#pragma unroll
          for (int ii = kk + 1; ii < 32; ++ii) a[ii] -= rk[r0 + ii] * f;
        }
      }
    }
  }
  __syncthreads();
  const bool ok = fail == 0;

  // back substitution: z[k] = w[k] / U[k][k], then w[i] -= U[i][k] z[k] for i < k
  for (int pb = RB - 1; pb >= 0; --pb) {
#pragma unroll
    for (int kk = 31; kk >= 0; --kk) {
      const int k = pb * 32 + kk;
      float* zb = zk[kk & 1];
      if (rb == pb && rhs) {
        const float zv = a[kk] * __builtin_amdgcn_rcpf(ucol[k * US + k]);
        a[kk] = zv;
        zb[j] = zv;
      }
      __syncthreads();
      if (rhs && rb <= pb) {
        const float zv = zb[j];
        const float* uc = ucol + k * US + r0;
        if (rb < pb) {
#pragma unroll
          for (int ii = 0; ii < 32; ++ii) a[ii] -= uc[ii] * zv;
        } else {
#pragma unroll
          for (int ii = 0; ii < kk; ++ii) a[ii] -= uc[ii] * zv;
        }
      }
    }
  }

  // outputs: Z^T in fp32 and as bf16 hi/lo pairs (the update's MFMA operand)
  double sz = 0.0;
  if (rhs) {
    const int dd = j - MP;
    float* zr = z + ((size_t)u * D + dd) * MP + r0;
    u16* hr = zhi + ((size_t)u * D + dd) * MP + r0;
    u16* lr = zlo + ((size_t)u * D + dd) * MP + r0;
#pragma unroll
    for (int ii = 0; ii < 32; ++ii) {
      const float zv = ok ? a[ii] : 0.f;
      zr[ii] = zv;
      const __bf16 h = (__bf16)zv;
      hr[ii] = __builtin_bit_cast(u16, h);
      lr[ii] = __builtin_bit_cast(u16, (__bf16)(zv - (float)h));
      if (r0 + ii < m) sz += (double)zv * zv;
    }
  }
  // ||Y||^2 and ||R||^2 over the m real rows
  const float* yu = y + (size_t)u * MP * D;
  double sy = 0.0, sr = 0.0;
  for (int e = tid; e < m * D; e += blockDim.x) {
    const double yv = yu[e], rv = ru[e];
    sy += yv * yv;
    sr += rv * rv;
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
    for (int k = 0; k < RB * 4; ++k) { Y2 += red[0][k]; R2 += red[1][k]; Z2 += red[2][k]; }
    const double dn = Y2 > 0 ? Y2 : 1.0;
    const double dbefore = R2 / dn;
    const double dafter = ok ? (double)lam * lam * Z2 / dn : dbefore;
    const float st[4] = {(float)Y2, (float)dbefore, (float)dafter, ok ? 0.f : (float)GRKV_UNIT_SINGULAR};
    for (int k = 0; k < 4; ++k) {
      stats_ws[u * 4 + k] = st[k];
      if (stats_user) stats_user[u * 4 + k] = st[k];
    }
  }
}

// ---------------------------------------------------------------- update ----
// v_out = V0 + X_G^T Z for 512 retained slots per block (fixed slots, and every
// slot of a unit whose system was singular, get V0).  X is recomputed from the
// window queries, K0 and the retained-set log-sum-exp rather than stored:
// S = Q K0^T on the MFMA leaves each lane holding eight rows (two groups of
// four) of one key's column, which is exactly the A operand of X_G^T Z with
// the rows as the contraction index; Z^T arrives as bf16 hi/lo from the solve.
// Q and Z^T are staged in LDS once per block.
constexpr int kUpdWaves = 8;          // waves per update block
constexpr int kUpdSlots = 512;        // retained slots per update block

template <int MP, int D>
__global__ __launch_bounds__(kUpdWaves * 64) void update_kernel(
    const u16* q, const u16* k0, const float* lse_log2, const uint8_t* fixed, const u16* zhi,
    const u16* zlo, const float* stats_ws, const u16* v0c, float* v_out, int m, int w, int c,
    int causal, float scale_log2) {
  constexpr int QS = D + 8;    // LDS row stride (bf16) of Q rows
  constexpr int ZS = MP + 8;   // LDS row stride (bf16) of Z^T rows
  constexpr int NTH = kUpdWaves * 64;
  extern __shared__ __attribute__((aligned(16))) u16 sm[];
  u16* qs = sm;                  // [MP][QS]
  u16* zh = qs + MP * QS;        // [D][ZS]
  u16* zl = zh + D * ZS;         // [D][ZS]
  const int u = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g = lane >> 4;
  const bool singular = stats_ws[u * 4 + 3] != 0.f;
  const uint8_t* fu = fixed + (size_t)u * c;
  const int win0 = c - w;   // first window slot of the retained set
  const int slot0 = blockIdx.x * kUpdSlots;

  if (!singular) {
    const u16* qu = q + (size_t)u * m * D;
    for (int e = tid; e < MP * (D / 8); e += NTH) {
      const int r = e / (D / 8), ch = e % (D / 8);
      const uint4 v = r < m ? *reinterpret_cast<const uint4*>(qu + (size_t)r * D + ch * 8)
                            : make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4*>(qs + r * QS + ch * 8) = v;
    }
    const u16* zhu = zhi + (size_t)u * D * MP;
    const u16* zlu = zlo + (size_t)u * D * MP;
    for (int e = tid; e < D * (MP / 8); e += NTH) {
      const int r = e / (MP / 8), ch = e % (MP / 8);
      *reinterpret_cast<uint4*>(zh + r * ZS + ch * 8) =
          *reinterpret_cast<const uint4*>(zhu + (size_t)r * MP + ch * 8);
      *reinterpret_cast<uint4*>(zl + r * ZS + ch * 8) =
          *reinterpret_cast<const uint4*>(zlu + (size_t)r * MP + ch * 8);
    }
    __syncthreads();
  }
  float lse[MP / 16][4];
  bool rowok[MP / 16][4];
  int rowwin[MP / 16][4];
#pragma unroll
  for (int rt = 0; rt < MP / 16; ++rt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = rt * 16 + 4 * g + i;
      lse[rt][i] = lse_log2[(size_t)u * MP + row];
      rowok[rt][i] = row < m;
      rowwin[rt][i] = causal ? row % w : 0x3fffffff;
    }

  // this wave's 16-slot tiles: slot0 + 16 * (wave + kUpdWaves * j)
  constexpr int TILES = kUpdSlots / 16 / kUpdWaves;
  auto kload = [&](int tb, uint4 (&kb)[D / 32]) {
    const int t = tb + l16;
    const u16* kr = k0 + ((size_t)u * c + (t < c ? t : c - 1)) * D;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) kb[ks] = *reinterpret_cast<const uint4*>(kr + ks * 32 + 8 * g);
  };
  uint4 kb[D / 32], kn[D / 32];
  int tb = slot0 + 16 * wave;
  if (!singular && tb < c) kload(tb, kn);
  for (int j = 0; j < TILES; ++j, tb += 16 * kUpdWaves) {
    if (tb >= c) break;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) kb[ks] = kn[ks];
    if (!singular && j + 1 < TILES && tb + 16 * kUpdWaves < c) kload(tb + 16 * kUpdWaves, kn);
    const int t = tb + l16;   // the slot whose column this lane holds
    f32x4 acc[D / 16];
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) acc[dt] = zero4();
    const bool free_slot = t < c && !fu[t];
    if (!singular) {
      const int tw = t - win0;   // window index of slot t (< 0 outside the window)
#pragma unroll
      for (int rp = 0; rp < MP / 32; ++rp) {
        float x8[8];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int rt = 2 * rp + h;
          f32x4 st = zero4();
#pragma unroll
          for (int ks = 0; ks < D / 32; ++ks) {
            const bf16x8 qa = as_bf16x8(*reinterpret_cast<const uint4*>(qs + (rt * 16 + l16) * QS + ks * 32 + 8 * g));
            st = mfma_bf16(qa, as_bf16x8(kb[ks]), st);
          }
          // st[i] = q_row . k_t for row = 16rt + 4g + i
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool ok = free_slot && rowok[rt][i] && tw <= rowwin[rt][i];
            x8[4 * h + i] = ok ? __builtin_amdgcn_exp2f(fmaf(st[i], scale_log2, -lse[rt][i])) : 0.f;
          }
        }
        bf16x8 ah, al;
        split8(x8, ah, al);
        // Z rows {32rp + 4g + i, 32rp + 16 + 4g + i}, column dd = 16dt + l16
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) {
          const u16* zr = zh + (dt * 16 + l16) * ZS + 32 * rp + 4 * g;
          const u16* zr2 = zl + (dt * 16 + l16) * ZS + 32 * rp + 4 * g;
          const uint2 h0 = *reinterpret_cast<const uint2*>(zr);
          const uint2 h1 = *reinterpret_cast<const uint2*>(zr + 16);
          const uint2 l0 = *reinterpret_cast<const uint2*>(zr2);
          const uint2 l1 = *reinterpret_cast<const uint2*>(zr2 + 16);
          const bf16x8 bh = as_bf16x8(make_uint4(h0.x, h0.y, h1.x, h1.y));
          const bf16x8 bl = as_bf16x8(make_uint4(l0.x, l0.y, l1.x, l1.y));
          acc[dt] = mfma_bf16(ah, bh, acc[dt]);
          acc[dt] = mfma_bf16(ah, bl, acc[dt]);
          acc[dt] = mfma_bf16(al, bh, acc[dt]);
        }
      }
    }
    // lane holds dV[slot = tb + 4g + i][dd = 16dt + l16]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ts = tb + 4 * g + i;
      if (ts >= c) continue;
      const bool upd = !singular && !fu[ts];
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const size_t o = ((size_t)u * c + ts) * D + dt * 16 + l16;
        const float v0 = bf16_to_f32(v0c[o]);
        v_out[o] = upd ? v0 + acc[dt][i] : v0;
      }
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
hipError_t launch_solve_t(const Plan& p, const float* npart, const float* y, const float* resid,
                          float* gram, float* z, u16* zhi, u16* zlo, float* stats_ws,
                          float* stats_user, hipStream_t s) {
  hipLaunchKernelGGL((solve_kernel<MP, D>), dim3(p.U), dim3(MP / 32 * 256), 0, s, npart, p.S3, y,
                     resid, gram, z, zhi, zlo, stats_ws, stats_user, p.m, p.lam);
  return hipGetLastError();
}

template <int MP, int D>
hipError_t launch_update_t(const Plan& p, const void* q, const void* k0, const float* lse_log2,
                           const uint8_t* fixed, const u16* zhi, const u16* zlo,
                           const float* stats_ws, const u16* v0c, float* v_out, hipStream_t s) {
  const size_t lds = ((size_t)MP * (D + 8) + 2 * (size_t)D * (MP + 8)) * sizeof(u16);
  hipError_t e = hipFuncSetAttribute((const void*)update_kernel<MP, D>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const float scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  hipLaunchKernelGGL((update_kernel<MP, D>), dim3((p.c + kUpdSlots - 1) / kUpdSlots, p.U),
                     dim3(kUpdWaves * 64), lds, s,
                     (const u16*)q, (const u16*)k0, lse_log2, fixed, zhi, zlo, stats_ws, v0c,
                     v_out, p.m, p.w, p.c, p.opt.causal_window ? 1 : 0, scale_log2);
  return hipGetLastError();
}

}  // namespace

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

hipError_t launch_solve(const Plan& p, const float* npart, const float* y, const float* resid,
                        float* gram, float* z, u16* zhi, u16* zlo, float* stats_ws,
                        float* stats_user, hipStream_t s) {
#define GRKV_SOLVE(MPV, DV)                                                                   \
  if (p.mp == MPV && p.d == DV)                                                               \
    return launch_solve_t<MPV, DV>(p, npart, y, resid, gram, z, zhi, zlo, stats_ws, stats_user, s);
  GRKV_SOLVE(32, 64) GRKV_SOLVE(32, 128) GRKV_SOLVE(64, 64) GRKV_SOLVE(64, 128)
  GRKV_SOLVE(128, 64) GRKV_SOLVE(128, 128)
#undef GRKV_SOLVE
  return hipErrorInvalidValue;
}

hipError_t launch_update(const Plan& p, const void* q, const void* k0, const float* lse_log2,
                         const uint8_t* fixed, const u16* zhi, const u16* zlo,
                         const float* stats_ws, const u16* v0c, float* v_out, hipStream_t s) {
#define GRKV_UPD(MPV, DV)                                                                     \
  if (p.mp == MPV && p.d == DV)                                                               \
    return launch_update_t<MPV, DV>(p, q, k0, lse_log2, fixed, zhi, zlo, stats_ws, v0c, v_out, s);
  GRKV_UPD(32, 64) GRKV_UPD(32, 128) GRKV_UPD(64, 64) GRKV_UPD(64, 128)
  GRKV_UPD(128, 64) GRKV_UPD(128, 128)
#undef GRKV_UPD
  return hipErrorInvalidValue;
}

}  // namespace grkv
