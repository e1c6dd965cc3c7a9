// Streamed window attention over a key set (the full cache, or the gathered
// retained keys) for all m stacked window rows of a unit at once.
//
// Pass A ("lse"): per split of the keys, the row maximum and the sum of
//   2^(t - max) of the log2-scaled logits t = q.k * log2(e)/sqrt(d), with the
//   causal window rule applied; the combine step turns the splits into the
//   log-sum-exp of every row.
// Pass B ("prob"): with the final log-sum-exp known, P = softmax(Q K^T/sqrt(d))
//   is formed tile by tile and three things are taken from it: the partial
//   attention output P V of the split (fp32, MFMA), the SnapKV column sums
//   s_j = sum_r P[r][j] of the prefix keys, and optionally P itself.
//
// Layout and work split: grid (splits, units); a block has one wave per 32
// rows.  Keys stream through LDS in tiles of 32 (K row-major, V transposed for
// the bf16 path), with the next tile's global loads in flight while the
// current tile is multiplied.  Logits are computed as S^T = K Q^T so that a
// lane ends up holding four consecutive keys of one row, which is both the
// operand layout P V needs and a layout where column sums are a 16-lane
// reduction.
#include <type_traits>

#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {

struct PassK {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* kpos;
  int U, m, mp, w;
  int64_t n;
  int causal;
  int nk, S, chunk;
  float scale_log2;
  float* pmax;
  double* psum;
  const float* lse_log2;
  float* ypart;
  float* colsum;
  int prefix;
  float* xout;
  int split_p;
};

template <bool BF, int D, int WAVES>
struct Cfg {
  using T = typename std::conditional<BF, u16, float>::type;
  static constexpr int kThreads = WAVES * 64;
  static constexpr int kElemsPerChunk = 16 / (int)sizeof(T);
  static constexpr int kChunksPerRow = D / kElemsPerChunk;
  static constexpr int kChunks = kKeyTile * kChunksPerRow;
  static constexpr int kPerThread = (kChunks + kThreads - 1) / kThreads;
  static constexpr int kKStride = BF ? D + 8 : D + 4;          // K tile row (elements)
  static constexpr int kVStride = BF ? kKeyTile + 4 : D + 4;   // V^T row (bf16) / V row (f32)
  static constexpr int kVRows = BF ? D : kKeyTile;
  static constexpr int kQFrags = BF ? D / 32 : D / 4;
};

// Global -> register staging of one key tile (K and optionally V).
template <bool BF, int D, int WAVES, bool WITH_V>
struct Stage {
  using C = Cfg<BF, D, WAVES>;
  uint4 kr[C::kPerThread];
  uint4 vr[WITH_V ? C::kPerThread : 1];
  int pos;

  __device__ __forceinline__ void load(const PassK& a, const char* kbase, const char* vbase,
                                       const int32_t* kposu, int tile0, int key_end) {
#pragma unroll
    for (int c = 0; c < C::kPerThread; ++c) {
      int chunk = threadIdx.x + c * C::kThreads;
      int key = chunk / C::kChunksPerRow, cc = chunk % C::kChunksPerRow;
      int gkey = tile0 + key;
      uint4 zk = make_uint4(0, 0, 0, 0), zv = zk;
      if (chunk < C::kChunks && gkey < key_end) {
        size_t off = ((size_t)gkey * D) * sizeof(typename C::T) + (size_t)cc * 16;
        zk = *reinterpret_cast<const uint4*>(kbase + off);
        if (WITH_V) zv = *reinterpret_cast<const uint4*>(vbase + off);
      }
      kr[c] = zk;
      if (WITH_V) vr[c] = zv;
    }
    pos = -1;
    if (threadIdx.x < kKeyTile) {
      int gkey = tile0 + threadIdx.x;
      if (gkey < key_end) pos = kposu ? kposu[gkey] : gkey;
    }
  }

  __device__ __forceinline__ void store(typename C::T* Ks, typename C::T* Vs, int* kp) const {
#pragma unroll
    for (int c = 0; c < C::kPerThread; ++c) {
      int chunk = threadIdx.x + c * C::kThreads;
      if (chunk < C::kChunks) {
        int key = chunk / C::kChunksPerRow, cc = chunk % C::kChunksPerRow;
        *reinterpret_cast<uint4*>(&Ks[key * C::kKStride + cc * C::kElemsPerChunk]) = kr[c];
        if (WITH_V) {
          if (BF) {
            const u16* e = reinterpret_cast<const u16*>(&vr[c]);
#pragma unroll
            for (int t = 0; t < 8; ++t)
              reinterpret_cast<u16*>(Vs)[(cc * 8 + t) * C::kVStride + key] = e[t];
          } else {
            *reinterpret_cast<uint4*>(&Vs[key * C::kVStride + cc * C::kElemsPerChunk]) = vr[c];
          }
        }
      }
    }
    if (threadIdx.x < kKeyTile) kp[threadIdx.x] = pos;
  }
};

// Loads this lane's query fragments (the B operand of S^T = K Q^T).
template <bool BF, int D, int WAVES>
__device__ __forceinline__ void load_q(const PassK& a, int u, int wave, int lane,
                                       uint4 (&qb)[2][D / 32], float (&qf)[2][D / 4]) {
  const int l16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    int row = wave * kRowsPerWave + rt * 16 + l16;
    if (BF) {
      const u16* q = reinterpret_cast<const u16*>(a.q) + ((size_t)u * a.m + row) * D;
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks)
        qb[rt][ks] = row < a.m ? *reinterpret_cast<const uint4*>(q + ks * 32 + 8 * g)
                               : make_uint4(0, 0, 0, 0);
    } else {
      const float* q = reinterpret_cast<const float*>(a.q) + ((size_t)u * a.m + row) * D;
#pragma unroll
      for (int ks = 0; ks < D / 4; ++ks) qf[rt][ks] = row < a.m ? q[ks * 4 + g] : 0.f;
    }
  }
}

// st[kt][rt][i] = q_row . k_key for key = kt*16 + 4*(lane/16) + i of the tile
// and row = rt*16 + lane%16 of the wave.
template <bool BF, int D, int WAVES>
__device__ __forceinline__ void logits_tile(const typename Cfg<BF, D, WAVES>::T* Ks, int lane,
                                            const uint4 (&qb)[2][D / 32],
                                            const float (&qf)[2][D / 4], f32x4 (&st)[2][2]) {
  using C = Cfg<BF, D, WAVES>;
  const int l16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) st[kt][rt] = zero4();
  if (BF) {
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        uint4 kv = *reinterpret_cast<const uint4*>(&Ks[(kt * 16 + l16) * C::kKStride + ks * 32 + 8 * g]);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
          st[kt][rt] = mfma_bf16(as_bf16x8(kv), as_bf16x8(qb[rt][ks]), st[kt][rt]);
      }
    }
  } else {
#pragma unroll
    for (int ks = 0; ks < D / 4; ++ks) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        float kv = reinterpret_cast<const float*>(Ks)[(kt * 16 + l16) * C::kKStride + ks * 4 + g];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) st[kt][rt] = mfma_f32(kv, qf[rt][ks], st[kt][rt]);
      }
    }
  }
}

template <bool BF, int D, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void lse_pass_kernel(PassK a) {
  using C = Cfg<BF, D, WAVES>;
  using T = typename C::T;
  __shared__ __attribute__((aligned(16))) T Ks[kKeyTile * C::kKStride];
  __shared__ int kp[kKeyTile];

  const int s = blockIdx.x, u = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int key0 = s * a.chunk;
  const int key_end = min(key0 + a.chunk, a.nk);
  const int ntiles = key_end > key0 ? (key_end - key0 + kKeyTile - 1) / kKeyTile : 0;
  const char* kbase = reinterpret_cast<const char*>(a.k) + (size_t)u * a.nk * D * sizeof(T);
  const int32_t* kposu = a.kpos ? a.kpos + (size_t)u * a.nk : nullptr;

  uint4 qb[2][D / 32];
  float qf[2][D / 4];
  load_q<BF, D, WAVES>(a, u, wave, lane, qb, qf);

  int rowpos[2];
  bool rowok[2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    int row = wave * kRowsPerWave + rt * 16 + l16;
    rowok[rt] = row < a.m;
    rowpos[rt] = a.causal ? (int)(a.n - a.w + (row % a.w)) : 0x7fffffff;
  }
  float mrun[2] = {-INFINITY, -INFINITY};
  double srun[2] = {0.0, 0.0};

  Stage<BF, D, WAVES, false> st_regs;
  if (ntiles > 0) st_regs.load(a, kbase, nullptr, kposu, key0, key_end);
  for (int t = 0; t < ntiles; ++t) {
    __syncthreads();
    st_regs.store(Ks, nullptr, kp);
    __syncthreads();
    if (t + 1 < ntiles) st_regs.load(a, kbase, nullptr, kposu, key0 + (t + 1) * kKeyTile, key_end);
    f32x4 st[2][2];
    logits_tile<BF, D, WAVES>(Ks, lane, qb, qf, st);
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      float tv[2][4];
      float tmax = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int pos = kp[kt * 16 + 4 * g + i];
          bool ok = rowok[rt] && pos >= 0 && pos <= rowpos[rt];
          tv[kt][i] = ok ? st[kt][rt][i] * a.scale_log2 : -INFINITY;
          tmax = fmaxf(tmax, tv[kt][i]);
        }
      tmax = max_over_groups(tmax);
      if (tmax == -INFINITY) continue;
      if (tmax > mrun[rt]) {
        if (mrun[rt] != -INFINITY) srun[rt] *= exp2((double)mrun[rt] - (double)tmax);
        mrun[rt] = tmax;
      }
      float acc = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc += exp2f(tv[kt][i] - mrun[rt]);
      srun[rt] += (double)acc;
    }
  }
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    double tot = sum_over_groups(srun[rt]);
    int row = wave * kRowsPerWave + rt * 16 + l16;
    if (g == 0) {
      size_t o = ((size_t)u * a.S + s) * a.mp + row;
      a.pmax[o] = mrun[rt];
      a.psum[o] = tot;
    }
  }
}

template <bool BF, int D, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void prob_pass_kernel(PassK a) {
  using C = Cfg<BF, D, WAVES>;
  using T = typename C::T;
  __shared__ __attribute__((aligned(16))) T Ks[kKeyTile * C::kKStride];
  __shared__ __attribute__((aligned(16))) T Vs[C::kVRows * C::kVStride];
  __shared__ int kp[kKeyTile];
  __shared__ float colpart[WAVES][kKeyTile];

  const int s = blockIdx.x, u = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int key0 = s * a.chunk;
  const int key_end = min(key0 + a.chunk, a.nk);
  const int ntiles = key_end > key0 ? (key_end - key0 + kKeyTile - 1) / kKeyTile : 0;
  const size_t ubytes = (size_t)u * a.nk * D * sizeof(T);
  const char* kbase = reinterpret_cast<const char*>(a.k) + ubytes;
  const char* vbase = reinterpret_cast<const char*>(a.v) + ubytes;
  const int32_t* kposu = a.kpos ? a.kpos + (size_t)u * a.nk : nullptr;

  uint4 qb[2][D / 32];
  float qf[2][D / 4];
  load_q<BF, D, WAVES>(a, u, wave, lane, qb, qf);

  int rowpos[2];
  bool rowok[2];
  float lse[2];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    int row = wave * kRowsPerWave + rt * 16 + l16;
    rowok[rt] = row < a.m;
    rowpos[rt] = a.causal ? (int)(a.n - a.w + (row % a.w)) : 0x7fffffff;
    lse[rt] = a.lse_log2[(size_t)u * a.mp + row];
  }

  f32x4 y[2][D / 16];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) y[rt][dt] = zero4();

  Stage<BF, D, WAVES, true> st_regs;
  if (ntiles > 0) st_regs.load(a, kbase, vbase, kposu, key0, key_end);
  for (int t = 0; t < ntiles; ++t) {
    const int tile0 = key0 + t * kKeyTile;
    __syncthreads();
    st_regs.store(Ks, Vs, kp);
    __syncthreads();
    if (t + 1 < ntiles) st_regs.load(a, kbase, vbase, kposu, tile0 + kKeyTile, key_end);
    f32x4 st[2][2];
    logits_tile<BF, D, WAVES>(Ks, lane, qb, qf, st);

    float pv[2][2][4];  // [kt][rt][i]
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int pos = kp[kt * 16 + 4 * g + i];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          bool ok = rowok[rt] && pos >= 0 && pos <= rowpos[rt];
          pv[kt][rt][i] = ok ? exp2f(fmaf(st[kt][rt][i], a.scale_log2, -lse[rt])) : 0.f;
        }
      }

    if (a.colsum) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float c = sum16(pv[kt][0][i] + pv[kt][1][i]);
          if (l16 == 0) colpart[wave][kt * 16 + 4 * g + i] = c;
        }
      __syncthreads();
      if (threadIdx.x < kKeyTile) {
        int key = tile0 + threadIdx.x;
        if (key < key_end && key < a.prefix) {
          float c = 0.f;
#pragma unroll
          for (int wv = 0; wv < WAVES; ++wv) c += colpart[wv][threadIdx.x];
          a.colsum[(size_t)u * a.prefix + key] = c;
        }
      }
    }
    if (a.xout) {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        int row = wave * kRowsPerWave + rt * 16 + l16;
        float* xr = a.xout + ((size_t)u * a.mp + row) * a.nk;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            int key = tile0 + kt * 16 + 4 * g + i;
            if (key < key_end) xr[key] = pv[kt][rt][i];
          }
      }
    }

    if (BF) {
      bf16x8 ahi[2], alo[2];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        float x8[8] = {pv[0][rt][0], pv[0][rt][1], pv[0][rt][2], pv[0][rt][3],
                       pv[1][rt][0], pv[1][rt][1], pv[1][rt][2], pv[1][rt][3]};
        split8(x8, ahi[rt], alo[rt]);
      }
      const u16* Vt = reinterpret_cast<const u16*>(Vs);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const u16* vr = Vt + (dt * 16 + l16) * C::kVStride;
        uint2 v0 = *reinterpret_cast<const uint2*>(vr + 4 * g);
        uint2 v1 = *reinterpret_cast<const uint2*>(vr + 16 + 4 * g);
        bf16x8 b = as_bf16x8(make_uint4(v0.x, v0.y, v1.x, v1.y));
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
          y[rt][dt] = mfma_bf16(ahi[rt], b, y[rt][dt]);
          if (a.split_p) y[rt][dt] = mfma_bf16(alo[rt], b, y[rt][dt]);
        }
      }
    } else {
      const float* Vf = reinterpret_cast<const float*>(Vs);
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt) {
            float b = Vf[(kt * 16 + 4 * g + i) * C::kVStride + dt * 16 + l16];
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) y[rt][dt] = mfma_f32(pv[kt][rt][i], b, y[rt][dt]);
          }
    }
  }

  float* yp = a.ypart + ((size_t)u * a.S + s) * a.mp * D;
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int row = wave * kRowsPerWave + rt * 16 + 4 * g + i;
        yp[(size_t)row * D + dt * 16 + l16] = y[rt][dt][i];
      }
}

// The partials of a row are loaded kBatch at a time (all in flight), then
// reduced in split order, so the result does not depend on the batching.
constexpr int kCombineBatch = 16;

// Log-sum-exp of split partials (max, sum of 2^(t - max)): one thread per
// (row, split class s mod kLseLanes), which sums its splits against a running
// maximum with all loads of a batch in flight; the classes of a row sit in
// adjacent lanes and merge by shuffles.  Fixed order, so deterministic.
constexpr int kLseLanes = 8;

__device__ __forceinline__ double lse_rescale(double sum, float from, float to) {
  return from == -INFINITY ? 0.0 : sum * exp2((double)from - (double)to);
}

__global__ __launch_bounds__(256) void lse_combine_kernel(const float* pmax, const double* psum,
                                                          int S, int mp, int total, double* lse,
                                                          float* lse_log2) {
  const int gid = blockIdx.x * blockDim.x + threadIdx.x;
  const int id = gid / kLseLanes, c = gid % kLseLanes;
  const bool live = id < total;
  const int u = live ? id / mp : 0, row = live ? id % mp : 0;
  const size_t base = (size_t)u * S * mp + row;
  float M = -INFINITY;
  double sum = 0.0;
  if (live) {
    for (int s0 = c; s0 < S; s0 += kLseLanes * kCombineBatch) {
      float ms[kCombineBatch];
      double ps[kCombineBatch];
#pragma unroll
      for (int k = 0; k < kCombineBatch; ++k) {
        const int sp = s0 + k * kLseLanes;
        const bool in = sp < S;
        ms[k] = in ? pmax[base + (size_t)sp * mp] : -INFINITY;
        ps[k] = in ? psum[base + (size_t)sp * mp] : 0.0;
      }
      float bm = M;
#pragma unroll
      for (int k = 0; k < kCombineBatch; ++k) bm = fmaxf(bm, ms[k]);
      if (bm == -INFINITY) continue;
      sum = lse_rescale(sum, M, bm);
#pragma unroll
      for (int k = 0; k < kCombineBatch; ++k)
        if (ms[k] != -INFINITY) sum += ps[k] * exp2((double)ms[k] - (double)bm);
      M = bm;
    }
  }
#pragma unroll
  for (int off = 1; off < kLseLanes; off <<= 1) {
    const float Mo = __shfl_xor(M, off);
    const double so = __shfl_xor(sum, off);
    const float Mn = fmaxf(M, Mo);
    sum = lse_rescale(sum, M, Mn) + lse_rescale(so, Mo, Mn);
    M = Mn;
  }
  if (!live || c != 0) return;
  if (M == -INFINITY) {  // padding row: no visible key
    lse[id] = -INFINITY;
    lse_log2[id] = 0.f;
    return;
  }
  const double l2 = (double)M + log2(sum);
  lse[id] = l2 * 0.69314718055994530942;
  lse_log2[id] = (float)l2;
}

__global__ void combine_rows_kernel(const float* part, int S, size_t per_unit, size_t total,
                                    const float* base, float* out) {
  size_t id = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= total) return;
  size_t u = id / per_unit, e = id % per_unit;
  const float* p0 = part + u * S * per_unit + e;
  float acc = 0.f;
  for (int s0 = 0; s0 < S; s0 += kCombineBatch) {
    float v[kCombineBatch];
#pragma unroll
    for (int k = 0; k < kCombineBatch; ++k) v[k] = s0 + k < S ? p0[(size_t)(s0 + k) * per_unit] : 0.f;
#pragma unroll
    for (int k = 0; k < kCombineBatch; ++k)
      if (s0 + k < S) acc += v[k];
  }
  out[id] = base ? base[id] - acc : acc;
}

// Up to four partial arrays summed over their splits in one launch: segment
// i covers U * per_unit[i] consecutive ids, each summing S[i] splits.
struct CombineSeg {
  const float* part[kCombineSegs];
  float* out[kCombineSegs];
  size_t per_unit[kCombineSegs];
  int S[kCombineSegs];
};

__global__ void combine_segments_kernel(CombineSeg g, int U, size_t total) {
  size_t id = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (id >= total) return;
  int i = 0;
  while (i < kCombineSegs - 1 && id >= (size_t)U * g.per_unit[i]) {
    id -= (size_t)U * g.per_unit[i];
    ++i;
  }
  const size_t pu = g.per_unit[i], u = id / pu, e = id % pu;
  const int S = g.S[i];
  const float* p0 = g.part[i] + u * S * pu + e;
  float acc = 0.f;
  for (int s0 = 0; s0 < S; s0 += kCombineBatch) {
    float v[kCombineBatch];
#pragma unroll
    for (int k = 0; k < kCombineBatch; ++k) v[k] = s0 + k < S ? p0[(size_t)(s0 + k) * pu] : 0.f;
#pragma unroll
    for (int k = 0; k < kCombineBatch; ++k)
      if (s0 + k < S) acc += v[k];
  }
  g.out[i][id] = acc;
}

template <bool BF, int D, int WAVES>
hipError_t launch_pass(const Plan& p, const AttnPass& a, hipStream_t s, bool pass_b) {
  PassK k;
  k.q = a.q; k.k = a.k; k.v = a.v; k.kpos = a.kpos;
  k.U = p.U; k.m = p.m; k.mp = p.mp; k.w = p.w; k.n = p.n;
  k.causal = p.opt.causal_window ? 1 : 0;
  k.nk = a.nk; k.S = a.S; k.chunk = a.chunk;
  k.scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  k.pmax = a.pmax; k.psum = a.psum; k.lse_log2 = a.lse_log2;
  k.ypart = a.ypart; k.colsum = a.colsum; k.prefix = a.prefix; k.xout = a.xout;
  k.split_p = a.split_p ? 1 : 0;
  dim3 grid(a.S, p.U), block(WAVES * 64);
  if (pass_b)
    hipLaunchKernelGGL((prob_pass_kernel<BF, D, WAVES>), grid, block, 0, s, k);
  else
    hipLaunchKernelGGL((lse_pass_kernel<BF, D, WAVES>), grid, block, 0, s, k);
  return hipGetLastError();
}

template <bool BF, int D>
hipError_t dispatch_waves(const Plan& p, const AttnPass& a, hipStream_t s, bool pass_b) {
  switch (p.waves) {
    case 1: return launch_pass<BF, D, 1>(p, a, s, pass_b);
    case 2: return launch_pass<BF, D, 2>(p, a, s, pass_b);
    case 3: return launch_pass<BF, D, 3>(p, a, s, pass_b);
    case 4: return launch_pass<BF, D, 4>(p, a, s, pass_b);
    case 5: return launch_pass<BF, D, 5>(p, a, s, pass_b);
    case 6: return launch_pass<BF, D, 6>(p, a, s, pass_b);
    case 7: return launch_pass<BF, D, 7>(p, a, s, pass_b);
    case 8: return launch_pass<BF, D, 8>(p, a, s, pass_b);
  }
  return hipErrorInvalidValue;
}

hipError_t dispatch(const Plan& p, const AttnPass& a, hipStream_t s, bool pass_b) {
  bool bf = p.dtype == GRKV_BF16;
  if (bf && p.d == 128) return dispatch_waves<true, 128>(p, a, s, pass_b);
  if (bf && p.d == 64) return dispatch_waves<true, 64>(p, a, s, pass_b);
  if (!bf && p.d == 128) return dispatch_waves<false, 128>(p, a, s, pass_b);
  if (!bf && p.d == 64) return dispatch_waves<false, 64>(p, a, s, pass_b);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_lse_pass(const Plan& p, const AttnPass& a, hipStream_t s) {
  return dispatch(p, a, s, false);
}

hipError_t launch_prob_pass(const Plan& p, const AttnPass& a, hipStream_t s) {
  return dispatch(p, a, s, true);
}

hipError_t launch_lse_combine(const Plan& p, const float* pmax, const double* psum, int S,
                              double* lse, float* lse_log2, hipStream_t s) {
  const int total = p.U * p.mp;
  const int threads = total * kLseLanes;
  hipLaunchKernelGGL(lse_combine_kernel, dim3((threads + 255) / 256), dim3(256), 0, s, pmax, psum,
                     S, p.mp, total, lse, lse_log2);
  return hipGetLastError();
}

hipError_t launch_combine_rows(const Plan& p, const float* part, int S, const float* base,
                               float* out, hipStream_t s) {
  size_t per_unit = (size_t)p.mp * p.d, total = per_unit * p.U;
  hipLaunchKernelGGL(combine_rows_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                     part, S, per_unit, total, base, out);
  return hipGetLastError();
}

hipError_t launch_combine_parts(int U, const int S[kCombineSegs],
                                const float* const part[kCombineSegs],
                                float* const out[kCombineSegs],
                                const size_t per_unit[kCombineSegs], hipStream_t s) {
  CombineSeg g;
  size_t total = 0;
  for (int i = 0; i < kCombineSegs; ++i) {
    g.part[i] = part[i];
    g.out[i] = out[i];
    g.per_unit[i] = per_unit[i];
    g.S[i] = S[i];
    total += (size_t)U * per_unit[i];
  }
  hipLaunchKernelGGL(combine_segments_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                     g, U, total);
  return hipGetLastError();
}

}  // namespace grkv
