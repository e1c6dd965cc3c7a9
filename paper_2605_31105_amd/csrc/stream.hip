// bf16 streaming window attention for gfx950 (pass A: log-sum-exp partials,
// pass B: P.V partials, SnapKV column sums, optional P).  Same contract as the
// generic kernels in attention.hip, built for bandwidth:
//
//  * K and V tiles go from HBM straight into an LDS ring (global_load_lds,
//    16 bytes per lane, no register staging).  Each ring stage is its own
//    LDS array and the tile loop is unrolled by the ring depth, so every
//    access names its stage at compile time; the compiler can then see that
//    the loads refilling one stage do not alias the stage being read and does
//    not stall on them.  NSTAGE-1 tiles stay in flight per block.
//  * A tile is 4096 elements per tensor (32 keys of d=128, 64 keys of d=64),
//    row-major with the 16-byte chunks of row r XOR-swizzled by r, which keeps
//    the MFMA operand reads of K free of bank conflicts.
//  * Pass B's P.V takes fp16 P times the V tile converted to fp16 in LDS (one
//    MFMA); a split whose V leaves the fp16 range is flagged and recomputed
//    by the exact mode with P as a bf16 hi+lo pair (two MFMAs, about 16 bits
//    of P), which the retained pass also uses.
//  * The P.V B-operand (four consecutive keys of one d column per lane) is
//    read from the row-major V tile with the LDS transpose read
//    ds_read_b64_tr_b16: within a 16-lane group, lane 4e+q supplies the
//    address of key row e, columns 4q..4q+3, and lane i receives column i of
//    the four rows.
//  * Pass A keeps a reference exponent and a sum per lane (its own keys of its
//    row) and merges the four lanes of a row once at the end; pass B's column
//    sums are one DPP reduce-scatter within 16-lane rows.  Neither touches the
//    LDS for reductions inside the tile loop except one 32-float exchange per
//    tile for column sums.
//  * Window positions are the last w key slots of both key sets (the full
//    cache, and the retained set whose last w entries are the window), so the
//    causal rule needs no position array.
//  * Pass B combines pass A's split partials into the log-sum-exp in its
//    prologue, or reads it combined already (calls with many splits per unit).
//  * With ragged budgets the retained pass runs as one flat grid: a per-unit
//    table gives each block its unit, split and first slot, and its partials
//    are indexed by the flat split.
#include "grkv_device.h"
#include "grkv_internal.h"

namespace grkv {
namespace {


struct StreamK {
  const u16* q;
  const u16* k;
  const u16* v;
  int m, mp, w;
  int causal;
  int nk, S, chunk;
  float scale_log2;
  float* pmax;
  double* psum;
  const float* lse_log2;
  // full-cache pass B: the log-sum-exp is combined here from pass A's split
  // partials (pmax, psum); blocks of split 0 write it to lse_out (natural,
  // fp64) and lse_log2_out (log2 domain, fp32) for the later kernels
  double* lse_out;
  float* lse_log2_out;
  int lse_ready;          // full-cache pass B: read the combined LSE from lse_log2_out
  float* ypart;
  float* colsum;
  int prefix;
  const uint8_t* fixed;   // retained pass: fixed flag per retained slot
  float* npart;           // retained pass: Gram partials [U][S][mp][mp]
  float* mpart;           // retained pass: row sums of P [U][S][mp]
  float lse_bias;         // pass B: P = 2^(t - (lse_log2 - lse_bias))
  int* redo;              // full-cache pass B: per-split flag [U][S] (see the modes)
  // retained passes: rows of K (gather_k) and/or V (gather_v) are read
  // through kpos [U][nk] from tensors of src_rows rows per unit
  const int32_t* kpos;
  int64_t src_rows;
  int gather_k, gather_v;
  u16* kcopy;             // if set, every K tile is also copied to [U][nk][D]
  // retained pass with ragged budgets (gathered rows only): a flat grid of
  // splits; block f belongs to unit split_unit[f], whose entry in rag gives
  // its slot count and first slot (the per-unit arrays kpos, fixed and kcopy
  // are packed), and its partials are indexed by f
  const RagUnit* rag;
  const int32_t* split_unit;
  const int32_t* split_order;   // flat split run by each block (largest first)
};

constexpr int kTileElems = 4096;   // elements of one tensor per tile
// The full-cache pass B forms P scaled by 2^kFullPBias (P <= 1, so the scaled
// value stays below 2^15 and inside fp16's range): probabilities down to
// 2^-29 stay normal fp16 numbers in the fp16 P.V, where unscaled ones below
// 2^-14 would become subnormals whose rounding, the same for every equal
// term of a flat long-context row, biases Y.  Y and the column sums are
// scaled back by the exact power of two.
constexpr float kFullPBias = 15.f;
constexpr float kFullPUnscale = 0x1p-15f;
constexpr int kRetMaxSlots = 4096;  // retained pass: key slots per block (the plan's split bound)
constexpr int kPrologueSplits = 8;  // pass B: split partials combined from one batch of loads
constexpr int kTileBytes = kTileElems * 2;

// Sum of each of NV values (8 or 16) over the 16 lanes of a DPP row, as a
// reduce-scatter: each step pairs lanes that differ in one bit b of l16 (and
// agree on the bits of the earlier steps); a lane keeps the upper half of its
// list when b is set, the lower half otherwise, and adds its partner's copy
// of that half.  Pairings: bit 3 by row_mirror (l ^ 15), bit 2 by
// row_half_mirror (l ^ 7), bit 1 by quad_perm [2,3,0,1] (l ^ 2), bit 0 by
// quad_perm [1,0,3,2] (l ^ 1); over the four steps a lane collects all 16
// lanes.  With NV = 8 the last step is a plain pair sum.  Returns the sum of
// value *v, v = the kept index (8 b3 + 4 b2 + 2 b1 + b0 for NV = 16,
// 4 b3 + 2 b2 + b1 for NV = 8).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, true));
}

template <int L, int STEP>
__device__ __forceinline__ void rs_step(float* c, int l16) {
  constexpr int CTRL = STEP == 0 ? 0x140 : STEP == 1 ? 0x141 : STEP == 2 ? 0x4E : 0xB1;
  const bool up = (l16 >> (3 - STEP)) & 1;
#pragma unroll
  for (int k = 0; k < L / 2; ++k) {
    const float keep = up ? c[k + L / 2] : c[k];
    const float send = up ? c[k] : c[k + L / 2];
    c[k] = keep + dpp_f<CTRL>(send);
  }
}

template <int NV>
__device__ __forceinline__ float row_reduce_scatter(float (&c)[NV], int l16, int* v) {
  static_assert(NV == 8 || NV == 16, "8 or 16 values");
  rs_step<NV, 0>(c, l16);
  rs_step<NV / 2, 1>(c, l16);
  rs_step<NV / 4, 2>(c, l16);
  if constexpr (NV == 16) {
    rs_step<2, 3>(c, l16);
    *v = l16;
    return c[0];
  } else {
    *v = l16 >> 1;
    return c[0] + dpp_f<0xB1>(c[0]);
  }
}

// 2^x on the transcendental unit (v_exp_f32).  Results below 2^-126 flush to
// zero, far below the precision any probability here is used at.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int D>
struct Geo {
  static constexpr int TK = kTileElems / D;           // keys per tile
  static constexpr int CPR = D / 8;                   // 16-byte chunks per row
  static constexpr int NKT = TK / 16;                 // 16-key MFMA tiles per tile
  static constexpr int RPI = 64 / CPR;                // rows filled by one wave instruction
  static constexpr int INSTR = kTileBytes / 1024;     // wave instructions per tensor per tile (8)
};

// Chunk permutation of row r.  K tiles are read as 16 rows x one chunk
// (MFMA A operand) and use r mod 16; V tiles are read by the transpose read as
// 4 rows x 2 adjacent chunks per 16 lanes (8 rows per half wave) and use
// 2(r mod 4) + 8(floor(r/4) mod 2), which puts those 16 chunks on distinct
// bank groups.
template <int D, bool VT>
__device__ __forceinline__ int swz_key(int r) {
  return (VT ? ((r & 3) << 1) | (((r >> 2) & 1) << 3) : r) & (Geo<D>::CPR - 1);
}

// Byte offset, inside a tile, of logical 16-byte chunk `ch` of row `r`.
template <int D, bool VT = false>
__device__ __forceinline__ int swz(int r, int ch) {
  return (r * Geo<D>::CPR + (ch ^ swz_key<D, VT>(r))) * 16;
}

// Direct-to-LDS loads of one tensor tile; each wave issues its share, one
// 16-byte chunk per lane and 1 KB of LDS per wave instruction.
//
// A whole tile (the common case) is addressed as the block's first key plus
// a per-lane 32-bit offset that is the same for every tile (row and swizzled
// chunk inside the tile) plus a uniform tile offset.  (The global form of the
// LDS-destination load is used: the compiler tracks which LDS array it
// writes, so reads of the other ring stages need not wait for it.)
template <int D, int WAVES, bool VT>
struct TileLoads {
  using G = Geo<D>;
  static constexpr int PER = G::INSTR / WAVES;
  const char* base;
  uint32_t off[PER];

  __device__ __forceinline__ void init(const u16* b, int key0, int wave, int lane) {
    base = reinterpret_cast<const char*>(b + (size_t)key0 * D);
#pragma unroll
    for (int it = 0; it < PER; ++it) {
      const int r = (wave * PER + it) * G::RPI + lane / G::CPR;
      const int ch = (lane % G::CPR) ^ swz_key<D, VT>(r);
      off[it] = (uint32_t)(r * D + ch * 8) * 2u;
    }
  }

  // whole tile starting `tkey` keys after the block's first key
  __device__ __forceinline__ void whole(int tkey, char* lds_tile, int wave) const {
    const char* tb = base + (size_t)tkey * D * 2;
#pragma unroll
    for (int it = 0; it < PER; ++it)
      __builtin_amdgcn_global_load_lds(tb + off[it], (lds_void*)(lds_tile + (wave * PER + it) * 1024),
                                       16, 0, 0);
  }
};

// The last, partial tile of a block: rows at or past key_end are clamped to
// key_end-1 (finite data, masked later).  With `pos` (LDS, one source row per
// key slot of the block, starting at slot key0) the rows are gathered: slot
// key reads source row pos[key - key0].
template <int D, int WAVES, bool VT>
__device__ __forceinline__ void load_tile_rows(const u16* base, int tile0, int key_end, char* lds_tile,
                                               int wave, int lane, const int32_t* pos = nullptr,
                                               int key0 = 0) {
  using G = Geo<D>;
  constexpr int PER = G::INSTR / WAVES;
#pragma unroll
  for (int it = 0; it < PER; ++it) {
    const int instr = wave * PER + it;
    const int r = instr * G::RPI + lane / G::CPR;       // row inside the tile
    const int ch = (lane % G::CPR) ^ swz_key<D, VT>(r); // logical chunk stored there
    int key = tile0 + r;
    key = key < key_end ? key : key_end - 1;
    const int64_t row = pos ? (int64_t)pos[key - key0] : (int64_t)key;
    const u16* src = base + (size_t)row * D + ch * 8;
    __builtin_amdgcn_global_load_lds(src, (lds_void*)(lds_tile + instr * 1024), 16, 0, 0);
  }
}

// Kernel modes: pass A (log-sum-exp partials), pass B over the full cache
// (P.V partials and SnapKV column sums), pass B over the retained set (P.V
// partials and the Gram matrix X_G X_G^T of the fixed-masked probabilities).
//  * kModeFull: P.V in fp16 (fp16 P times the fp16-converted V tile); a split
//    whose P.V comes out non-finite (a V element beyond the fp16 range) sets
//    its redo flag;
//  * kModeFullExact: P as a bf16 hi+lo pair times the bf16 V tile, run on the
//    splits whose redo flag is set (the other blocks exit at once).
enum { kModeLse = 0, kModeFull = 1, kModeRetained = 2, kModeFullExact = 3 };

template <int MODE>
constexpr bool is_full() { return MODE == kModeFull || MODE == kModeFullExact; }

template <bool B>
struct BoolTag {
  static constexpr bool value = B;
};

// Row tiles (16 rows) per wave: two in the full-cache passes, one in the
// retained pass (which runs twice the waves, so that its Gram and X V0
// accumulators fit two waves per SIMD).
template <int MODE>
constexpr int row_tiles() { return MODE == kModeRetained ? 1 : 2; }

// Per-block state of one (unit, split) stream.
template <int D, int MODE, int NT>
struct State {
  static constexpr int RT = row_tiles<MODE>();
  uint4 qb[RT][D / 32];
  int rowwin[RT];
  bool rowok[RT];
  float lse[RT];
  float mref[RT];   // pass A: per-lane reference exponent (an integer, or -inf
                    // before the lane's first visible key)
  double srun[RT];  // pass A: per-lane sum of 2^(t - mref) over this lane's keys
  float msum[RT];   // retained pass B: per-lane row sum of P over this lane's keys
  f32x4 y[RT][MODE != kModeLse ? D / 16 : 1];
  f32x4 n[RT][MODE == kModeRetained ? NT : 1];   // Gram rows of this wave
};

template <int D, int WAVES, int MODE, int NSTAGE>
struct Stream {
  using G = Geo<D>;
  static constexpr bool PASS_B = MODE != kModeLse;
  // P as a bf16 hi+lo pair in P.V: Y and X V0 form the residual R the solve
  // works on, and plain bf16 P (2^-9 per term) moves D_after by up to ~3e-3
  static constexpr bool SPLIT = true;
  static constexpr int RT = row_tiles<MODE>();
  static constexpr int TK = G::TK, NKT = G::NKT, NT = RT * WAVES;
  static constexpr int LOADS = (G::INSTR / WAVES) * (PASS_B ? 2 : 1);  // per thread per tile

  const StreamK& a;
  const u16* kbase;
  const u16* vbase;
  int u, key0, key_end, ntiles, win0, lane, wave, l16, g;
  size_t slot0;              // first slot of this unit in the per-slot arrays
  bool all_rows;             // m == mp: no padding rows to mask
  float (*colpart)[WAVES][TK];
  uint4* xg;                 // retained pass: fragment exchange [NT][2][64]
  const uint8_t* fixs;       // retained pass: fixed flags of this split (LDS)
  // Row tile (16 rows) held as row tile rt of this wave: tiles w and NT-1-w,
  // which pairs a short and a long row of the Gram matrix's lower triangle.
  __device__ __forceinline__ int rtile(int rt) const {
    return RT == 1 ? wave : rt == 0 ? wave : NT - 1 - wave;
  }
  const int32_t* posl;       // gathered rows: source row of each slot of this split (LDS)
  // retained pass: first fragment of this wave's row tile in the exchange
  // (a non-negative uniform value the compiler treats as opaque, so the store
  // addresses stay plain offsets into the exchange array)
  int xrow;

  TileLoads<D, WAVES, false> kld;
  TileLoads<D, WAVES, true> vld;
  // Per-lane LDS byte offsets inside a tile, computed once: K operand chunk
  // ks of key row l16 (key tile kt adds kt*16 rows), and the V transpose-read
  // address of column block dt for key row 4g + l16/4 (key pair kp adds 32
  // rows, the second half 16 rows).  The swizzle keys depend only on the row
  // modulo 8 or 16, so those row steps are plain constant offsets.
  uint32_t koff[D / 32];
  uint32_t voff[D / 16];

  __device__ __forceinline__ void init_offsets() {
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) koff[ks] = (uint32_t)swz<D>(l16, ks * 4 + g);
    const int e = l16 >> 2, qq = l16 & 3;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      const int col = dt * 16 + 4 * qq;
      voff[dt] = (uint32_t)(swz<D, true>(4 * g + e, col >> 3) + (col & 7) * 2);
    }
  }
  __device__ __forceinline__ const uint4* kaddr(const char* cur, int kt, int ks) const {
    const uint32_t o = koff[ks];
    __builtin_assume(o < kTileBytes);
    return reinterpret_cast<const uint4*>(cur + o + kt * 16 * D * 2);
  }

  __device__ __forceinline__ void issue(int t, char* stage) {
    if (t >= ntiles) return;
    const int tile0 = key0 + t * TK;
    if constexpr (MODE == kModeRetained) {
      // gathered rows (retained set read through its positions)
      if (a.gather_k || a.gather_v || tile0 + TK > key_end) {
        load_tile_rows<D, WAVES, false>(kbase, tile0, key_end, stage, wave, lane,
                                        a.gather_k ? posl : nullptr, key0);
        load_tile_rows<D, WAVES, true>(vbase, tile0, key_end, stage + kTileBytes, wave, lane,
                                       a.gather_v ? posl : nullptr, key0);
        return;
      }
    }
    if (tile0 + TK <= key_end) {
      kld.whole(t * TK, stage, wave);
      if (PASS_B) vld.whole(t * TK, stage + kTileBytes, wave);
    } else {
      load_tile_rows<D, WAVES, false>(kbase, tile0, key_end, stage, wave, lane);
      if (PASS_B) load_tile_rows<D, WAVES, true>(vbase, tile0, key_end, stage + kTileBytes, wave, lane);
    }
  }

  // Copy of the K tile in stage `cur` to kcopy (rows in key order).
  __device__ __forceinline__ void copy_k(int t, const char* cur) {
    const int tile0 = key0 + t * TK;
    for (int c = threadIdx.x; c < TK * G::CPR; c += WAVES * 64) {
      const int r = c / G::CPR, ch = c % G::CPR;
      const int key = tile0 + r;
      if (key < key_end)
        *reinterpret_cast<uint4*>(a.kcopy + (slot0 + key) * D + ch * 8) =
            *reinterpret_cast<const uint4*>(cur + swz<D>(r, ch));
    }
  }

  __device__ __forceinline__ void flush_colsum(int t) {
    // column sums of tile t (every wave wrote its part before the last
    // barrier), by the first TK lanes of wave 0 (a wave-uniform test: no
    // per-step use of the thread index, which would otherwise be held in a
    // register for the whole loop)
    if (wave == 0 && lane < TK) {
      const int key = key0 + t * TK + lane;
      if (key < key_end && key < a.prefix) {
        float c = 0.f;
#pragma unroll
        for (int wv = 0; wv < WAVES; ++wv) c += colpart[t & 1][wv][lane];
        a.colsum[(size_t)u * a.prefix + key] = c * kFullPUnscale;
      }
    }
  }

  // Gram contribution of 32 keys (16-key tiles 2kp, 2kp+1): this wave's
  // X_G fragments (hi/lo) go to LDS, then every wave forms the blocks N[I][J]
  // of its row tile I against all row tiles J (the lower triangle, J <= I, is
  // written out).  X_G is P with fixed slots zeroed.
  __device__ __forceinline__ void gram_step(int t, int kp, const float (&pv)[NKT][RT][4],
                                            State<D, MODE, NT>& S) {
    static_assert(RT == 1, "the retained pass holds one row tile per wave");
    // One exchange buffer: the step barrier between tiles, and this barrier
    // between the key pairs of one tile (64-key tiles), separate every wave's
    // reads of it from the next writes.
    if (kp > 0) lds_barrier();
    const int tl = t * TK;   // key offset of this tile inside the split
    bf16x8 fh, fl;
    {
      float x8[8];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int kl = tl + (2 * kp + h) * 16 + 4 * g + i;   // slot offset in the split
          x8[4 * h + i] = fixs[kl] ? 0.f : pv[2 * kp + h][0][i];
        }
      split8(x8, fh, fl);
      xg[xrow + lane] = __builtin_bit_cast(uint4, fh);
      xg[xrow + 64 + lane] = __builtin_bit_cast(uint4, fl);
    }
    lds_barrier();
    // All column blocks, straight-line, in two batches of fragment reads (the
    // blocks above the diagonal are computed and not written out; the MFMA
    // pipe has room for them, and a branch per block would expose an LDS
    // round trip each).
    constexpr int HB = NT > 4 ? NT / 2 : NT;
#pragma unroll
    for (int b0 = 0; b0 < NT; b0 += HB) {
      uint4 bh[HB], bl[HB];
#pragma unroll
      for (int j = 0; j < HB; ++j) {
        bh[j] = xg[((b0 + j) * 2 + 0) * 64 + lane];
        bl[j] = xg[((b0 + j) * 2 + 1) * 64 + lane];
      }
#pragma unroll
      for (int j = 0; j < HB; ++j) {
        S.n[0][b0 + j] = mfma_bf16(fh, as_bf16x8(bh[j]), S.n[0][b0 + j]);
        S.n[0][b0 + j] = mfma_bf16(fh, as_bf16x8(bl[j]), S.n[0][b0 + j]);
        S.n[0][b0 + j] = mfma_bf16(fl, as_bf16x8(bh[j]), S.n[0][b0 + j]);
      }
    }
  }

  // Full-cache pass B with fp16 P.V: tile t is computed while this thread's
  // share of tile t+1 (already complete) is converted to fp16; tiles t+2 and
  // t+3 are in flight (a four-stage ring).  The barrier at the start of each
  // step publishes the conversion made in the step before.
  __device__ __forceinline__ void step_f16(int t, char* cur, char* nxt, char* refill,
                                           State<D, MODE, NT>& S) {
    static_assert(NSTAGE == 4, "four-stage ring");
    // Every step issues one tile (past the end, the last tile again, into the
    // stage freed last step), so exactly the loads of tile t+2 may still be in
    // flight here: the wait is the same constant in every step, which keeps
    // the compiler's count of outstanding LDS loads exact.
    wait_vmcnt<LOADS>();
    lds_barrier();
    if (a.colsum && t > 0) flush_colsum(t - 1);
    issue(min(t + 3, ntiles - 1), refill);
    if (t + 1 < ntiles) v_to_f16(nxt + kTileBytes);
    // keep the scheduler from hoisting the tile's loads above the conversion
    // (register pressure)
    __builtin_amdgcn_sched_barrier(0);
    const int tile0 = key0 + t * TK;
    const bool interior = all_rows && tile0 + TK <= key_end && tile0 + TK <= win0;
    if (interior) body_full<true, true>(t, tile0, cur, S);
    else body_full<false, true>(t, tile0, cur, S);
  }

  // One tile: wait for it, refill the stage freed last step, compute.
  template <bool F16>
  __device__ __forceinline__ void step(int t, char* cur, char* refill,
                                       State<D, MODE, NT>& S) {
    if (t >= ntiles) return;
    const int ahead = min(ntiles - 1 - t, NSTAGE - 2);
    if (NSTAGE > 4 && ahead >= 3) wait_vmcnt<(NSTAGE > 4 ? 3 : 0) * LOADS>();
    else if (ahead >= 2) wait_vmcnt<2 * LOADS>();
    else if (ahead == 1) wait_vmcnt<LOADS>();
    else wait_vmcnt<0>();
    lds_barrier();
    if (is_full<MODE>() && a.colsum && t > 0) flush_colsum(t - 1);
    if (MODE == kModeRetained && a.kcopy) copy_k(t, cur);
    // The retained pass refills at the end of the step: its Gram exchange
    // has one LDS access that the compiler makes wait for every tile load in
    // flight, and a load issued at the start of the same step would still be
    // in flight there.
    if (MODE != kModeRetained) issue(t + NSTAGE - 1, refill);

    const int tile0 = key0 + t * TK;
    // An interior tile has every key valid and outside the window, and the
    // block has no padding rows: nothing to mask.
    const bool interior = all_rows && tile0 + TK <= key_end && tile0 + TK <= win0;
    if constexpr (is_full<MODE>()) {
      if (interior) body_full<true, F16>(t, tile0, cur, S);
      else body_full<false, F16>(t, tile0, cur, S);
    } else {
      f32x4 st[NKT][RT];
      logits(cur, S, st);
      float pv[NKT][RT][4];
      if (interior) body<true>(t, tile0, cur, st, pv, S);
      else body<false>(t, tile0, cur, st, pv, S);
      // once, after the branch: the exchange stores of a Gram step in both
      // branches would be merged into one store that has lost the record of
      // which LDS array it writes, and that store would wait for every tile
      // load in flight
      if constexpr (MODE == kModeRetained) {
#pragma unroll
        for (int kp = 0; kp < NKT / 2; ++kp) gram_step(t, kp, pv, S);
        issue(t + NSTAGE - 1, refill);
      }
    }
  }

  // Logits of the tile in stage `cur` for this wave's two row tiles:
  // st[kt][rt] = K[16 keys of kt] . Q[16 rows of rt]^T.
  __device__ __forceinline__ void logits(const char* cur, const State<D, MODE, NT>& S,
                                         f32x4 (&st)[NKT][RT]) {
    uint4 kv[D / 32][NKT];
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
        kv[ks][kt] = *kaddr(cur, kt, ks);
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) st[kt][rt] = zero4();
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          st[kt][rt] = mfma_bf16(as_bf16x8(kv[ks][kt]), as_bf16x8(S.qb[rt][ks]), st[kt][rt]);
  }

  // bf16 -> fp16 in place for this thread's share of the V tile at vt (the
  // element order, and so the swizzle, is unchanged).  Exact for magnitudes in
  // [2^-14, 65504]; smaller ones become fp16 subnormals (absolute error at
  // most 2^-25), larger ones overflow to infinity, which the caller detects.
  __device__ __forceinline__ void v_to_f16(char* vt) {
    constexpr int CH = kTileBytes / 16, PER = CH / (WAVES * 64);
    static_assert(PER * WAVES * 64 == CH, "whole chunks per thread");
    uint4 x[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) x[k] = *reinterpret_cast<const uint4*>(vt + (threadIdx.x + k * WAVES * 64) * 16);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      x[k].x = bf16x2_to_f16x2(x[k].x);
      x[k].y = bf16x2_to_f16x2(x[k].y);
      x[k].z = bf16x2_to_f16x2(x[k].z);
      x[k].w = bf16x2_to_f16x2(x[k].w);
      *reinterpret_cast<uint4*>(vt + (threadIdx.x + k * WAVES * 64) * 16) = x[k];
    }
  }

  // V operand fragment of keys 32kp + (4g + e, +16), columns dt*16 + 4q..+3
  // (lane 4e + q of group g supplies the address), by the LDS transpose read.
  __device__ __forceinline__ uint4 v_frag(const char* vt, int kp, int dt) const {
    const uint32_t o = voff[dt];
    __builtin_assume(o < kTileBytes);
    const char* p0 = vt + o + kp * 32 * D * 2;
    v4i16 b0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p0);
    v4i16 b1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0 + 16 * D * 2));
    return __builtin_bit_cast(uint4, (v8i16){b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]});
  }

  // Full-cache pass B on one tile, ordered by row tile so that the VALU work
  // of one row tile (exponentials, operand packing) can run beside the MFMAs
  // of the other.  F16: P.V as fp16 P times the fp16 V tile (one MFMA per
  // fragment); otherwise P as a bf16 hi+lo pair times the bf16 V tile.
  template <bool INTERIOR, bool F16>
  __device__ __forceinline__ void body_full(int t, int tile0, const char* cur,
                                            State<D, MODE, NT>& S) {
    uint4 kv[D / 32][NKT];
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
        kv[ks][kt] = *kaddr(cur, kt, ks);
    f32x4 st[2][NKT];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        st[rt][kt] = zero4();
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks)
          st[rt][kt] = mfma_bf16(as_bf16x8(kv[ks][kt]), as_bf16x8(S.qb[rt][ks]), st[rt][kt]);
      }
    // V operand fragments of the whole tile (shared by both row tiles), read
    // once the K fragments are dead
    const char* vt = cur + kTileBytes;
    uint4 b[NKT / 2][D / 16];
#pragma unroll
    for (int kp = 0; kp < NKT / 2; ++kp)
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) b[kp][dt] = v_frag(vt, kp, dt);
    float pv[2][NKT][4];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float x = fast_exp2(fmaf(st[rt][kt][i], a.scale_log2, -S.lse[rt]));
          if (INTERIOR) {
            pv[rt][kt][i] = x;
          } else {
            const int key = tile0 + kt * 16 + 4 * g + i;
            pv[rt][kt][i] = (S.rowok[rt] && key < key_end && key - win0 <= S.rowwin[rt]) ? x : 0.f;
          }
        }
#pragma unroll
      for (int kp = 0; kp < NKT / 2; ++kp) {
        const float x8[8] = {pv[rt][2 * kp][0], pv[rt][2 * kp][1], pv[rt][2 * kp][2],
                             pv[rt][2 * kp][3], pv[rt][2 * kp + 1][0], pv[rt][2 * kp + 1][1],
                             pv[rt][2 * kp + 1][2], pv[rt][2 * kp + 1][3]};
        if constexpr (F16) {
          const f16x8 ph = to_f16x8(x8);
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt)
            S.y[rt][dt] = mfma_f16(ph, __builtin_bit_cast(f16x8, b[kp][dt]), S.y[rt][dt]);
        } else {
          bf16x8 ahi, alo;
          split8(x8, ahi, alo);
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt) {
            S.y[rt][dt] = mfma_bf16(ahi, as_bf16x8(b[kp][dt]), S.y[rt][dt]);
            S.y[rt][dt] = mfma_bf16(alo, as_bf16x8(b[kp][dt]), S.y[rt][dt]);
          }
        }
      }
    }
    // column sums over this wave's 32 rows: the two row tiles first, then the
    // 16 lanes of each DPP row (one reduce-scatter; lane l16 ends with key
    // v = kt*4 + i of its group, v taken from the high bits of l16; with 8
    // values both lanes of a pair hold the same sum and store it)
    float cs[NKT * 4];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) cs[kt * 4 + i] = pv[0][kt][i] + pv[1][kt][i];
    int v;
    const float c = row_reduce_scatter<NKT * 4>(cs, l16, &v);
    if (NKT * 4 == 16 || (l16 & 1) == 0) colpart[t & 1][wave][(v >> 2) * 16 + 4 * g + (v & 3)] = c;
  }

  // The tile's work after the logits.  INTERIOR skips every mask.
  template <bool INTERIOR>
  __device__ __forceinline__ void body(int t, int tile0, const char* cur, const f32x4 (&st)[NKT][RT],
                                       float (&pv)[NKT][RT][4], State<D, MODE, NT>& S) {
    bool ok[NKT][RT][4];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = tile0 + kt * 16 + 4 * g + i;
        const int kw = key - win0;   // < 0 outside the window
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          ok[kt][rt][i] = INTERIOR || (S.rowok[rt] && key < key_end && kw <= S.rowwin[rt]);
      }

    if (!PASS_B) {
      // Sum of 2^(t - ref) against a per-lane integer reference.  The
      // reference is set from the first visible tile (ceil of its largest
      // scaled logit) and moved up only when a tile's partial sum exceeds
      // 2^64, so the tile maximum is taken only on those rare tiles, and a
      // move rescales the running sum exactly (a power of two).  Terms below
      // the float range (2^-126 under the reference) are at least 2^-125
      // smaller than the sum and drop out.
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const float nref = -S.mref[rt];
        float acc = 0.f;
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float e = fast_exp2(fmaf(st[kt][rt][i], a.scale_log2, nref));
            acc += ok[kt][rt][i] ? e : 0.f;
          }
        // also taken when the reference is still -inf and a key is visible
        // (the sum is then +inf)
        if (!(acc <= 0x1p64f)) {
          float smax = -INFINITY;
#pragma unroll
          for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) smax = fmaxf(smax, ok[kt][rt][i] ? st[kt][rt][i] : -INFINITY);
          acc = 0.f;
          if (smax != -INFINITY) {
            const float ref = ceilf(smax * a.scale_log2);
            S.srun[rt] = S.mref[rt] == -INFINITY ? 0.0 : ldexp(S.srun[rt], (int)(S.mref[rt] - ref));
            S.mref[rt] = ref;
#pragma unroll
            for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const float e = fast_exp2(fmaf(st[kt][rt][i], a.scale_log2, -ref));
                acc += ok[kt][rt][i] ? e : 0.f;
              }
          }
        }
        S.srun[rt] += (double)acc;
      }
      return;
    }

#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = fast_exp2(fmaf(st[kt][rt][i], a.scale_log2, -S.lse[rt]));
          pv[kt][rt][i] = ok[kt][rt][i] ? e : 0.f;
        }
    if (MODE == kModeRetained && a.mpart) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        float acc = 0.f;
#pragma unroll
        for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc += pv[kt][rt][i];
        S.msum[rt] += acc;
      }
    }
    const char* vt = cur + kTileBytes;
#pragma unroll
    for (int kp = 0; kp < NKT / 2; ++kp) {
      bf16x8 ahi[RT], alo[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        float x8[8] = {pv[2 * kp][rt][0], pv[2 * kp][rt][1], pv[2 * kp][rt][2], pv[2 * kp][rt][3],
                       pv[2 * kp + 1][rt][0], pv[2 * kp + 1][rt][1], pv[2 * kp + 1][rt][2],
                       pv[2 * kp + 1][rt][3]};
        if (SPLIT) {
          split8(x8, ahi[rt], alo[rt]);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) ahi[rt][q] = (__bf16)x8[q];
        }
      }
      bf16x8 b[D / 16];
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) b[dt] = as_bf16x8(v_frag(vt, kp, dt));
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          S.y[rt][dt] = mfma_bf16(ahi[rt], b[dt], S.y[rt][dt]);
          if (SPLIT) S.y[rt][dt] = mfma_bf16(alo[rt], b[dt], S.y[rt][dt]);
        }
    }
  }
};

template <int D, int WAVES, int MODE>
__global__ __launch_bounds__(WAVES * 64)
__attribute__((amdgpu_waves_per_eu(MODE == kModeLse ? 4 : 2))) void stream_kernel(StreamK a) {
  using G = Geo<D>;
  constexpr bool PASS_B = MODE != kModeLse;
  constexpr int RT = row_tiles<MODE>();
  constexpr int TK = G::TK, NT = RT * WAVES;
  // ring depth: pass A 5 x 8 KB (four blocks per CU at 4 waves per SIMD);
  // pass B 4 x 16 KB (one stage holds the tile whose V is being converted);
  // retained pass 5 x 16 KB (one block of twice the waves per CU, so its
  // ring is deeper)
  constexpr int NSTAGE = MODE == kModeFull ? 4 : MODE == kModeFullExact ? 3 : 5;
  static_assert(NSTAGE >= 3 && NSTAGE <= 5, "ring depths with an unrolled loop below");
  constexpr int STAGE_BYTES = kTileBytes * (PASS_B ? 2 : 1);
  __shared__ __attribute__((aligned(16))) char stg0[STAGE_BYTES];
  __shared__ __attribute__((aligned(16))) char stg1[STAGE_BYTES];
  __shared__ __attribute__((aligned(16))) char stg2[STAGE_BYTES];
  __shared__ __attribute__((aligned(16))) char stg3[NSTAGE > 3 ? STAGE_BYTES : 16];
  __shared__ __attribute__((aligned(16))) char stg4[NSTAGE > 4 ? STAGE_BYTES : 16];
  __shared__ float colpart[2][WAVES][TK];
  // retained pass only: X_G fragment exchange [NT][2][64], fixed flags and
  // source rows of the split's slots (static arrays, so the compiler can tell
  // them apart from the ring stages the tile loads are filling)
  constexpr bool RET = MODE == kModeRetained;
  __shared__ __attribute__((aligned(16))) uint4 xgs[RET ? NT * 2 * 64 : 1];
  __shared__ uint8_t fixl[RET ? kRetMaxSlots : 1];
  __shared__ int32_t posl[RET ? kRetMaxSlots : 1];

  if (MODE == kModeFullExact && !a.redo[(size_t)blockIdx.y * a.S + blockIdx.x]) return;
  Stream<D, WAVES, MODE, NSTAGE> sm{a};
  // unit, split, key count and partial index of this block
  int s = blockIdx.x, nk = a.nk;
  size_t pidx = (size_t)blockIdx.y * a.S + blockIdx.x;
  sm.u = blockIdx.y;
  sm.slot0 = (size_t)blockIdx.y * a.nk;
  if (RET && a.rag) {
    const int f = a.split_order[blockIdx.x];
    sm.u = a.split_unit[f];
    const RagUnit ru = a.rag[sm.u];
    s = f - ru.s0;
    nk = ru.c;
    sm.slot0 = (size_t)ru.off;
    pidx = (size_t)f;
  }
  sm.lane = threadIdx.x & 63;
  sm.wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  sm.l16 = sm.lane & 15;
  sm.g = sm.lane >> 4;
  sm.key0 = s * a.chunk;
  sm.key_end = min(sm.key0 + a.chunk, nk);
  sm.ntiles = sm.key_end > sm.key0 ? (sm.key_end - sm.key0 + TK - 1) / TK : 0;
  sm.kbase = a.k + (size_t)sm.u * (a.gather_k ? a.src_rows : (int64_t)nk) * D;
  sm.vbase = a.v + (size_t)sm.u * (a.gather_v ? a.src_rows : (int64_t)nk) * D;
  sm.win0 = nk - a.w;
  sm.all_rows = a.m == a.mp;
  sm.init_offsets();
  // (the gathered retained pass does not use these)
  sm.kld.init(sm.kbase, sm.key0, sm.wave, sm.lane);
  if (PASS_B) sm.vld.init(sm.vbase, sm.key0, sm.wave, sm.lane);
  sm.colpart = colpart;
  sm.xg = xgs;
  {
    int x = sm.rtile(0) * 2 * 64;
    asm("" : "+s"(x));
    sm.xrow = x;
  }
  sm.fixs = fixl;
  sm.posl = posl;
  const int u = sm.u, wave = sm.wave, l16 = sm.l16, g = sm.g;
  const int nsl = sm.ntiles * TK;   // <= kRetMaxSlots in the retained pass (host check)

  if (RET) {
    // fixed flags of this split's slots (padded with "fixed" past the end)
    for (int i = threadIdx.x; i < nsl; i += WAVES * 64) {
      const int key = sm.key0 + i;
      fixl[i] = key < sm.key_end ? a.fixed[sm.slot0 + key] : 1;
    }
    if (a.gather_k || a.gather_v) {
      // source row of each slot, clamped into the source tensor
      for (int i = threadIdx.x; i < nsl; i += WAVES * 64) {
        const int key = min(sm.key0 + i, sm.key_end - 1);
        const int64_t r = a.kpos[sm.slot0 + key];
        posl[i] = (int32_t)(r < 0 ? 0 : r >= a.src_rows ? a.src_rows - 1 : r);
      }
    }
  }
  if (RET) __syncthreads();

  State<D, MODE, NT> S;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int row = sm.rtile(rt) * 16 + l16;
    S.rowok[rt] = row < a.m;
    S.rowwin[rt] = a.causal ? row % a.w : 0x3fffffff;
    // rows past m read row m - 1 (in bounds) and are masked: the loads are
    // issued without branches, in flight together
    const u16* q = a.q + ((size_t)u * a.m + min(row, a.m - 1)) * D;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const uint4 v = *reinterpret_cast<const uint4*>(q + ks * 32 + 8 * g);
      S.qb[rt][ks] = S.rowok[rt] ? v : make_uint4(0, 0, 0, 0);
    }
    if (is_full<MODE>() && a.lse_ready) {
      S.lse[rt] = a.lse_log2_out[(size_t)u * a.mp + row] - kFullPBias;
    } else if constexpr (is_full<MODE>()) {
      // fixed-order combine of pass A's split partials: M = max of the
      // integer reference exponents, sum = sum_s psum_s 2^(ref_s - M) (exact
      // powers of two), LSE (log2) = M + log2(sum).  Up to kPrologueSplits
      // splits have all their partials loaded at once (indices past S
      // clamped, not used).
      float M = -INFINITY;
      double l2 = 0.0;
      if (a.S <= kPrologueSplits) {
        float pm[kPrologueSplits];
        double pz[kPrologueSplits];
#pragma unroll
        for (int k = 0; k < kPrologueSplits; ++k) {
          const size_t o = ((size_t)u * a.S + min(k, a.S - 1)) * a.mp + row;
          pm[k] = a.pmax[o];
          pz[k] = a.psum[o];
        }
#pragma unroll
        for (int k = 0; k < kPrologueSplits; ++k)
          if (k < a.S) M = fmaxf(M, pm[k]);
        if (M != -INFINITY) {
          double sum = 0.0;
#pragma unroll
          for (int k = 0; k < kPrologueSplits; ++k)
            if (k < a.S && pm[k] != -INFINITY) sum += pz[k] * exp2((double)pm[k] - (double)M);
          l2 = (double)M + log2(sum);
        }
      } else {
        for (int sp = 0; sp < a.S; ++sp) M = fmaxf(M, a.pmax[((size_t)u * a.S + sp) * a.mp + row]);
        if (M != -INFINITY) {
          double sum = 0.0;
          for (int sp = 0; sp < a.S; ++sp) {
            const size_t o = ((size_t)u * a.S + sp) * a.mp + row;
            const float ms = a.pmax[o];
            if (ms != -INFINITY) sum += a.psum[o] * exp2((double)ms - (double)M);
          }
          l2 = (double)M + log2(sum);
        }
      }
      S.lse[rt] = (float)l2 - kFullPBias;
      if (s == 0 && g == 0) {
        a.lse_out[(size_t)u * a.mp + row] = M != -INFINITY ? l2 * 0.69314718055994530942 : -INFINITY;
        a.lse_log2_out[(size_t)u * a.mp + row] = (float)l2;
      }
    } else {
      S.lse[rt] = PASS_B ? a.lse_log2[(size_t)u * a.mp + row] - a.lse_bias : 0.f;
    }
    S.msum[rt] = 0.f;
    S.mref[rt] = -INFINITY;
    S.srun[rt] = 0.0;
#pragma unroll
    for (int dt = 0; dt < (PASS_B ? D / 16 : 1); ++dt) S.y[rt][dt] = zero4();
#pragma unroll
    for (int bt = 0; bt < (MODE == kModeRetained ? NT : 1); ++bt) S.n[rt][bt] = zero4();
  }

  auto run = [&](auto f16) {
    constexpr bool F16 = decltype(f16)::value;
    if constexpr (F16) {
      // tiles 0..2 (clamped to the last tile) in flight; tile 0 converted
      // before the loop (published by step 0's barrier)
      const int last = sm.ntiles - 1;
      if (last >= 0) {
        sm.issue(0, stg0);
        sm.issue(min(1, last), stg1);
        sm.issue(min(2, last), stg2);
        wait_vmcnt<2 * decltype(sm)::LOADS>();
        lds_barrier();
        sm.v_to_f16(stg0 + kTileBytes);
      }
      // whole groups of four steps as straight-line code (every step names
      // its stages at compile time), then the remaining zero to three steps
      int t = 0;
      for (; t + 4 <= sm.ntiles; t += 4) {
        sm.step_f16(t + 0, stg0, stg1, stg3, S);
        sm.step_f16(t + 1, stg1, stg2, stg0, S);
        sm.step_f16(t + 2, stg2, stg3, stg1, S);
        sm.step_f16(t + 3, stg3, stg0, stg2, S);
      }
      if (t < sm.ntiles) sm.step_f16(t, stg0, stg1, stg3, S);
      if (t + 1 < sm.ntiles) sm.step_f16(t + 1, stg1, stg2, stg0, S);
      if (t + 2 < sm.ntiles) sm.step_f16(t + 2, stg2, stg3, stg1, S);
      // the clamped loads past the end must land before the block's LDS is
      // released
      wait_vmcnt<0>();
    } else {
      sm.issue(0, stg0);
      sm.issue(1, stg1);
      if constexpr (NSTAGE >= 4) sm.issue(2, stg2);
      if constexpr (NSTAGE == 5) sm.issue(3, stg3);
      for (int t = 0; t < sm.ntiles; t += NSTAGE) {
        if constexpr (NSTAGE == 3) {
          sm.template step<F16>(t + 0, stg0, stg2, S);
          sm.template step<F16>(t + 1, stg1, stg0, S);
          sm.template step<F16>(t + 2, stg2, stg1, S);
        } else if constexpr (NSTAGE == 4) {
          sm.template step<F16>(t + 0, stg0, stg3, S);
          sm.template step<F16>(t + 1, stg1, stg0, S);
          sm.template step<F16>(t + 2, stg2, stg1, S);
          sm.template step<F16>(t + 3, stg3, stg2, S);
        } else {
          sm.template step<F16>(t + 0, stg0, stg4, S);
          sm.template step<F16>(t + 1, stg1, stg0, S);
          sm.template step<F16>(t + 2, stg2, stg1, S);
          sm.template step<F16>(t + 3, stg3, stg2, S);
          sm.template step<F16>(t + 4, stg4, stg3, S);
        }
      }
    }
    if (is_full<MODE>() && a.colsum && sm.ntiles > 0) {
      lds_barrier();
      sm.flush_colsum(sm.ntiles - 1);
    }
  };

  if constexpr (MODE == kModeFull) {
    run(BoolTag<true>{});
    // A V element beyond the fp16 range (|v| > 65504) makes this split's P.V
    // non-finite: flag the split for the exact pass.
    bool bad = false;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) bad |= !__builtin_isfinite(S.y[rt][dt][i]);
    bad = __syncthreads_or(bad);
    if (threadIdx.x == 0) a.redo[pidx] = bad ? 1 : 0;
    if (bad) return;
  } else {
    run(BoolTag<false>{});
  }

  if (PASS_B) {
    float* yp = a.ypart + pidx * a.mp * D;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = sm.rtile(rt) * 16 + 4 * g + i;
          yp[(size_t)row * D + dt * 16 + l16] =
              is_full<MODE>() ? S.y[rt][dt][i] * kFullPUnscale : S.y[rt][dt][i];
        }
    if (MODE == kModeRetained) {
      if (a.mpart) {
        // row sums: the four lane groups of a row hold disjoint keys
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          float v = S.msum[rt];
          v += __shfl_xor(v, 16);
          v += __shfl_xor(v, 32);
          if (g == 0) a.mpart[pidx * a.mp + sm.rtile(rt) * 16 + l16] = v;
        }
      }
      // lower blocks N[I][J] (J <= I) and their mirrors N[J][I]
      float* np = a.npart + pidx * a.mp * a.mp;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int bt = 0; bt < (MODE == kModeRetained ? NT : 1); ++bt) {
          const int I = sm.rtile(rt);
          if (bt > I) continue;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            np[(size_t)(I * 16 + 4 * g + i) * a.mp + bt * 16 + l16] = S.n[rt][bt][i];
          if (bt < I)
            *reinterpret_cast<float4*>(np + (size_t)(bt * 16 + l16) * a.mp + I * 16 + 4 * g) =
                make_float4(S.n[rt][bt][0], S.n[rt][bt][1], S.n[rt][bt][2], S.n[rt][bt][3]);
        }
    }
  } else {
    // merge the four lanes of each row: M = max ref_g, sum = sum_g s_g 2^(ref_g - M)
    // (integer exponents: exact)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      float M = max_over_groups(S.mref[rt]);
      double part = (S.mref[rt] == -INFINITY) ? 0.0 : ldexp(S.srun[rt], (int)(S.mref[rt] - M));
      const double tot = sum_over_groups(part);
      const int row = sm.rtile(rt) * 16 + l16;
      if (g == 0) {
        const size_t o = pidx * a.mp + row;
        a.pmax[o] = M;
        a.psum[o] = M == -INFINITY ? 0.0 : tot;
      }
    }
  }
}

template <int D, int WAVES, int MODE>
hipError_t launch_stream_t(const Plan& p, const AttnPass& a, hipStream_t s) {
  StreamK k;
  k.q = (const u16*)a.q; k.k = (const u16*)a.k; k.v = (const u16*)a.v;
  k.m = p.m; k.mp = p.mp; k.w = p.w; k.causal = p.opt.causal_window ? 1 : 0;
  k.nk = a.nk; k.S = a.S; k.chunk = a.chunk;
  k.scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)D));
  k.pmax = a.pmax; k.psum = a.psum; k.lse_log2 = a.lse_log2;
  k.lse_out = const_cast<double*>(a.lse); k.lse_log2_out = const_cast<float*>(a.lse_log2);
  k.lse_ready = a.lse_ready ? 1 : 0;
  k.ypart = a.ypart; k.colsum = a.colsum; k.prefix = a.prefix;
  k.fixed = a.fixed; k.npart = a.npart; k.mpart = a.mpart; k.lse_bias = a.lse_bias;
  k.redo = a.redo;
  k.kpos = a.kpos; k.src_rows = a.src_rows;
  k.gather_k = a.gather_k ? 1 : 0; k.gather_v = a.gather_v ? 1 : 0;
  k.kcopy = (u16*)a.kcopy;
  k.rag = MODE == kModeRetained ? p.rag : nullptr;
  k.split_unit = p.rag_split_unit;
  k.split_order = p.rag_split_order;
  if ((k.gather_k || k.gather_v) && (!a.kpos || a.src_rows < 1)) return hipErrorInvalidValue;
  // ragged budgets: gathered rows only (the per-unit source tensors are the
  // full caches, never a [U][nk][d] array of one budget)
  if (k.rag && (!k.gather_k || !k.gather_v || !k.split_unit || !k.split_order ||
                p.rag_splits < 1))
    return hipErrorInvalidValue;
  if (MODE == kModeRetained) {
    const int tk = kTileElems / D;
    if ((size_t)((a.chunk + tk - 1) / tk) * tk > (size_t)kRetMaxSlots) return hipErrorInvalidValue;
  } else if (k.gather_k || k.gather_v) {
    return hipErrorInvalidValue;   // only the retained pass reads rows through positions
  }
  const dim3 grid = k.rag ? dim3(p.rag_splits, 1) : dim3(a.S, p.U);
  hipLaunchKernelGGL((stream_kernel<D, WAVES, MODE>), grid, dim3(WAVES * 64), 0, s, k);
  return hipGetLastError();
}

template <int D, int MODE>
hipError_t launch_stream_w(const Plan& p, const AttnPass& a, hipStream_t s) {
  // one wave per row tile in the retained pass, one per two elsewhere
  const int waves = p.mp / (16 * row_tiles<MODE>());
  switch (waves) {
    case 1:
      // (the retained pass has at least two row tiles)
      if constexpr (MODE != kModeRetained) return launch_stream_t<D, 1, MODE>(p, a, s);
      break;
    case 2: return launch_stream_t<D, 2, MODE>(p, a, s);
    case 4: return launch_stream_t<D, 4, MODE>(p, a, s);
    case 8: return launch_stream_t<D, 8, MODE>(p, a, s);
  }
  return hipErrorInvalidValue;
}

template <int D>
hipError_t launch_stream_d(const Plan& p, const AttnPass& a, int mode, hipStream_t s) {
  if (mode == kModeLse) return launch_stream_w<D, kModeLse>(p, a, s);
  if (mode == kModeFull) {
    // fp16 pass, then the exact pass on the splits it flagged
    if (!a.redo) return hipErrorInvalidValue;
    hipError_t e = launch_stream_w<D, kModeFull>(p, a, s);
    if (e != hipSuccess) return e;
    return launch_stream_w<D, kModeFullExact>(p, a, s);
  }
  return launch_stream_w<D, kModeRetained>(p, a, s);
}

}  // namespace

bool stream_supported(const Plan& p) {
  return p.dtype == GRKV_BF16 && (p.d == 64 || p.d == 128) &&
         (p.waves == 1 || p.waves == 2 || p.waves == 4 || p.waves == 8);
}

hipError_t launch_stream(const Plan& p, const AttnPass& a, int mode, hipStream_t s) {
  if (p.d == 128) return launch_stream_d<128>(p, a, mode, s);
  return launch_stream_d<64>(p, a, mode, s);
}

}  // namespace grkv
