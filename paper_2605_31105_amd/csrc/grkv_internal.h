// Internal declarations shared by the host API and the kernel launchers of the
// gfx950 GRKV path.  Not installed; the public interface is include/grkv.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "grkv.h"

namespace grkv {

constexpr int kRowsPerWave = 32;   // each wave owns 32 stacked window rows
constexpr int kKeyTile = 32;       // keys per streamed tile
constexpr int kSelectThreads = 1024;
// The fast retained pass forms P = 2^(t - LSE + kRetainedBias) against the
// full-cache log-sum-exp: retained attention masses down to 2^-108 stay
// well inside the float range (P <= 2^48, Gram entries <= 2^96).
constexpr float kRetainedBias = 48.f;
// From this many full-cache splits per unit (small calls), pass A's partials
// and the Y partials are combined by their own kernels over all rows at once
// instead of serially inside every pass-B block and every solve block.
constexpr int kPrecombineSplits = 16;
// The same for the retained-pass partials (X V0, Gram, row masses) from this
// many retained splits per unit.
constexpr int kPrecombineRetSplits = 8;

// Ragged budgets: one entry per unit, in device memory.  The packed outputs
// hold unit u's c slots from slot `off`; its retained-pass splits are the
// flat blocks s0 .. s0 + ns - 1 (their partials are indexed by the flat block
// number), its update blocks ub0 .. ub0 + nub - 1; ntop is the size of its
// score-ranked fixed subset, min(floor(beta c), c - w).
struct RagUnit {
  int32_t off, c, s0, ns, ntop, ub0, nub, pad;
};

// Everything a call needs, derived on the host from the arguments.
struct Plan {
  // shape
  int U, G, w, m, mp, waves, d, dtype;
  int64_t n;
  int c, s_sel, prefix, k_pool, n_top_fixed;
  float lam;
  grkv_options opt;
  // work split of the full-cache passes: S1 splits of chunk1 keys per unit
  int S1, chunk1;
  // retained-cache passes over the c retained keys
  int S2, chunk2;
  // Gram-matrix splits over the c retained columns (the retained-pass splits
  // on the fast value-step path, where that pass produces the Gram partials)
  int S3, chunk3;
  bool fast_merge;
  // blocks per unit of the fast solve (column tiles of Z split between them,
  // each block factoring N itself): more than one only for calls with few
  // units, where one block per unit leaves most of the GPU idle
  int csplit;
  // ragged budgets (bf16 fast path): device tables, null for one budget.
  // p.c is then the largest budget, chunk2 the uniform split length of the
  // retained pass and upd_spb the slots per update block.
  // Blocks are launched largest first (split f = *_order[blockIdx.x]), so
  // that the short remainder splits fill the compute units that finish early.
  const RagUnit* rag;
  const int32_t* rag_split_unit;   // [rag_splits] unit of each retained-pass split
  const int32_t* rag_upd_unit;     // [rag_upd_blocks] unit of each update block
  const int32_t* rag_split_order;  // [rag_splits] split run by each retained-pass block
  const int32_t* rag_upd_order;    // [rag_upd_blocks] update block run by each block
  int rag_splits, rag_upd_blocks, upd_spb;
  // workspace offsets (bytes)
  size_t pmax1, psum1, lse1, lse1_log2, ypart, y, colsum, pooled, fixed, v0c, redo;
  size_t pmax2, psum2, lse2, lse2_log2, xvpart, x, resid, npart, mpart, gram, z, zhi, zlo, stats_ws;
  // [U][kZParts] double (csplit > 1): ||Z||^2 of each solve block's columns,
  // and ||Y||^2 in the last entry
  size_t zpart;
  // retained-pass partials summed over the splits (small calls only)
  size_t xvcomb, ncomb, mcomb;
  size_t rag_tab;   // ragged tables: RagUnit [U], then the two block-to-unit maps
  size_t total;
};

constexpr int kZParts = 16;   // solve blocks per unit at most, plus ||Y||^2 (entry 15)

// Fills `plan`; returns GRKV_OK or the error the call must report.
int make_plan(const grkv_problem* prob, int64_t n, int32_t window,
              int32_t budget, int32_t pool_kernel, float lambda,
              const grkv_options* opt, Plan* plan);

// One streamed attention pass over nk keys per unit.
struct AttnPass {
  const void* q;       // [U][m][d] stacked window rows
  const void* k;       // [U][nk][d]
  const void* v;       // [U][nk][d] (pass B only)
  const int32_t* kpos; // [U][nk] token position of each key, or null (= key index)
  int nk;              // keys per unit
  int S, chunk;        // splits per unit and keys per split
  float* pmax;         // pass A out [U][S][mp]: row max of log2-scaled logits
  double* psum;        // pass A out [U][S][mp]: sum of 2^(t - max)
  const double* lse;   // in: [U][mp] natural LSE (combine output)
  const float* lse_log2; // pass B in: [U][mp] log2-domain LSE
  float* ypart;        // pass B out [U][S][mp][d]
  float* colsum;       // pass B out [U][prefix] column sums over rows, or null
  int prefix;          // only keys < prefix get a column sum
  float* xout;         // pass B out [U][mp][nk] probabilities, or null (generic path)
  bool split_p;        // P.V with P as a bf16 hi+lo pair (else bf16 P)
  bool lse_ready;      // full-cache pass B (bf16 streaming): lse / lse_log2 already
                       // combined from pass A's partials (else combined per block)
  const uint8_t* fixed; // retained pass B (fast path): fixed flags [U][nk]
  float* npart;        // retained pass B (fast path): Gram partials [U][S][mp][mp]
  // streaming passes over the retained set: read K and/or V rows through
  // kpos from tensors of src_rows rows per unit (instead of [U][nk][d]), and
  // optionally copy the K tiles to kcopy [U][nk][d]
  bool gather_k, gather_v;
  int64_t src_rows;
  void* kcopy;
  // retained pass B (fast path): P = 2^(t - (lse_log2 - lse_bias)) against
  // the full-cache LSE, with its row sums in mpart [U][S][mp]
  float lse_bias;
  float* mpart;
  // full-cache pass B (bf16 streaming): per-split flags [U][S] of the fp16
  // P.V pass; flagged splits are recomputed exactly
  int* redo;
};

hipError_t launch_lse_pass(const Plan& p, const AttnPass& a, hipStream_t s);
hipError_t launch_lse_combine(const Plan& p, const float* pmax,
                              const double* psum, int S, double* lse,
                              float* lse_log2, hipStream_t s);
hipError_t launch_prob_pass(const Plan& p, const AttnPass& a, hipStream_t s);
// out[i][u][e] = sum over s < S[i] of part[i][u][s][e], e < per_unit[i], for
// up to four arrays i (a per_unit of 0 leaves that array out); one launch.
constexpr int kCombineSegs = 4;
hipError_t launch_combine_parts(int U, const int S[kCombineSegs],
                                const float* const part[kCombineSegs],
                                float* const out[kCombineSegs],
                                const size_t per_unit[kCombineSegs], hipStream_t s);
// out[u][r][c] = (base ? base[u][r][c] : 0) +/- sum_s part[u][s][r][c]
hipError_t launch_combine_rows(const Plan& p, const float* part, int S,
                               const float* base, float* out, hipStream_t s);

// bf16 streaming passes (direct-to-LDS ring); used when stream_supported().
// mode 0: pass A; 1: full-cache pass B (column sums); 2: retained pass B with
// the Gram partials of the fixed-masked probabilities (needs mp <= 128).
bool stream_supported(const Plan& p);
hipError_t launch_stream(const Plan& p, const AttnPass& a, int mode, hipStream_t s);

hipError_t launch_select(const Plan& p, const float* colsum, float* pooled,
                         int32_t* idx, uint8_t* fixed, hipStream_t s);
// K0 -> k_out, V0 -> v0c (input dtype); V0 as fp32 -> v_out when v_out is not null.
hipError_t launch_gather(const Plan& p, const void* K, const void* V,
                         const int32_t* idx, void* k_out, void* v0c,
                         float* v_out, hipStream_t s);
hipError_t launch_gram(const Plan& p, const float* x, const uint8_t* fixed,
                       float* npart, hipStream_t s);

// Fast value step (bf16, mp <= 128): the solve combines the Y, X V0 and Gram
// partials (writing y, resid and gram) and solves by blocked Cholesky; then
// v_out = V0 + X_G^T Z is written in one pass from the compact V0 copy.
bool merge_fast_supported(const Plan& p);
// mpart: row sums of the retained P partials [U][S2][mp] when P was formed
// against the full-cache LSE lse1_log2 scaled by 2^lse_bias (X = P / row sum;
// the retained LSE is written to lse2_log2), or null when X itself was used.
// ypart holds S1 partials per unit (p.S1, or 1 when Y was combined already);
// xvpart, npart and mpart S2 (p.S2, or 1), unless p.rag gives each unit's own.
// Units it marks GRKV_UNIT_RANGE (with mpart: a window row's retained mass
// below what P against the full-cache LSE resolves) get the value step again
// in the same launch, by their first block, against the retained set's own
// row maxima (range_fix.h), from q_obs, K0 (k0 = k_out), V through idx and
// the fixed flags; it writes the retained LSE, R, N, Z^T and the stats where
// the solve does.
hipError_t launch_solve(const Plan& p, const float* ypart, int S1, int S2, const float* xvpart,
                        const float* npart, const float* mpart, const float* lse1_log2,
                        float lse_bias, float* lse2_log2, float* y, float* resid,
                        float* gram, float* z, uint16_t* zhi, uint16_t* zlo,
                        float* stats_ws, float* stats_user, double* zpart, const void* q,
                        const void* k0, const void* V, const int32_t* idx,
                        const uint8_t* fixed, hipStream_t s);
// X is recomputed from q_obs, K0 (k_out) and the retained log-sum-exp; V0
// rows are read from V [U][n][d] through idx.
// Slots per update block for budget c (blocks per unit = ceil(c / spb)).
int update_slots_per_block(const Plan& p, int c);
hipError_t launch_update(const Plan& p, const void* q, const void* k0,
                         const float* lse_log2, const uint8_t* fixed,
                         const uint16_t* zhi, const uint16_t* zlo,
                         const float* stats_ws, const void* V, const int32_t* idx,
                         float* v_out, const double* zpart, float* stats_user, hipStream_t s);

// Generic value step (any dtype, mp up to 256): Cholesky in LDS; the update
// adds X_G^T Z into v_out, which the gather filled with V0.
// Writes the per-unit stats to stats_ws (always) and stats_user (if not null).
hipError_t launch_cholesky_solve(const Plan& p, const float* npart,
                                 const float* y, const float* resid,
                                 float* gram, float* z, float* stats_ws,
                                 float* stats_user, hipStream_t s);
// The same solve for mp = 256 (G * w in (128, 256]) with d 64 or 128: blocked
// MFMA factorisation of N held block-packed in LDS, one 8-wave block per unit.
// npart holds S3 Gram partials per unit; it may be gram itself when S3 is 1
// (each element is read before the same thread overwrites it with N).
bool solve_big_supported(const Plan& p);
hipError_t launch_solve_big(const Plan& p, const float* npart, int S3, const float* y,
                            const float* resid, float* gram, float* z, float* stats_ws,
                            float* stats_user, hipStream_t s);
// v_out = V0 + X_G^T Z over every retained slot from the stored X [U][mp][c],
// Z^T and the compact V0 copy v0c (input dtype), for the generic value step
// (any dtype, mp up to 256, d 64/128); fixed slots and singular units get V0.
hipError_t launch_update_gen(const Plan& p, const float* x, const uint8_t* fixed, const float* z,
                             const float* stats_ws, const void* v0c, float* v_out,
                             hipStream_t s);
hipError_t launch_update_add(const Plan& p, const float* x, const uint8_t* fixed,
                             const float* z, const float* stats_ws, float* v_out,
                             hipStream_t s);

// Key step (bf16 path, mp <= 128): conjugate gradients on the dual system of
// the linearized key ridge problem, then K* = K0 + J_G^T alpha.  Per-unit CG
// state values (cg[u][3], reported in cg_info[u][2] as the GRKV_KEY_* codes).
enum { kKeyRunning = 0, kKeyConverged = 1, kKeyMaxIter = 2, kKeySkipped = 3, kKeyBreakdown = 4 };

struct KeyPlan {
  int S4, chunk4;           // splits of the retained keys per unit, later CG iterations
  int S4r, chunk4r;         // the same for the ring passes (at most S4)
  int S_full, chunk_full;   // the same for the first iterations and the final pass
  size_t Fm, alpha, r, p, sdot, W, opart, hpart, cg;   // offsets after Plan::total
  // later alternating steps (steps > 1): fp32 copies of Q and V0, the compact
  // bf16 V0, X [U][mp][c] of the fp32 value step, the current keys
  size_t q32, v0f, v0c, x, kcur;
  // the ring kernel's pass (key_ring.hip) applies: V* as bf16 hi and lo
  // tensors [U][c][d] each, the X^T tiles [U][ceil(c / 32)][4096] (fp32)
  bool ring;
  size_t vsplit, xs;
  size_t total;
};

struct KeyArgs {
  const uint16_t* q;        // [U][m][d] window queries
  const uint16_t* k0;       // [U][c][d] retained keys K0
  const float* kcur;        // [U][c][d] current keys (fp32) at a later alternating step, or null (K0)
  const float* vs;          // [U][c][d] merged values V*
  uint16_t* vh;             // [U][c][d] V* hi and lo (bf16), or null: the
  uint16_t* vl;             // ring kernel's pass is not used
  float* xs;                // [U][ceil(c / 32)][4096] X^T tiles (ring kernel)
  const float* lse2;        // [U][mp] retained log-sum-exp (log2 domain)
  const uint8_t* fixed;     // [U][c]
  const int32_t* idx;       // [U][c] retained positions
  const float* y;           // [U][mp][d] Y
  const float* zt;          // [U][d][mp] Z^T of the value step
  const float* stats_ws;    // [U][4] value-step stats (status in [3])
  float *Fm, *alpha, *r, *p, *W, *opart, *hpart;
  float* sdot;              // [U][mp] rowdot(F, p) of the current direction
  double* cg;               // [U][4] {r.r, r0.r0, iterations, state}
  float* kstar;             // [U][c][d] out
  float* cg_info;           // [U][4] out or null
  float lam_k, tol;
  int max_iter;
};

bool key_supported(const Plan& p);
hipError_t launch_key(const Plan& p, const KeyPlan& kp, const KeyArgs& a, hipStream_t s);
// Key-pass ring kernel (mp = 128, d = 128, bf16, first alternating step):
// V* split into bf16 hi/lo and the retained-set softmax X written as tiles
// once per key step (key_prep), then the operator (final = false, direction
// dir) or final (dir = alpha) pass over S splits.
bool key_ring_supported(const Plan& p);
size_t key_x_bytes(const Plan& p);
hipError_t launch_key_prep(const Plan& p, const KeyArgs& a, hipStream_t s);
hipError_t launch_key_ring(const Plan& p, const KeyArgs& a, bool final, int S, int chunk,
                           float* dir, bool fuse, hipStream_t s);
hipError_t launch_to_f32(const uint16_t* src, float* dst, size_t n, hipStream_t s);

// H2O accumulated-attention scores (bf16, d 64/128, G in {1, 2, 4, 8}): row
// log-sum-exps of every prompt position into lse2 [U][G][n], then the prefix
// column sums into scores [U][P].
bool h2o_supported(int dtype, int d, int G);
hipError_t launch_h2o(const void* q_all, const void* K, int U, int G, int d, int64_t n, int P,
                      float* lse2, float* scores, hipStream_t s);

// Adaptive per-head budgets: one block per layer of H adjacent units.
hipError_t launch_adaptive_budgets(const float* pooled, int layers, int H, int P, int64_t kk,
                                   int w, int32_t* budgets, hipStream_t s);

// Carrier-concentration diagnostics (bf16 keys, d 64/128, c <= 8192).
bool carrier_supported(int dtype, int d, int c);
hipError_t launch_carrier(const void* K, const int32_t* idx, int U, int64_t n, int c, int d,
                          const float* stats, int32_t* assign, int32_t* counts, float* metrics,
                          float* l_common, hipStream_t s);

}  // namespace grkv
