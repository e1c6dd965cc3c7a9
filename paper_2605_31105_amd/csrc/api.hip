// Host side of the C ABI: argument checks, the workspace plans and the launch
// sequences of grkv_compress, the key step (grkv_compress_kv), ragged budgets
// and the budget rules, and the carrier diagnostics.  Everything is enqueued
// on the caller's stream; the only host-to-device transfer is the ragged
// call's copy of its per-unit table.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "grkv_internal.h"

namespace grkv {

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Split a key range of length len over at most `want` blocks of >= min_len keys,
// each a whole number of key tiles.
static void split_range(int64_t len, int64_t want, int64_t min_len, int* S, int* chunk) {
  int64_t s = want < 1 ? 1 : want;
  int64_t cap = ceil_div(len, min_len);
  if (s > cap) s = cap;
  if (s < 1) s = 1;
  int64_t ch = ceil_div(len, s);
  ch = ceil_div(ch, kKeyTile) * kKeyTile;
  if (ch < kKeyTile) ch = kKeyTile;
  *chunk = (int)ch;
  *S = (int)(len > 0 ? ceil_div(len, ch) : 1);
}

static void layout_plan(Plan* p, size_t slots, size_t splits2, size_t splits3, size_t tab);

int make_plan(const grkv_problem* prob, int64_t n, int32_t window, int32_t budget,
              int32_t pool_kernel, float lambda, const grkv_options* opt, Plan* p) {
  if (!prob) return GRKV_ERR_INVALID;
  if (prob->units < 1 || prob->group < 1) return GRKV_ERR_INVALID;
  if (prob->dtype != GRKV_BF16 && prob->dtype != GRKV_F32) return GRKV_ERR_INVALID;
  if (window < 1 || budget < window || (int64_t)budget > n || n > (int64_t(1) << 30))
    return GRKV_ERR_INVALID;
  if (pool_kernel < 1 || pool_kernel % 2 == 0) return GRKV_ERR_INVALID;
  if (!(lambda >= 0.f) || !isfinite(lambda)) return GRKV_ERR_INVALID;
  grkv_options o;
  grkv_default_options(&o);
  if (opt) o = *opt;
  if (o.n_sink < 0 || !(o.beta >= 0.f && o.beta <= 1.f)) return GRKV_ERR_INVALID;
  if (prob->head_dim != 64 && prob->head_dim != 128) return GRKV_ERR_UNSUPPORTED;
  int64_t m = (int64_t)prob->group * window;
  if (m > 256) return GRKV_ERR_UNSUPPORTED;

  memset(p, 0, sizeof(*p));
  p->U = prob->units;
  p->G = prob->group;
  p->w = window;
  p->m = (int)m;
  // one wave per 32 rows, a power of two of them (1, 2, 4 or 8)
  int waves = 1;
  while (waves * kRowsPerWave < m) waves *= 2;
  p->waves = waves;
  p->mp = waves * kRowsPerWave;
  p->d = prob->head_dim;
  p->dtype = prob->dtype;
  p->n = n;
  p->c = budget;
  p->s_sel = budget - window;
  p->prefix = (int)(n - window);
  p->k_pool = pool_kernel;
  int64_t top = (int64_t)floor((double)o.beta * (double)budget);
  p->n_top_fixed = (int)(top < p->s_sel ? top : p->s_sel);
  p->lam = lambda;
  p->opt = o;

  // Target about 1024 blocks per launch (four per CU) for the full-cache
  // streaming passes, and about one block per CU for the bf16 retained pass
  // (which holds one block per CU): fewer splits mean fewer partials for the
  // solve to combine.
  int64_t target = 1024, target_ret = 256;
  if (const char* e = getenv("GRKV_TARGET_BLOCKS")) target = atoll(e);       // tuning experiments
  if (const char* e = getenv("GRKV_TARGET_RET_BLOCKS")) target_ret = atoll(e);
  const int64_t want = ceil_div(target, p->U);
  split_range(n, want, 512, &p->S1, &p->chunk1);
  p->fast_merge = merge_fast_supported(*p);
  if (p->fast_merge) {
    split_range(budget, ceil_div(target_ret, p->U), 128, &p->S2, &p->chunk2);
    if (p->chunk2 > 4096) split_range(budget, ceil_div(budget, 4096), 128, &p->S2, &p->chunk2);
  } else {
    split_range(budget, want, 128, &p->S2, &p->chunk2);
    if (p->chunk2 > 8192) split_range(budget, ceil_div(budget, 8192), 128, &p->S2, &p->chunk2);
  }
  // calls with few units split the solve's right-hand-side columns over up
  // to d / 16 blocks per unit (one per compute unit at most)
  p->csplit = 1;
  if (p->fast_merge && (size_t)p->U * (p->d / 16) <= 256) p->csplit = p->d / 16;
  if (p->fast_merge) {
    p->S3 = p->S2;
    p->chunk3 = p->chunk2;
  } else {
    split_range(budget, ceil_div(256, p->U), 256, &p->S3, &p->chunk3);
  }

  layout_plan(p, (size_t)p->U * budget, (size_t)p->U * p->S2, (size_t)p->U * p->S3, 0);
  return GRKV_OK;
}

// Workspace offsets: `slots` retained slots and `splits2` / `splits3`
// retained-pass and Gram partial blocks over all units, then `tab` bytes of
// ragged tables.
static void layout_plan(Plan* p, size_t slots, size_t splits2, size_t splits3, size_t tab) {
  const size_t U = p->U, mp = p->mp, d = p->d, P = p->prefix;
  const size_t esz = p->dtype == GRKV_BF16 ? 2 : 4;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o2 = off; off = align256(off + bytes); return o2; };
  p->pmax1 = take(U * p->S1 * mp * sizeof(float));
  p->psum1 = take(U * p->S1 * mp * sizeof(double));
  p->lse1 = take(U * mp * sizeof(double));
  p->lse1_log2 = take(U * mp * sizeof(float));
  p->ypart = take(U * p->S1 * mp * d * sizeof(float));
  p->y = take(U * mp * d * sizeof(float));
  p->colsum = take(U * (P > 0 ? P : 1) * sizeof(float));
  p->pooled = take(U * (P > 0 ? P : 1) * sizeof(float));
  p->fixed = take(slots);
  p->redo = take(U * p->S1 * sizeof(int32_t));
  // the compact V0 copy serves the generic retained passes only; the fast
  // path reads V0 rows through idx
  const bool fast_path = stream_supported(*p) && merge_fast_supported(*p);
  p->v0c = take(fast_path ? 0 : slots * d * esz);
  p->pmax2 = take(splits2 * mp * sizeof(float));
  p->psum2 = take(splits2 * mp * sizeof(double));
  p->lse2 = take(U * mp * sizeof(double));
  p->lse2_log2 = take(U * mp * sizeof(float));
  p->xvpart = take(splits2 * mp * d * sizeof(float));
  p->x = take(p->fast_merge ? 0 : mp * slots * sizeof(float));   // generic path only
  p->resid = take(U * mp * d * sizeof(float));
  p->npart = take(splits3 * mp * mp * sizeof(float));
  p->mpart = take(fast_path ? splits2 * mp * sizeof(float) : 0);
  const size_t comb = fast_path && p->S2 >= kPrecombineRetSplits ? U : 0;
  p->xvcomb = take(comb * mp * d * sizeof(float));
  p->ncomb = take(comb * mp * mp * sizeof(float));
  p->mcomb = take(comb * mp * sizeof(float));
  p->gram = take(U * mp * mp * sizeof(float));
  p->z = take(U * d * mp * sizeof(float));
  p->zhi = take(U * d * mp * 2);
  p->zlo = take(U * d * mp * 2);
  p->stats_ws = take(U * 4 * sizeof(float));
  p->zpart = take(U * kZParts * sizeof(double));
  p->rag_tab = take(tab);
  p->total = off;
}

// Workspace of the key step, after the compress workspace.  A key-pass block
// holds all m rows of a unit and a split of its retained keys.
static void make_key_plan(const Plan& p, int steps, KeyPlan* kp) {
  // about 256 blocks (one per compute unit) while every unit is iterating;
  // about 2048 later, when a unit's iteration spanning several compute units
  // keeps it short once only a few units are still converging
  split_range(p.c, ceil_div(256, p.U), 64, &kp->S_full, &kp->chunk_full);
  split_range(p.c, ceil_div(2048, p.U), 64, &kp->S4, &kp->chunk4);
  // the ring passes' later iterations: about 1024 blocks (fewer partials for
  // the separate CG update to combine, measured faster than 2048)
  split_range(p.c, ceil_div(1024, p.U), 64, &kp->S4r, &kp->chunk4r);
  const int Smax = kp->S4 > kp->S_full ? kp->S4 : kp->S_full;
  const size_t U = p.U, mp = p.mp, d = p.d;
  size_t off = p.total;
  auto take = [&](size_t bytes) { size_t o2 = off; off = align256(off + bytes); return o2; };
  kp->Fm = take(U * mp * d * sizeof(float));
  kp->alpha = take(U * mp * d * sizeof(float));
  kp->r = take(U * mp * d * sizeof(float));
  kp->p = take(U * mp * d * sizeof(float));
  kp->sdot = take(U * mp * sizeof(float));
  kp->W = take(U * mp * mp * sizeof(float));
  kp->opart = take(U * Smax * mp * d * sizeof(float));
  kp->hpart = take(U * Smax * mp * sizeof(float));
  kp->cg = take(U * 4 * sizeof(double));
  const size_t later = steps > 1 ? 1 : 0;
  kp->q32 = take(later * U * p.m * d * sizeof(float));
  kp->v0f = take(later * U * p.c * d * sizeof(float));
  kp->v0c = take(later * U * p.c * d * sizeof(uint16_t));
  kp->x = take(later * U * mp * p.c * sizeof(float));
  kp->kcur = take(later * U * p.c * d * sizeof(float));
  kp->ring = key_ring_supported(p);
  kp->vsplit = take(kp->ring ? 2 * U * p.c * d * sizeof(uint16_t) : 0);
  kp->xs = take(kp->ring ? key_x_bytes(p) : 0);
  kp->total = off;
}

}  // namespace grkv

using namespace grkv;

extern "C" {

void grkv_default_options(grkv_options* opt) {
  if (!opt) return;
  opt->n_sink = 4;
  opt->beta = 0.10f;
  opt->fix_window = 1;
  opt->causal_window = 1;
}

const char* grkv_status_string(int status) {
  switch (status) {
    case GRKV_OK: return "ok";
    case GRKV_ERR_INVALID: return "invalid argument";
    case GRKV_ERR_WORKSPACE: return "workspace too small";
    case GRKV_ERR_UNSUPPORTED: return "unsupported shape (head_dim must be 64 or 128, group*window <= 256)";
    case GRKV_ERR_HIP: return "HIP launch failed";
  }
  return "unknown status";
}

size_t grkv_workspace_bytes(const grkv_problem* prob, int64_t n, int32_t window, int32_t budget) {
  Plan p;
  if (make_plan(prob, n, window, budget, 1, 0.f, nullptr, &p) != GRKV_OK) return 0;
  return p.total;
}

int grkv_workspace_layout(const grkv_problem* prob, int64_t n, int32_t window, int32_t budget,
                          grkv_layout* layout) {
  if (!layout) return GRKV_ERR_INVALID;
  Plan p;
  int st = make_plan(prob, n, window, budget, 1, 0.f, nullptr, &p);
  if (st != GRKV_OK) return st;
  layout->lse = p.lse1;
  layout->y = p.y;
  layout->score = p.colsum;
  layout->pooled = p.pooled;
  layout->fixed = p.fixed;
  layout->resid = p.resid;
  layout->gram = p.gram;
  layout->z = p.z;
  layout->total = p.total;
  return GRKV_OK;
}

}  // extern "C"

namespace {

// Pointer checks shared by the entry points.
int check_pointers(const void* q_obs, const void* K, const void* V, const grkv_problem* prob,
                   const grkv_outputs* out) {
  if (!q_obs || !K || !V || !prob || !out) return GRKV_ERR_INVALID;
  if (!out->idx || !out->k_out || !out->v_out || !out->workspace) return GRKV_ERR_INVALID;
  if (((uintptr_t)out->workspace & 255) != 0) return GRKV_ERR_INVALID;
  return GRKV_OK;
}

// The launch sequence of one call (arguments already checked).
int run_compress(const Plan& p, const void* q_obs, const void* K, const void* V, int64_t n,
                 hipStream_t s, const grkv_outputs* out, const float* ext_scores = nullptr) {
  char* ws = (char*)out->workspace;
  auto F = [&](size_t o) { return (float*)(ws + o); };
  auto Dd = [&](size_t o) { return (double*)(ws + o); };

#define GRKV_TRY(x) do { if ((x) != hipSuccess) return GRKV_ERR_HIP; } while (0)
  void** ev = out->stage_events;
  auto mark = [&](int stage, int end) -> hipError_t {
    if (!ev || !ev[2 * stage] || !ev[2 * stage + 1]) return hipSuccess;
    return hipEventRecord((hipEvent_t)ev[2 * stage + end], s);
  };
#define GRKV_STAGE(id, call) do { GRKV_TRY(mark(id, 0)); GRKV_TRY(call); GRKV_TRY(mark(id, 1)); } while (0)
  // 1. window attention over the full cache: LSE, then Y and the SnapKV scores
  AttnPass full = {};
  full.q = q_obs; full.k = K; full.v = V; full.kpos = nullptr; full.nk = (int)n;
  full.S = p.S1; full.chunk = p.chunk1;
  full.pmax = F(p.pmax1); full.psum = Dd(p.psum1);
  full.lse = Dd(p.lse1); full.lse_log2 = F(p.lse1_log2);
  // (with caller-supplied selection scores the window's column sums are not formed)
  full.ypart = F(p.ypart); full.colsum = p.prefix > 0 && !ext_scores ? F(p.colsum) : nullptr;
  full.prefix = p.prefix; full.xout = nullptr; full.split_p = true;
  full.redo = (int*)(ws + p.redo);
  const bool fast = stream_supported(p);
  auto pass_a = [&](const AttnPass& a) { return fast ? launch_stream(p, a, 0, s) : launch_lse_pass(p, a, s); };
  auto pass_b = [&](const AttnPass& a) { return fast ? launch_stream(p, a, 1, s) : launch_prob_pass(p, a, s); };
  GRKV_STAGE(GRKV_STAGE_FULL_LSE, pass_a(full));
  // (the bf16 streaming pass B combines the split partials itself, unless a
  // unit has so many splits that a kernel of its own does it faster)
  const bool pre = fast && p.fast_merge && p.S1 >= kPrecombineSplits;
  full.lse_ready = pre;
  if (!fast || pre)
    GRKV_STAGE(GRKV_STAGE_FULL_LSE_COMBINE,
               launch_lse_combine(p, full.pmax, full.psum, p.S1, Dd(p.lse1), F(p.lse1_log2), s));
  GRKV_STAGE(GRKV_STAGE_FULL_PROB, pass_b(full));
  // (the fast value step combines the Y partials inside its solve, again
  // unless there are many)
  // (with many retained splits too, the Y partials join the retained
  // partials' combine below: one launch for both)
  const bool pre2 = fast && p.fast_merge && !p.rag && p.S2 >= kPrecombineRetSplits;
  if (!p.fast_merge || (pre && !pre2))
    GRKV_STAGE(GRKV_STAGE_FULL_Y, launch_combine_rows(p, F(p.ypart), p.S1, nullptr, F(p.y), s));
  // 2. pooled top-k retention and the fixed set; gather K0, V0
  uint8_t* fixed = (uint8_t*)(ws + p.fixed);
  GRKV_STAGE(GRKV_STAGE_SELECT, launch_select(p, ext_scores ? ext_scores : F(p.colsum), F(p.pooled),
                                              out->idx, fixed, s));
  const bool fast_merge = p.fast_merge;
  // fast path: the retained pass A reads the K rows through idx and copies
  // them to k_out; V0 rows are read through idx where needed
  const bool direct = fast && fast_merge;
  if (!direct)
    GRKV_STAGE(GRKV_STAGE_GATHER, launch_gather(p, K, V, out->idx, out->k_out, ws + p.v0c,
                                                nullptr, s));
  // 3. window attention over the retained cache: X and X V0, then R = Y - X V0
  AttnPass ret = {};
  ret.q = q_obs; ret.k = out->k_out; ret.v = ws + p.v0c; ret.kpos = out->idx; ret.nk = p.c;
  ret.S = p.S2; ret.chunk = p.chunk2;
  ret.pmax = F(p.pmax2); ret.psum = Dd(p.psum2);
  ret.lse = Dd(p.lse2); ret.lse_log2 = F(p.lse2_log2);
  ret.ypart = F(p.xvpart); ret.colsum = nullptr; ret.prefix = 0;
  ret.xout = fast_merge ? nullptr : F(p.x);
  ret.split_p = true;
  ret.fixed = fixed; ret.npart = F(p.npart);
  if (direct) {
    // one pass over the retained set: K and V rows through idx (K tiles also
    // copied to k_out), P against the full-cache LSE; the solve normalises by
    // the retained row sums, so no retained log-sum-exp pass is needed
    ret.k = K; ret.gather_k = true; ret.kcopy = out->k_out;
    ret.v = V; ret.gather_v = true; ret.src_rows = n;
    ret.lse_log2 = F(p.lse1_log2); ret.lse_bias = kRetainedBias; ret.mpart = F(p.mpart);
  } else {
    GRKV_STAGE(GRKV_STAGE_RET_LSE, pass_a(ret));
    GRKV_STAGE(GRKV_STAGE_RET_LSE_COMBINE,
               launch_lse_combine(p, ret.pmax, ret.psum, p.S2, Dd(p.lse2), F(p.lse2_log2), s));
  }
  // the generic value step needs X itself, which only the generic pass writes
  GRKV_STAGE(GRKV_STAGE_RET_PROB,
             fast_merge ? launch_stream(p, ret, 2, s) : launch_prob_pass(p, ret, s));
  if (!fast_merge)
    GRKV_STAGE(GRKV_STAGE_RESID,
               launch_combine_rows(p, F(p.xvpart), p.S2, F(p.y), F(p.resid), s));
  // 4. value step: N, Cholesky solve for Z, V* = V0 + X_G^T Z
  if (!fast_merge) GRKV_STAGE(GRKV_STAGE_GRAM, launch_gram(p, F(p.x), fixed, F(p.npart), s));
  if (fast_merge) {
    // many retained splits per unit (small uniform calls): their partials are
    // summed by one launch over all units first
    if (pre2) {
      const float* part[kCombineSegs] = {F(p.xvpart), F(p.npart), F(p.mpart), F(p.ypart)};
      float* const outs[kCombineSegs] = {F(p.xvcomb), F(p.ncomb), F(p.mcomb), F(p.y)};
      const size_t per[kCombineSegs] = {(size_t)p.mp * p.d, (size_t)p.mp * p.mp, (size_t)p.mp,
                                        pre ? (size_t)p.mp * p.d : 0};
      const int S[kCombineSegs] = {p.S2, p.S2, p.S2, p.S1};
      GRKV_STAGE(GRKV_STAGE_RESID, launch_combine_parts(p.U, S, part, outs, per, s));
    }
    GRKV_TRY(mark(GRKV_STAGE_SOLVE, 0));
    GRKV_TRY(launch_solve(p, pre ? F(p.y) : F(p.ypart), pre ? 1 : p.S1, pre2 ? 1 : p.S2,
                          pre2 ? F(p.xvcomb) : F(p.xvpart), pre2 ? F(p.ncomb) : F(p.npart),
                          direct ? (pre2 ? F(p.mcomb) : F(p.mpart)) : nullptr, F(p.lse1_log2),
                          kRetainedBias, F(p.lse2_log2), F(p.y), F(p.resid), F(p.gram), F(p.z),
                          (uint16_t*)(ws + p.zhi), (uint16_t*)(ws + p.zlo), F(p.stats_ws),
                          out->stats, Dd(p.zpart), q_obs, out->k_out, V, out->idx, fixed, s));
    GRKV_TRY(mark(GRKV_STAGE_SOLVE, 1));
    GRKV_STAGE(GRKV_STAGE_UPDATE,
               launch_update(p, q_obs, out->k_out, F(p.lse2_log2), fixed,
                             (const uint16_t*)(ws + p.zhi),
                             (const uint16_t*)(ws + p.zlo), F(p.stats_ws),
                             V, out->idx, out->v_out, Dd(p.zpart), out->stats, s));
  } else {
    // 256 stacked rows: blocked MFMA factorisation (block-packed in LDS);
    // otherwise the column-by-column one
    if (solve_big_supported(p)) {
      // the Gram partials summed over all units first (one wide launch, in
      // split order: the solve's own sum, spread over the GPU), into gram,
      // which the solve then reads and overwrites with N
      const float* Np = F(p.npart);
      int S3 = p.S3;
      GRKV_TRY(mark(GRKV_STAGE_SOLVE, 0));
      if (S3 > 1) {
        const float* part[kCombineSegs] = {F(p.npart), nullptr, nullptr, nullptr};
        float* const outs[kCombineSegs] = {F(p.gram), nullptr, nullptr, nullptr};
        const size_t per[kCombineSegs] = {(size_t)p.mp * p.mp, 0, 0, 0};
        const int Sc[kCombineSegs] = {p.S3, 0, 0, 0};
        GRKV_TRY(launch_combine_parts(p.U, Sc, part, outs, per, s));
        Np = F(p.gram);
        S3 = 1;
      }
      GRKV_TRY(launch_solve_big(p, Np, S3, F(p.y), F(p.resid), F(p.gram), F(p.z), F(p.stats_ws),
                                out->stats, s));
      GRKV_TRY(mark(GRKV_STAGE_SOLVE, 1));
    } else {
      GRKV_STAGE(GRKV_STAGE_SOLVE, launch_cholesky_solve(p, F(p.npart), F(p.y), F(p.resid),
                                                         F(p.gram), F(p.z), F(p.stats_ws),
                                                         out->stats, s));
    }
    GRKV_STAGE(GRKV_STAGE_UPDATE,
               launch_update_gen(p, F(p.x), fixed, F(p.z), F(p.stats_ws), ws + p.v0c,
                                 out->v_out, s));
  }
#undef GRKV_STAGE
#undef GRKV_TRY
  return GRKV_OK;
}

}  // namespace

extern "C" {

int grkv_compress(const void* q_obs, const void* K, const void* V, int64_t n, int32_t window,
                  int32_t budget, int32_t pool_kernel, float lambda, void* stream,
                  const grkv_problem* prob, const grkv_options* opt, const grkv_outputs* out) {
  int st = check_pointers(q_obs, K, V, prob, out);
  if (st != GRKV_OK) return st;
  Plan p;
  st = make_plan(prob, n, window, budget, pool_kernel, lambda, opt, &p);
  if (st != GRKV_OK) return st;
  if (out->workspace_bytes < p.total) return GRKV_ERR_WORKSPACE;
  return run_compress(p, q_obs, K, V, n, (hipStream_t)stream, out);
}

int grkv_compress_scored(const void* q_obs, const void* K, const void* V, int64_t n,
                         int32_t window, int32_t budget, int32_t pool_kernel, float lambda,
                         void* stream, const grkv_problem* prob, const grkv_options* opt,
                         const float* scores, const grkv_outputs* out) {
  int st = check_pointers(q_obs, K, V, prob, out);
  if (st != GRKV_OK) return st;
  if (!scores && n > window) return GRKV_ERR_INVALID;
  Plan p;
  st = make_plan(prob, n, window, budget, pool_kernel, lambda, opt, &p);
  if (st != GRKV_OK) return st;
  if (out->workspace_bytes < p.total) return GRKV_ERR_WORKSPACE;
  return run_compress(p, q_obs, K, V, n, (hipStream_t)stream, out, scores);
}

size_t grkv_h2o_workspace_bytes(const grkv_problem* prob, int64_t n) {
  if (!prob || prob->units < 1 || prob->group < 1 || n < 1 || n > (int64_t(1) << 30)) return 0;
  if (!h2o_supported(prob->dtype, prob->head_dim, prob->group)) return 0;
  return (size_t)prob->units * prob->group * (size_t)n * sizeof(float);
}

int grkv_h2o_scores(const void* q_all, const void* K, int64_t n, int32_t window, void* stream,
                    const grkv_problem* prob, float* scores, void* workspace,
                    size_t workspace_bytes) {
  if (!q_all || !K || !prob || !workspace || (!scores && n > window)) return GRKV_ERR_INVALID;
  if (prob->units < 1 || prob->group < 1) return GRKV_ERR_INVALID;
  if (prob->dtype != GRKV_BF16 && prob->dtype != GRKV_F32) return GRKV_ERR_INVALID;
  if (window < 1 || (int64_t)window > n || n > (int64_t(1) << 30)) return GRKV_ERR_INVALID;
  if (((uintptr_t)workspace & 255) != 0) return GRKV_ERR_INVALID;
  if (!h2o_supported(prob->dtype, prob->head_dim, prob->group)) return GRKV_ERR_UNSUPPORTED;
  if (workspace_bytes < grkv_h2o_workspace_bytes(prob, n)) return GRKV_ERR_WORKSPACE;
  if (launch_h2o(q_all, K, prob->units, prob->group, prob->head_dim, n, (int)(n - window),
                 (float*)workspace, scores, (hipStream_t)stream) != hipSuccess)
    return GRKV_ERR_HIP;
  return GRKV_OK;
}

void grkv_default_key_options(grkv_key_options* kopt, float lambda) {
  if (!kopt) return;
  kopt->lambda_k = lambda;
  kopt->max_iter = 64;
  kopt->tol = 1e-5f;
  kopt->steps = 1;
}

size_t grkv_workspace_bytes_kv(const grkv_problem* prob, int64_t n, int32_t window,
                               int32_t budget, int32_t steps) {
  Plan p;
  if (steps < 1 || steps > 16) return 0;
  if (make_plan(prob, n, window, budget, 1, 0.f, nullptr, &p) != GRKV_OK) return 0;
  if (!key_supported(p)) return 0;
  KeyPlan kp;
  make_key_plan(p, steps, &kp);
  return kp.total;
}

int grkv_compress_kv(const void* q_obs, const void* K, const void* V, int64_t n, int32_t window,
                     int32_t budget, int32_t pool_kernel, float lambda, void* stream,
                     const grkv_problem* prob, const grkv_options* opt, const grkv_outputs* out,
                     const grkv_key_options* kopt, float* k_star, float* cg_info) {
  int st = check_pointers(q_obs, K, V, prob, out);
  if (st != GRKV_OK) return st;
  if (!k_star) return GRKV_ERR_INVALID;
  grkv_key_options ko;
  grkv_default_key_options(&ko, lambda);
  if (kopt) ko = *kopt;
  if (!(ko.lambda_k >= 0.f) || !isfinite(ko.lambda_k)) return GRKV_ERR_INVALID;
  if (ko.max_iter < 0 || ko.max_iter > 4096 || !(ko.tol >= 0.f) || !isfinite(ko.tol))
    return GRKV_ERR_INVALID;
  if (ko.steps < 1 || ko.steps > 16) return GRKV_ERR_INVALID;
  Plan p;
  st = make_plan(prob, n, window, budget, pool_kernel, lambda, opt, &p);
  if (st != GRKV_OK) return st;
  if (!key_supported(p)) return GRKV_ERR_UNSUPPORTED;
  KeyPlan kp;
  make_key_plan(p, ko.steps, &kp);
  if (out->workspace_bytes < kp.total) return GRKV_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  st = run_compress(p, q_obs, K, V, n, s, out);
  if (st != GRKV_OK) return st;

  char* ws = (char*)out->workspace;
  auto F = [&](size_t o) { return (float*)(ws + o); };
  KeyArgs a = {};
  a.q = (const uint16_t*)q_obs;
  a.k0 = (const uint16_t*)out->k_out;
  a.vs = out->v_out;
  if (kp.ring) {
    a.vh = (uint16_t*)(ws + kp.vsplit);
    a.vl = a.vh + (size_t)p.U * p.c * p.d;
    a.xs = F(kp.xs);
  }
  a.lse2 = F(p.lse2_log2);
  a.fixed = (const uint8_t*)(ws + p.fixed);
  a.idx = out->idx;
  a.y = F(p.y);
  a.zt = F(p.z);
  a.stats_ws = F(p.stats_ws);
  a.Fm = F(kp.Fm);
  a.alpha = F(kp.alpha);
  a.r = F(kp.r);
  a.p = F(kp.p);
  a.sdot = F(kp.sdot);
  a.W = F(kp.W);
  a.opart = F(kp.opart);
  a.hpart = F(kp.hpart);
  a.cg = (double*)(ws + kp.cg);
  a.kstar = k_star;
  a.cg_info = cg_info;
  a.lam_k = ko.lambda_k;
  a.tol = ko.tol;
  a.max_iter = ko.max_iter;
  void** ev = out->stage_events;
  const bool timed = ev && ev[2 * GRKV_STAGE_KEY] && ev[2 * GRKV_STAGE_KEY + 1];
  if (timed && hipEventRecord((hipEvent_t)ev[2 * GRKV_STAGE_KEY], s) != hipSuccess)
    return GRKV_ERR_HIP;
  if (launch_key(p, kp, a, s) != hipSuccess) return GRKV_ERR_HIP;

  // Later alternating steps (Algorithm 1, S > 1): the value step at the
  // current fp32 keys K^(t) (still anchored at V0) on the generic fp32
  // kernels, then the key step linearized at K^(t).
  if (ko.steps > 1) {
    Plan p32 = p;
    p32.dtype = GRKV_F32;
    float* q32 = F(kp.q32);
    float* v0f = F(kp.v0f);
    float* kcur = F(kp.kcur);
    float* x = F(kp.x);
    const size_t vbytes = (size_t)p.U * p.c * p.d * sizeof(float);
    if (launch_to_f32((const uint16_t*)q_obs, q32, (size_t)p.U * p.m * p.d, s) != hipSuccess)
      return GRKV_ERR_HIP;
    if (launch_gather(p, K, V, out->idx, out->k_out, ws + kp.v0c, v0f, s) != hipSuccess)
      return GRKV_ERR_HIP;
    a.kcur = kcur;
    for (int t = 1; t < ko.steps; ++t) {
      if (hipMemcpyAsync(kcur, k_star, vbytes, hipMemcpyDeviceToDevice, s) != hipSuccess)
        return GRKV_ERR_HIP;
      AttnPass r = {};
      r.q = q32; r.k = kcur; r.v = v0f; r.kpos = out->idx; r.nk = p.c;
      r.S = p.S2; r.chunk = p.chunk2;
      r.pmax = F(p.pmax2); r.psum = (double*)(ws + p.psum2);
      r.lse = (double*)(ws + p.lse2); r.lse_log2 = F(p.lse2_log2);
      r.ypart = F(p.xvpart); r.colsum = nullptr; r.prefix = 0; r.xout = x; r.split_p = true;
      uint8_t* fixed = (uint8_t*)(ws + p.fixed);
      if (launch_lse_pass(p32, r, s) != hipSuccess ||
          launch_lse_combine(p32, r.pmax, r.psum, p.S2, (double*)(ws + p.lse2), F(p.lse2_log2),
                             s) != hipSuccess ||
          launch_prob_pass(p32, r, s) != hipSuccess ||
          launch_combine_rows(p32, F(p.xvpart), p.S2, F(p.y), F(p.resid), s) != hipSuccess ||
          launch_gram(p32, x, fixed, F(p.npart), s) != hipSuccess ||
          launch_cholesky_solve(p32, F(p.npart), F(p.y), F(p.resid), F(p.gram), F(p.z),
                                F(p.stats_ws), out->stats, s) != hipSuccess ||
          hipMemcpyAsync(out->v_out, v0f, vbytes, hipMemcpyDeviceToDevice, s) != hipSuccess ||
          launch_update_add(p32, x, fixed, F(p.z), F(p.stats_ws), out->v_out, s) != hipSuccess)
        return GRKV_ERR_HIP;
      if (launch_key(p, kp, a, s) != hipSuccess) return GRKV_ERR_HIP;
    }
  }
  if (timed && hipEventRecord((hipEvent_t)ev[2 * GRKV_STAGE_KEY + 1], s) != hipSuccess)
    return GRKV_ERR_HIP;
  return GRKV_OK;
}

int grkv_pyramid_budgets(int32_t layers, int32_t kv_heads, int32_t mean_budget, int32_t window,
                         int64_t n, float ratio, int32_t* budgets) {
  if (layers < 1 || kv_heads < 1 || !budgets || window < 1 || mean_budget < window ||
      (int64_t)mean_budget > n || !(ratio >= 0.f && ratio <= 1.f))
    return GRKV_ERR_INVALID;
  const int L = layers;
  int64_t* per = (int64_t*)malloc(sizeof(int64_t) * L);   // host scratch of the schedule
  if (!per) return GRKV_ERR_INVALID;
  if (L == 1) {
    per[0] = mean_budget;
  } else {
    const double top = (double)ratio * mean_budget, bot = (2.0 - (double)ratio) * mean_budget;
    int64_t sum = 0;
    for (int l = 0; l < L; ++l) {
      const double raw = bot + (top - bot) * (double)l / (double)(L - 1);
      int64_t b = (int64_t)floor(raw + 0.5);
      b = b < window ? window : b > n ? n : b;
      per[l] = b;
      sum += b;
    }
    // rounding remainder to the lowest layers, one token each, within [w, n]
    int64_t diff = (int64_t)L * mean_budget - sum;
    for (int i = 0; diff != 0 && i < 4 * L; ++i) {
      const int j = i % L;
      const int64_t step = diff > 0 ? 1 : -1;
      if (per[j] + step >= window && per[j] + step <= n) {
        per[j] += step;
        diff -= step;
      }
    }
  }
  for (int l = 0; l < L; ++l)
    for (int h = 0; h < kv_heads; ++h) budgets[(size_t)l * kv_heads + h] = (int32_t)per[l];
  free(per);
  return GRKV_OK;
}

int grkv_adaptive_budgets(const float* pooled, int32_t layers, int32_t kv_heads, int64_t n,
                          int32_t window, int32_t budget, void* stream, int32_t* budgets) {
  if (!pooled || !budgets || layers < 1 || kv_heads < 1 || window < 1 || budget < window ||
      (int64_t)budget > n)
    return GRKV_ERR_INVALID;
  if (kv_heads > 128) return GRKV_ERR_UNSUPPORTED;
  const int64_t P = n - window;
  if (P < 1 || (int64_t)kv_heads * P > (int64_t(1) << 31)) return GRKV_ERR_UNSUPPORTED;
  const int64_t kk = (int64_t)kv_heads * (budget - window);
  if (launch_adaptive_budgets(pooled, layers, kv_heads, (int)P, kk, window, budgets,
                              (hipStream_t)stream) != hipSuccess)
    return GRKV_ERR_HIP;
  return GRKV_OK;
}

// Native ragged plan (bf16 fast path): the budget-independent passes as for
// one budget; the retained pass in splits of one length over each unit's own
// budget, the update in blocks of one slot count, both as flat grids whose
// blocks find their unit in device tables.  `tab` receives the tables
// (RagUnit [U], the unit of every retained-pass split, the unit of every
// update block, then the two launch orders) for the caller to copy into the
// workspace.  *native is false
// when the shape takes the generic path (one call per run of equal budgets).
static int make_ragged_plan(const grkv_problem* prob, int64_t n, int32_t window,
                            const int32_t* budgets, int32_t pool_kernel, float lambda,
                            const grkv_options* opt, Plan* p, std::vector<int32_t>* tab,
                            bool* native) {
  *native = false;
  if (!prob || !budgets || prob->units < 1) return GRKV_ERR_INVALID;
  const int U = prob->units;
  int64_t sum = 0;
  int cmax = 0;
  for (int u = 0; u < U; ++u) {
    if (budgets[u] < window || (int64_t)budgets[u] > n || window < 1) return GRKV_ERR_INVALID;
    sum += budgets[u];
    cmax = budgets[u] > cmax ? budgets[u] : cmax;
  }
  if (sum > INT32_MAX) return GRKV_ERR_UNSUPPORTED;   // packed slot offsets are int32
  int cmean = (int)((sum + U / 2) / U);
  if (cmean < window) cmean = window;
  if (cmean > n) cmean = (int)n;
  const int st = make_plan(prob, n, window, cmean, pool_kernel, lambda, opt, p);
  if (st != GRKV_OK) return st;
  if (!(stream_supported(*p) && p->fast_merge)) return GRKV_OK;
  const int chunk = p->chunk2, spb = update_slots_per_block(*p, cmean);
  std::vector<int32_t> split_unit, upd_unit;
  tab->assign((size_t)8 * U, 0);
  int64_t off = 0;
  for (int u = 0; u < U; ++u) {
    const int c = budgets[u];
    RagUnit r;
    r.off = (int32_t)off;
    r.c = c;
    r.s0 = (int32_t)split_unit.size();
    r.ns = (c + chunk - 1) / chunk;
    const int64_t top = (int64_t)floor((double)p->opt.beta * (double)c);
    r.ntop = (int32_t)(top < c - window ? top : c - window);
    r.ub0 = (int32_t)upd_unit.size();
    r.nub = (c + spb - 1) / spb;
    r.pad = 0;
    split_unit.insert(split_unit.end(), r.ns, u);
    upd_unit.insert(upd_unit.end(), r.nub, u);
    memcpy(tab->data() + (size_t)8 * u, &r, sizeof(r));
    off += c;
  }
  p->rag_splits = (int)split_unit.size();
  p->rag_upd_blocks = (int)upd_unit.size();
  p->upd_spb = spb;
  // launch orders: splits (update blocks) by decreasing slot count, ties in
  // split order (a stable sort)
  auto order = [&](const std::vector<int32_t>& unit_of, int len, int first_of_unit) {
    std::vector<int32_t> o(unit_of.size()), size(unit_of.size());
    for (size_t f = 0; f < unit_of.size(); ++f) {
      const RagUnit* r = reinterpret_cast<const RagUnit*>(tab->data()) + unit_of[f];
      const int first = first_of_unit == 0 ? r->s0 : r->ub0;
      const int k = (int)f - first;
      const int rest = r->c - k * len;
      size[f] = rest < len ? rest : len;
      o[f] = (int32_t)f;
    }
    std::stable_sort(o.begin(), o.end(), [&](int32_t a, int32_t b) { return size[a] > size[b]; });
    return o;
  };
  const std::vector<int32_t> split_order = order(split_unit, chunk, 0);
  const std::vector<int32_t> upd_order = order(upd_unit, spb, 1);
  tab->insert(tab->end(), split_unit.begin(), split_unit.end());
  tab->insert(tab->end(), upd_unit.begin(), upd_unit.end());
  tab->insert(tab->end(), split_order.begin(), split_order.end());
  tab->insert(tab->end(), upd_order.begin(), upd_order.end());
  p->c = cmax;
  p->s_sel = cmax - window;
  layout_plan(p, (size_t)sum, split_unit.size(), split_unit.size(), tab->size() * sizeof(int32_t));
  *native = true;
  return GRKV_OK;
}

// Runs of consecutive units with one budget (generic path); the largest plan.
static int ragged_runs(const grkv_problem* prob, int64_t n, int32_t window,
                       const int32_t* budgets, int32_t pool_kernel, float lambda,
                       const grkv_options* opt, size_t* ws_max) {
  if (!prob || !budgets || prob->units < 1) return GRKV_ERR_INVALID;
  size_t mx = 0;
  for (int u0 = 0; u0 < prob->units;) {
    int u1 = u0 + 1;
    while (u1 < prob->units && budgets[u1] == budgets[u0]) ++u1;
    grkv_problem pr = *prob;
    pr.units = u1 - u0;
    Plan p;
    const int st = make_plan(&pr, n, window, budgets[u0], pool_kernel, lambda, opt, &p);
    if (st != GRKV_OK) return st;
    mx = p.total > mx ? p.total : mx;
    u0 = u1;
  }
  *ws_max = mx;
  return GRKV_OK;
}

size_t grkv_workspace_bytes_ragged(const grkv_problem* prob, int64_t n, int32_t window,
                                   const int32_t* budgets) {
  Plan p;
  std::vector<int32_t> tab;
  bool native = false;
  if (make_ragged_plan(prob, n, window, budgets, 1, 0.f, nullptr, &p, &tab, &native) != GRKV_OK)
    return 0;
  if (native) return p.total;
  size_t mx = 0;
  if (ragged_runs(prob, n, window, budgets, 1, 0.f, nullptr, &mx) != GRKV_OK) return 0;
  return mx;
}

int grkv_compress_ragged(const void* q_obs, const void* K, const void* V, int64_t n,
                         int32_t window, const int32_t* budgets, int32_t pool_kernel,
                         float lambda, void* stream, const grkv_problem* prob,
                         const grkv_options* opt, const grkv_outputs* out) {
  int st = check_pointers(q_obs, K, V, prob, out);
  if (st != GRKV_OK) return st;
  Plan rp;
  std::vector<int32_t> tab;
  bool native = false;
  st = make_ragged_plan(prob, n, window, budgets, pool_kernel, lambda, opt, &rp, &tab, &native);
  if (st != GRKV_OK) return st;
  if (native) {
    // one launch per stage over every unit; the tables go into the workspace
    // first (a pageable-memory copy: the host array is consumed on return)
    if (out->workspace_bytes < rp.total) return GRKV_ERR_WORKSPACE;
    char* ws = (char*)out->workspace;
    int32_t* dt = (int32_t*)(ws + rp.rag_tab);
    if (hipMemcpyAsync(dt, tab.data(), tab.size() * sizeof(int32_t), hipMemcpyHostToDevice,
                       (hipStream_t)stream) != hipSuccess)
      return GRKV_ERR_HIP;
    rp.rag = (const RagUnit*)dt;
    rp.rag_split_unit = dt + (size_t)8 * rp.U;
    rp.rag_upd_unit = rp.rag_split_unit + rp.rag_splits;
    rp.rag_split_order = rp.rag_upd_unit + rp.rag_upd_blocks;
    rp.rag_upd_order = rp.rag_split_order + rp.rag_splits;
    return run_compress(rp, q_obs, K, V, n, (hipStream_t)stream, out);
  }
  size_t need = 0;
  st = ragged_runs(prob, n, window, budgets, pool_kernel, lambda, opt, &need);
  if (st != GRKV_OK) return st;
  if (out->workspace_bytes < need) return GRKV_ERR_WORKSPACE;
  const size_t esz = prob->dtype == GRKV_BF16 ? 2 : 4;
  const size_t m = (size_t)prob->group * window, d = prob->head_dim;
  size_t off = 0;   // packed slot offset of unit u0
  for (int u0 = 0; u0 < prob->units;) {
    int u1 = u0 + 1;
    while (u1 < prob->units && budgets[u1] == budgets[u0]) ++u1;
    grkv_problem pr = *prob;
    pr.units = u1 - u0;
    Plan p;
    st = make_plan(&pr, n, window, budgets[u0], pool_kernel, lambda, opt, &p);
    if (st != GRKV_OK) return st;
    grkv_outputs o = *out;
    o.idx = out->idx + off;
    o.k_out = (char*)out->k_out + off * d * esz;
    o.v_out = out->v_out + off * d;
    o.stats = out->stats ? out->stats + (size_t)4 * u0 : nullptr;
    o.stage_events = nullptr;
    st = run_compress(p, (const char*)q_obs + (size_t)u0 * m * d * esz,
                      (const char*)K + (size_t)u0 * n * d * esz,
                      (const char*)V + (size_t)u0 * n * d * esz, n, (hipStream_t)stream, &o);
    if (st != GRKV_OK) return st;
    off += (size_t)(u1 - u0) * budgets[u0];
    u0 = u1;
  }
  return GRKV_OK;
}

int grkv_carrier_stats(const void* K, int64_t n, int32_t budget, const grkv_problem* prob,
                       const int32_t* idx, const float* stats, void* stream, int32_t* assign,
                       int32_t* counts, float* metrics, float* l_common) {
  if (!K || !prob || !idx || !assign || !metrics) return GRKV_ERR_INVALID;
  if (prob->units < 1 || prob->group < 1) return GRKV_ERR_INVALID;
  if (prob->dtype != GRKV_BF16 && prob->dtype != GRKV_F32) return GRKV_ERR_INVALID;
  if (budget < 1 || (int64_t)budget > n || n > (int64_t(1) << 30)) return GRKV_ERR_INVALID;
  if (!carrier_supported(prob->dtype, prob->head_dim, budget)) return GRKV_ERR_UNSUPPORTED;
  if (launch_carrier(K, idx, prob->units, n, budget, prob->head_dim, stats, assign, counts,
                     metrics, l_common, (hipStream_t)stream) != hipSuccess)
    return GRKV_ERR_HIP;
  return GRKV_OK;
}

}  // extern "C"
