/*
 * grkv.h - C ABI of the MI355X (gfx950) GRKV prefill-compression path.
 *
 * GRKV ("Global Regression for KV cache", arXiv 2605.31105) compresses each
 * (layer, KV head) slice of a prefilled KV cache in two stages:
 *
 *   1. SnapKV-style span retention.  The last w prompt queries (the surrogate
 *      query window, Sec. 3.2) attend to the whole cache; every prefix token
 *      is scored by the attention it receives from the window, the scores are
 *      pooled over a window of pool_kernel neighbouring tokens, and the
 *      budget - w best prefix tokens are kept together with the w window
 *      tokens (Sec. 1 and Sec. 2, SnapKV).
 *   2. The value step of the global ridge-regression merge (Eq. 6-8;
 *      Algorithm 1, value step; App. D.1 and D.3).  With X the window's
 *      attention over the retained keys and Y its attention output over the
 *      full cache (Eq. 4), the free retained values are moved to
 *      V*_G = V0_G + X_G^T (X_G X_G^T + lambda I_m)^-1 (Y - X V0),
 *      which minimises ||Y - X V||_F^2 + lambda ||V - V0||_F^2 over V_G.
 *      Fixed tokens (sinks, the window, the top beta of the retained set,
 *      Sec. 3.4 "Fixed tokens during optimization") keep their values.
 *      Keys are not moved: K* = K0.
 *
 * A "unit" is one (layer, KV head) slice; units are independent and are
 * processed in one batched call.  G query heads share each KV head (grouped
 * query attention); their windows are stacked into m = G*w rows, row
 * r = g*w + i holding query head g at window position i, which sits at token
 * position n - w + i.
 *
 * Memory: every pointer argument is DEVICE memory owned by the caller.  The
 * library allocates nothing and keeps no state between calls; calls with
 * distinct workspaces may run concurrently on different streams.
 * Calls are asynchronous on `stream`; results are valid once the stream has
 * been synchronised.  No exception crosses this interface.
 */
#ifndef GRKV_H
#define GRKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes.  Argument errors are found on the host before anything is
 * launched, and then nothing is written. */
typedef enum {
  GRKV_OK = 0,
  GRKV_ERR_INVALID = -1,     /* bad argument (null pointer, size out of range) */
  GRKV_ERR_WORKSPACE = -2,   /* workspace smaller than grkv_workspace_bytes() */
  GRKV_ERR_UNSUPPORTED = -3, /* valid but not built: head_dim not 64/128, m = G*w > 256 */
  GRKV_ERR_HIP = -4          /* a HIP launch failed */
} grkv_status;

/* Element type of q_obs, K, V and k_out. */
typedef enum { GRKV_BF16 = 0, GRKV_F32 = 1 } grkv_dtype;

/* Per-unit status in stats[u][3]. */
#define GRKV_UNIT_OK 0
#define GRKV_UNIT_SINGULAR 1 /* non-positive Cholesky pivot: v_out holds V0 */
#define GRKV_UNIT_RANGE 2    /* internal: a window row's attention mass on the
                                retained keys is below 2^-108 of its full-cache
                                mass.  The bf16 path then redoes that unit's
                                value step against the retained set's own row
                                maxima, so a call never returns this code */

typedef struct {
  int32_t units;    /* U >= 1: number of (layer, KV head) slices */
  int32_t group;    /* G >= 1: query heads per KV head */
  int32_t head_dim; /* d: 64 or 128 */
  int32_t dtype;    /* grkv_dtype */
} grkv_problem;

/* Fixed-token and masking options.  NULL selects the defaults
 * {n_sink = 4, beta = 0.10f, fix_window = 1, causal_window = 1}:
 * the paper keeps sink tokens, the window tokens and the top 10% retained
 * tokens fixed (Sec. 4.1 hyperparameters). */
typedef struct {
  int32_t n_sink;        /* retained positions below n_sink stay fixed (>= 0) */
  float beta;            /* in [0, 1]: the first floor(beta * budget) prefix
                            tokens of the selection order stay fixed */
  int32_t fix_window;    /* nonzero: the w window tokens stay fixed */
  int32_t causal_window; /* nonzero: window row at position p sees keys 0..p only */
} grkv_options;

/* Outputs, all device memory owned by the caller, c = budget:
 *   idx   int32 [U][c]      retained positions, ascending; the last w entries
 *                           are n-w .. n-1.  Ties in the pooled score go to the
 *                           lower position.
 *   k_out dtype [U][c][d]   K0 = K[idx], bit-exact copies of the input rows
 *   v_out float [U][c][d]   merged values V*
 *   stats float [U][4]      {||Y||_F^2, D_before, D_after, unit status}, where
 *                           D = ||Y - X V||_F^2 / ||Y||_F^2 (the raw numerator
 *                           when ||Y|| = 0) with V = V0 and V = V*; may be NULL
 *   workspace               at least grkv_workspace_bytes() bytes, 256-byte
 *                           aligned; its contents on return are described by
 *                           grkv_workspace_layout(). */
typedef struct {
  int32_t* idx;
  void* k_out;
  float* v_out;
  float* stats;
  void* workspace;
  size_t workspace_bytes;
  /* Optional timing hooks, may be NULL: an array of 2 * GRKV_NUM_STAGES
   * hipEvent_t owned by the caller.  For every stage s whose two slots are both
   * non-null, slot 2s is recorded on `stream` before the stage's kernels and
   * slot 2s+1 after them, so hipEventElapsedTime gives the stage's duration. */
  void** stage_events;
} grkv_outputs;

/* Stages of one call, in launch order (indices into stage_events / 2).  A stage
 * that a given call does not run leaves its two events unrecorded: the bf16
 * path (head_dim 64/128, G*w <= 128) folds FULL_Y, RESID and GRAM into
 * neighbouring stages, reads the retained rows inside RET_PROB (no GATHER) and
 * forms the retained softmax from the full-cache log-sum-exp (no RET_LSE). */
enum {
  GRKV_STAGE_FULL_LSE = 0,     /* full-cache pass A: reference / sum-exp per split */
  GRKV_STAGE_FULL_LSE_COMBINE, /* -> log-sum-exp of every window row */
  GRKV_STAGE_FULL_PROB,        /* full-cache pass B: P.V partials, SnapKV column sums */
  GRKV_STAGE_FULL_Y,           /* -> Y */
  GRKV_STAGE_SELECT,           /* pooling, top-k, fixed set */
  GRKV_STAGE_GATHER,           /* K0 -> k_out, V0 (generic path) */
  GRKV_STAGE_RET_LSE,          /* retained-cache pass A (generic path) */
  GRKV_STAGE_RET_LSE_COMBINE,
  GRKV_STAGE_RET_PROB,         /* retained-cache pass B: X V0 (and on the bf16 path
                                  K0 -> k_out, Gram and retained-mass partials) */
  GRKV_STAGE_RESID,            /* R = Y - X V0 */
  GRKV_STAGE_GRAM,             /* N partials */
  GRKV_STAGE_SOLVE,            /* (Y, R, N combines,) Cholesky, Z, stats */
  GRKV_STAGE_UPDATE,           /* V* = V0 + X_G^T Z */
  GRKV_STAGE_KEY,              /* key step (grkv_compress_kv only): CG, K* */
  GRKV_NUM_STAGES
};

/* Compress U units.
 *   q_obs  dtype [U][G][w][d]  the window queries (post-RoPE), query head
 *                               kv_head*G + g of unit u at [u][g]
 *   K, V   dtype [U][n][d]     the full cache (post-RoPE keys)
 *   n            tokens per unit, w <= budget <= n, n <= 2^30
 *   window       w >= 1
 *   budget       c: retained tokens including the w window tokens
 *   pool_kernel  odd k >= 1: scores are summed over positions j-(k-1)/2 ..
 *                j+(k-1)/2 (zero outside the prefix) before ranking
 *   lambda       ridge coefficient lambda_v >= 0 (finite)
 *   stream       hipStream_t, NULL for the default stream
 * Errors: GRKV_ERR_INVALID for null pointers, units < 1, group < 1,
 * window < 1, budget < window, budget > n, even or < 1 pool_kernel,
 * negative or non-finite lambda, beta outside [0, 1], n_sink < 0, an unknown
 * dtype; GRKV_ERR_UNSUPPORTED for head_dim not in {64, 128} or G*w > 256;
 * GRKV_ERR_WORKSPACE when out->workspace_bytes is too small; GRKV_ERR_HIP
 * when a launch fails (outputs are then undefined). */
int grkv_compress(const void* q_obs, const void* K, const void* V, int64_t n,
                  int32_t window, int32_t budget, int32_t pool_kernel,
                  float lambda, void* stream, const grkv_problem* prob,
                  const grkv_options* opt, const grkv_outputs* out);

/* grkv_compress for callers that cannot allocate device memory (code under
 * stream capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same computation, kernels and arguments, but the workspace is a device array
 * of GRKV_NOALLOC_SCRATCH_BYTES held by the library on every device it runs on
 * (until the process ends); out->workspace and out->workspace_bytes are not
 * read.  The call runs on the current device (stream must belong to it) and
 * calls no allocating routine.  The first call on a device looks up the
 * array's address there.  Every call on one device shares that array: calls
 * that overlap on one device (several streams or host threads) race on it.
 * Nothing in it needs to start at zero.  Errors: those of grkv_compress;
 * GRKV_ERR_WORKSPACE when grkv_workspace_bytes() for the shape exceeds
 * GRKV_NOALLOC_SCRATCH_BYTES (64 MiB holds, for example, a one-layer call of
 * 8 KV heads, n = 32768, w = 32, budget 2048, d = 128: 54.5 MiB). */
#define GRKV_NOALLOC_SCRATCH_BYTES (64ull << 20)
int grkv_compress_noalloc(const void* q_obs, const void* K, const void* V, int64_t n,
                          int32_t window, int32_t budget, int32_t pool_kernel,
                          float lambda, void* stream, const grkv_problem* prob,
                          const grkv_options* opt, const grkv_outputs* out);

/* Key step of GRKV (Sec. 3.4 "Key step" and "Linearized dual solution",
 * Eq. 9-10; Algorithm 1, key step; App. D.2 and D.3), run by grkv_compress_kv
 * after the value step with the merged values V* held fixed and the keys at K0
 * (one alternating step, S = 1, the paper's default).  With f(K) =
 * softmax(Q K^T / sqrt(d)) V* over the retained keys, E = Y - f(K0) and J_G the
 * derivative of f with respect to the free keys, the free keys move to
 *   K*_G = K0_G + unvec(J_G^T alpha),
 *   alpha = (J_G J_G^T + lambda_k I_{md})^-1 vec(E),
 * which minimises ||E - J_G dK||^2 + lambda_k ||dK||^2; fixed keys keep K0.
 * The md x md system is solved matrix-free by conjugate gradients from
 * alpha = 0.  NULL options select {lambda_k = lambda, max_iter = 64,
 * tol = 1e-5f, steps = 1} (the paper uses lambda_k = lambda_v and does not
 * state its CG settings). */
typedef struct {
  float lambda_k;   /* ridge coefficient of the keys, >= 0 and finite */
  int32_t max_iter; /* conjugate-gradient iterations at most, 0 .. 4096 */
  float tol;        /* stop once ||r|| <= tol ||rhs|| (recursive residual), >= 0 */
  int32_t steps;    /* alternating value/key steps S, 1 .. 16 (Algorithm 1; the
                       paper's default and best setting is 1).  Step t > 1 takes
                       the value step at the current keys K^(t) (X from K^(t),
                       the update still anchored at V0) and the key step
                       linearized at K^(t), whose right-hand side gains
                       J_G (K^(t) - K0).  All S steps run (the paper's early
                       stop at a change <= 1e-9 is below fp32 resolution). */
} grkv_key_options;

/* Per-unit key-step outcome in cg_info[u][2]. */
#define GRKV_KEY_CONVERGED 1 /* the residual reached tol */
#define GRKV_KEY_MAX_ITER 2  /* max_iter iterations ran first */
#define GRKV_KEY_SKIPPED 3   /* the unit's value step reported a non-zero
                                status (stats[u][3]): K* = K0 */
#define GRKV_KEY_BREAKDOWN 4 /* a CG step found p^T A p <= 0 (possible only
                                for lambda_k = 0); the last iterate is kept */

/* grkv_compress followed by the key step (and, for steps > 1, further
 * alternating value and key steps).  All arguments as for grkv_compress; in
 * addition
 *   kopt     key-step options, or NULL for the defaults above
 *   k_star   float [U][c][d]   merged keys K*, device memory (required);
 *                              k_out still receives K0
 *   cg_info  float [U][4]      of the last key step: {CG iterations, final
 *                              ||r|| / ||rhs||, GRKV_KEY_* outcome, ||rhs||_F},
 *                              or NULL
 * v_out and stats hold the last value step.  out->workspace_bytes must be at
 * least grkv_workspace_bytes_kv() for the same number of steps.
 * Errors: those of grkv_compress; GRKV_ERR_INVALID for a null k_star or bad
 * kopt; GRKV_ERR_UNSUPPORTED unless dtype is bf16 and G*w <= 128. */
int grkv_compress_kv(const void* q_obs, const void* K, const void* V, int64_t n,
                     int32_t window, int32_t budget, int32_t pool_kernel,
                     float lambda, void* stream, const grkv_problem* prob,
                     const grkv_options* opt, const grkv_outputs* out,
                     const grkv_key_options* kopt, float* k_star, float* cg_info);

/* Workspace bytes grkv_compress_kv needs for `steps` alternating steps; 0 if
 * invalid or unsupported. */
size_t grkv_workspace_bytes_kv(const grkv_problem* prob, int64_t n,
                               int32_t window, int32_t budget, int32_t steps);

/* The default key options for a value ridge coefficient lambda. */
void grkv_default_key_options(grkv_key_options* kopt, float lambda);

/* Per-unit (ragged) budgets: the back-ends the paper pairs GRKV with (Sec. 4,
 * compatibility) differ in how much of the cache each unit keeps (PyramidKV
 * per layer, Ada-KV per head); the merge is unchanged.  grkv_compress_ragged
 * compresses unit u exactly as grkv_compress would with budget budgets[u]
 * (w <= budgets[u] <= n; the fixed set uses floor(beta * budgets[u])).
 *   budgets  int32 [U], HOST memory
 *   out      packed outputs: idx int32 [sum c_u], k_out dtype [sum c_u][d],
 *            v_out float [sum c_u][d], unit u starting at slot
 *            off_u = budgets[0] + ... + budgets[u-1]; stats [U][4] as before
 * On the bf16 path (d 64/128, group * window <= 128) every stage is one launch
 * over all units: a per-unit table (slot offset, budget, splits) is copied
 * into the workspace from host memory on `stream` first (the host array may
 * be reused once the call returns; a copy from pageable memory, so the call
 * is not for HIP graph capture), and out->stage_events is honoured as for
 * grkv_compress.  Other shapes run consecutive units of equal budget as one
 * grkv_compress batch each (out->stage_events ignored).  The workspace is
 * grkv_workspace_bytes_ragged(); errors as for grkv_compress, and
 * GRKV_ERR_UNSUPPORTED when the budgets sum past 2^31 - 1. */
int grkv_compress_ragged(const void* q_obs, const void* K, const void* V, int64_t n,
                         int32_t window, const int32_t* budgets, int32_t pool_kernel,
                         float lambda, void* stream, const grkv_problem* prob,
                         const grkv_options* opt, const grkv_outputs* out);

size_t grkv_workspace_bytes_ragged(const grkv_problem* prob, int64_t n, int32_t window,
                                   const int32_t* budgets);

/* Pyramid schedule (PyramidKV: lower layers keep more of the cache, higher
 * layers less): budgets fall linearly from (2 - ratio) * mean_budget at layer
 * 0 to ratio * mean_budget at the top layer, rounded to nearest, clipped to
 * [window, n], with the rounding remainder given to the lowest layers so that
 * the layers' mean stays mean_budget where the clip allows.  Every head of a
 * layer gets the layer's budget; units are layer-major (u = layer * kv_heads
 * + head).  budgets: int32 [layers * kv_heads], HOST memory.  ratio in [0, 1];
 * errors: GRKV_ERR_INVALID. */
int grkv_pyramid_budgets(int32_t layers, int32_t kv_heads, int32_t mean_budget, int32_t window,
                         int64_t n, float ratio, int32_t* budgets);

/* Adaptive per-head budgets (Ada-KV: heads that need long-range context keep
 * more): inside each layer the kv_heads heads share kv_heads * (budget - w)
 * selected tokens, taken as the highest pooled scores over all its heads (ties
 * to the lower head, then the lower position); head h gets w plus the number
 * of its tokens taken.  pooled: float [U][n - w] device memory, the pooled
 * scores of a grkv_compress call (grkv_workspace_layout().pooled); budgets:
 * int32 [U] device memory, written asynchronously on stream.  kv_heads <= 128.
 * The scores must be finite and non-negative (pooled attention masses are);
 * one block per layer selects by radix over their bit patterns.
 * Errors: GRKV_ERR_INVALID, GRKV_ERR_UNSUPPORTED, GRKV_ERR_HIP. */
int grkv_adaptive_budgets(const float* pooled, int32_t layers, int32_t kv_heads, int64_t n,
                          int32_t window, int32_t budget, void* stream, int32_t* budgets);

/* Token scores of H2O (Sec. 2: heavy-hitter tokens kept by accumulated
 * attention scores; Sec. 4.3, compatibility), the token-based eviction
 * back-end GRKV is paired with.  For unit u the score of prefix token j < n - w
 * is the attention it receives summed over every prompt position i >= j of
 * every query head g of the unit's group, each row being the causal softmax of
 * q_{g,i} . k / sqrt(d) over keys 0..i:
 *   s_j = sum_g sum_{i >= j} exp(q_{g,i} . k_j / sqrt(d) - LSE_{g,i}).
 *   q_all    dtype [U][G][n][d]  the queries of every prompt position (post-RoPE)
 *   K        dtype [U][n][d]
 *   scores   float [U][n - w]    out (device memory)
 *   workspace                    >= grkv_h2o_workspace_bytes(), 256-byte aligned
 * bf16 only, head_dim 64 or 128, group 1, 2, 4 or 8.  The cost is that of a
 * prefill attention without P.V (two passes of O(n^2 d) MFMA work per head).
 * Errors: GRKV_ERR_INVALID (null pointers, window outside [1, n], bad sizes),
 * GRKV_ERR_UNSUPPORTED, GRKV_ERR_WORKSPACE, GRKV_ERR_HIP.  Asynchronous on
 * stream; allocates nothing. */
int grkv_h2o_scores(const void* q_all, const void* K, int64_t n, int32_t window, void* stream,
                    const grkv_problem* prob, float* scores, void* workspace,
                    size_t workspace_bytes);

/* Workspace bytes of grkv_h2o_scores (the row log-sum-exps, U * G * n floats);
 * 0 if the shape is invalid or unsupported. */
size_t grkv_h2o_workspace_bytes(const grkv_problem* prob, int64_t n);

/* grkv_compress with the selection driven by caller-supplied per-token scores
 * instead of the window attention's column sums: the form a token-based
 * eviction front-end such as H2O (scores from grkv_h2o_scores, pool_kernel 1)
 * takes.  scores: float [U][n - w] device memory, finite and non-negative
 * (attention masses are), pooled with pool_kernel exactly as the column sums
 * would be; the top floor(beta * c) fixed subset follows the same order.  The
 * window attention, Y and the value step are those of grkv_compress.  All
 * other arguments, outputs, workspace and errors as for grkv_compress
 * (GRKV_ERR_INVALID also for a null scores when n > window). */
int grkv_compress_scored(const void* q_obs, const void* K, const void* V, int64_t n,
                         int32_t window, int32_t budget, int32_t pool_kernel, float lambda,
                         void* stream, const grkv_problem* prob, const grkv_options* opt,
                         const float* scores, const grkv_outputs* out);

/* Carrier concentration of a local merge rule (App. B, "Quantitative Carrier
 * Concentration"; Sec. 1): the diagnostic the paper uses to show that, after
 * span-based eviction, a key-similarity matcher (as in D2O/KVMerger) loads a
 * few span-boundary tokens with most of the evicted tokens.  Every evicted
 * token j is assigned to the retained slot i with the highest key cosine
 * similarity cos(k_j, k_idx[i]) over all retained tokens (equal values go to
 * the lower slot; a zero key has cosine 0 with all), and with a_i the number of
 * tokens assigned to slot i:
 *   K        dtype [U][n][d]  the full cache keys (bf16 only)
 *   idx      int32 [U][c]     ascending retained positions (grkv_compress)
 *   stats    float [U][4]     the stats of a grkv_compress call, or NULL
 *   assign   int32 [U][n]     out: slot of each evicted position, -1 for the
 *                             retained positions (required)
 *   counts   int32 [U][c]     out: a_i, or NULL
 *   metrics  float [U][8]     out: {b = #(a_i > 0), b_eff = (sum a)^2 / sum a^2,
 *                             A_max = max a / mean a, Gini of the a_i (mean
 *                             absolute difference over all pairs / twice the
 *                             mean), boundary fraction (first and last slots
 *                             of each run of consecutive positions, over c),
 *                             boundary share of the assignments, enrichment
 *                             (share / fraction), boundary / interior mean
 *                             load (NaN without both kinds; the load figures
 *                             are NaN when nothing is evicted)}
 *   l_common float [1]        out (needs stats): the discrepancy summed over the
 *                             units, sum D_after ||Y||^2 / sum ||Y||^2 (the
 *                             paper's L_common over these units), or NULL
 * Errors: GRKV_ERR_INVALID for null required pointers, units or group < 1, an
 * unknown dtype, budget outside [1, n]; GRKV_ERR_UNSUPPORTED for fp32 keys, d
 * not 64/128 or budget > 8192; GRKV_ERR_HIP for a failed launch.  Allocates
 * nothing; asynchronous on stream. */
int grkv_carrier_stats(const void* K, int64_t n, int32_t budget, const grkv_problem* prob,
                       const int32_t* idx, const float* stats, void* stream, int32_t* assign,
                       int32_t* counts, float* metrics, float* l_common);

/* Workspace bytes grkv_compress needs for this shape; 0 if the shape is
 * invalid or unsupported. */
size_t grkv_workspace_bytes(const grkv_problem* prob, int64_t n,
                            int32_t window, int32_t budget);

/* Byte offsets, inside the workspace, of intermediates that remain readable
 * after grkv_compress returns (mp = m rounded up to 32, 64, 128 or 256; rows
 * m..mp-1 are padding; P = n - w):
 *   lse      double [U][mp]     natural log-sum-exp of each window row over the
 *                               full cache (window attention normaliser)
 *   y        float  [U][mp][d]  Y = A V, the full-cache window attention output
 *   score    float  [U][P]      SnapKV score s_j = sum_r A[r][j]
 *   pooled   float  [U][P]      pooled score p_j
 *   fixed    uint8  [U][c]      1 where the retained slot is fixed
 *   resid    float  [U][mp][d]  R = Y - X V0
 *   gram     float  [U][mp][mp] N = X_G X_G^T + lambda I (padding rows: identity)
 *   z        float  [U][d][mp]  Z^T, Z = N^-1 R
 * Returns GRKV_OK, or GRKV_ERR_INVALID / GRKV_ERR_UNSUPPORTED like
 * grkv_compress. */
typedef struct {
  size_t lse, y, score, pooled, fixed, resid, gram, z;
  size_t total;
} grkv_layout;

int grkv_workspace_layout(const grkv_problem* prob, int64_t n, int32_t window,
                          int32_t budget, grkv_layout* layout);

/* The default options (see grkv_options). */
void grkv_default_options(grkv_options* opt);

/* Static description of a return code; never NULL. */
const char* grkv_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* GRKV_H */
