/*
 * caddtree.h -- C ABI of the CaDDTree draft-tree construction library (MI355X / gfx950).
 *
 * What it computes (Cost-Aware Diffusion Draft Trees for Speculative Decoding,
 * arXiv 2606.01813):  a speculative-decoding round starts from a block-diffusion
 * drafter's logits l_1 .. l_L over a vocabulary of V tokens.  Per round the
 * library
 *   1. forms the full-vocabulary log-normaliser LSE_i and the top-K tokens of
 *      every position i with log q_i^(k) = l_i^(k) - LSE_i (Sec. 3.2, eq.
 *      marginals; the Require line of Algorithm 1);
 *   2. grows the draft tree best-first by prefix probability pi_s =
 *      prod_i q_i(s_i) (eq. prefix-prob) and stops at the first budget n where
 *      theta*(n) = (1 + Phi*(n)) / (C_d + C_v(n)) (eq. per-round) stops rising
 *      (Algorithm 1; Lemma 1, eq. stopping; Cor. 2);
 *   3. lays the tree out breadth-first and emits its tree-attention mask
 *      (each node sees itself and its ancestors, Sec. 3.3) and position ids.
 *
 * Conventions shared by every entry point:
 *   - Device pointers are HIP device memory on the plan's device; host pointers
 *     are named *_host.  The caller owns every buffer; the library allocates
 *     nothing per call (a plan owns one small device copy of its cost tables
 *     and context-length grid).
 *   - All work is enqueued on the given stream and runs asynchronously; the
 *     return value reports argument validation (done synchronously, before
 *     anything is enqueued) and launch errors, not kernel completion.
 *   - A non-OK status enqueues nothing new; caddtree_last_error() gives a
 *     message (thread-local).  No C++ exception crosses this interface.
 *   - Logits must be finite; results for NaN or +-Inf inputs are unspecified.
 *   - Layouts are row-major.  B rounds, L positions, V vocabulary, K kept tokens
 *     per position, cap = budget cap.  Logit row (b, i) starts at element
 *     (b * L + i) * row_stride, row_stride >= V elements.
 *   - Output slots at or beyond a round's n_star are left untouched; consumers
 *     read n_star.  n_star = 0 (an empty tree) is a legal result.
 *
 * Tie-breaking (the paper leaves it open; fixed here so results are unique):
 *   - top-K: value descending, then token id ascending;
 *   - expansion order: log prefix probability descending, then depth
 *     ascending, then the sum of raw logits along the path descending, then
 *     the rank tuple lexicographically ascending;
 *   - stop: theta_new <= theta_prev stops (ties keep the smaller tree), as in
 *     Algorithm 1;
 *   - output order: depth ascending, then rank tuple lexicographically
 *     ascending (parents precede children).
 */
#ifndef CADDTREE_H
#define CADDTREE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CADDTREE_MAX_L 32
#define CADDTREE_MAX_K 16
#define CADDTREE_MAX_CAP 4096
#define CADDTREE_MAX_CTX 64     /* context-length grid points */

typedef enum {
  CADDTREE_OK = 0,
  CADDTREE_E_INVALID = 1,      /* bad argument: NULL where required, negative or inconsistent size */
  CADDTREE_E_UNSUPPORTED = 2,  /* valid request beyond the library's limits (L, K, cap, V) */
  CADDTREE_E_COST = 3,         /* cost model rejected: C_d <= 0, non-finite, C_v decreasing or not convex */
  CADDTREE_E_WORKSPACE = 4,    /* workspace NULL, misaligned or smaller than caddtree_workspace_bytes() */
  CADDTREE_E_HIP = 5           /* a HIP runtime call or kernel launch failed */
} caddtree_status_t;

typedef enum { CADDTREE_F32 = 0, CADDTREE_BF16 = 1 } caddtree_dtype_t;

/* Tree-attention mask format.  U8: [B, cap, cap] bytes, mask[b][i][j] = 1 iff
 * node j is node i or an ancestor of i.  BITS32: [B, cap, ceil(cap/32)] u32
 * words, bit (j % 32) of word (j / 32), least significant bit first.  Only
 * rows i < n_star and columns j < n_star (words j/32 < ceil(n_star/32)) are
 * written; for BITS32 the bits of the last written word at or beyond n_star
 * are written as zero. */
typedef enum { CADDTREE_MASK_NONE = 0, CADDTREE_MASK_U8 = 1, CADDTREE_MASK_BITS32 = 2 } caddtree_mask_t;

/* flags */
#define CADDTREE_ALLOW_NONCONVEX 1u  /* accept a C_v that is non-decreasing but not convex (Assumption 1
                                        may then fail: the greedy stop is still taken, optimality is not claimed) */
#define CADDTREE_FIXED_BUDGET 2u     /* fixed-budget mode (the DDTree construction, Sec. 3.4): no stop rule;
                                        every round keeps the top min(budget_cap, sum_d K^d) nodes by prefix
                                        probability, in the same order and layout.  phi and theta are still
                                        reported, theta from the plan's cost model at that size. */

typedef struct caddtree_plan* caddtree_plan_t;   /* opaque, immutable after creation */

/* Static description of a workload. */
typedef struct {
  int32_t L;                 /* block positions, 1 .. CADDTREE_MAX_L */
  int64_t V;                 /* vocabulary size, K .. 2^31 - 1 */
  int32_t K;                 /* tokens kept per position, 1 .. CADDTREE_MAX_K */
  int32_t budget_cap;        /* maximum nodes per tree, 0 .. CADDTREE_MAX_CAP */
  caddtree_dtype_t dtype;    /* logits element type */
  caddtree_mask_t mask;      /* mask format written by caddtree_build / caddtree_emit */
  uint32_t flags;            /* CADDTREE_ALLOW_NONCONVEX | CADDTREE_FIXED_BUDGET, or 0 */
  double t_draft;            /* C_d > 0, drafting cost of one round (Sec. 4.2) */
  const double* t_verify_host; /* HOST array of max(n_ctx, 1) x (budget_cap + 1) values: row j is
                                  C_v(0 .. cap; L_j), the verification cost of a tree of n nodes at
                                  context length L_j (Sec. 4.2, Sec. 4.6).  Every row must be finite,
                                  non-decreasing and convex in n (Cor. 3) up to a relative rounding
                                  slack of 1e-12; copied at plan creation. */
  int32_t n_ctx;             /* J, context-length grid points: 0 or 1 = one cost table and no context
                                dependence (ctx_len is then ignored); 2 .. CADDTREE_MAX_CTX = one table
                                per grid point, interpolated per round (Sec. 4.6, eq. cv-interp) */
  const int64_t* ctx_grid_host; /* HOST, J context lengths 0 <= L_0 < L_1 < ... < L_{J-1} <= 2^53
                                   (used when J >= 2); copied at plan creation */
} caddtree_config_t;

/* Validates cfg, copies the cost table to the current device and returns a plan.
 * The plan holds what Algorithm 1 takes besides the marginals: K, the costs C_d
 * and C_v(n; l) of Sec. 4.2 / 4.6 (eq. per-round's denominator), with the budget
 * cap this library adds, and the launch layout.  Rejects a cost that breaks
 * Assumption 1 (C_v non-decreasing and convex, Cor. 3) with CADDTREE_E_COST.
 * The plan is bound to the device that is current at creation; *plan_out is
 * NULL on any error.  Not thread-safe against caddtree_plan_destroy of the
 * same plan; concurrent builds on one plan are safe (distinct outputs and
 * workspaces). */
caddtree_status_t caddtree_plan_create(const caddtree_config_t* cfg, caddtree_plan_t* plan_out);
/* Frees the plan (NULL is a no-op).  The caller ensures no enqueued work still uses it. */
void caddtree_plan_destroy(caddtree_plan_t plan);

/* Device workspace caddtree_build needs for B rounds (the top-K table when the
 * caller does not ask for it).  256-byte alignment is required. */
size_t caddtree_workspace_bytes(caddtree_plan_t plan, int64_t B);

/* Outputs of caddtree_build (DEVICE pointers).  Required: token_ids, parent,
 * depth, n_star.  Optional (NULL skips the output): everything else.
 *   token_ids [B, cap] int32  vocabulary id of node i (canonical order)
 *   parent    [B, cap] int32  index of the parent node, -1 when the parent is the root (bonus token)
 *   depth     [B, cap] int32  1 .. L
 *   path_prob [B, cap] float  pi_s of the node (eq. prefix-prob), rounded to fp32
 *   n_star    [B]      int32  chosen budget
 *   phi       [B]      float  Phi*(n_star) = sum of path_prob over the tree (eq. surrogate), fp32
 *   theta     [B]      float  theta*(n_star) (eq. per-round), fp32
 *   mask      see caddtree_mask_t; ignored when the plan's mask is NONE
 *   pos_ids   [B, cap] int32  pos_offset + depth
 *   topk_ids  [B, L, K] int32, topk_logit [B, L, K] float (raw logits),
 *   topk_lq   [B, L, K] float (log q_i^(k)), lse [B, L] double (LSE_i) */
typedef struct {
  int32_t* token_ids;
  int32_t* parent;
  int32_t* depth;
  float* path_prob;
  int32_t* n_star;
  float* phi;
  float* theta;
  void* mask;
  int32_t* pos_ids;
  int32_t* topk_ids;
  float* topk_logit;
  float* topk_lq;
  double* lse;
} caddtree_outputs_t;

/* Context length of each round (plans with J >= 2 cost tables).  ctx_len is a
 * DEVICE int64 array [B].  A round at context length l with L_j <= l < L_{j+1}
 * uses C_v(n; l) = (1 - a) C_v(n; L_j) + a C_v(n; L_{j+1}), a = (l - L_j) /
 * (L_{j+1} - L_j) (eq. cv-interp), each product and the sum rounded
 * separately in fp64; l <= L_0 uses the L_0 table and l >= L_{J-1} the
 * L_{J-1} table (no extrapolation, which could break convexity).  NULL is an
 * error for such plans and is allowed otherwise. */

/* The whole hot path for B rounds (Sec. 3.2-3.3 and Algorithm 1): per round the
 * full-vocabulary log-normaliser and top-K of every position (eq. marginals),
 * the best-first expansion with the greedy stop of Lemma 1 (eq. stopping; the
 * tree T*_{n*} of eq. phistar at n* = the first maximiser of eq. per-round,
 * Cor. 2), and the tree-attention mask and position ids (Sec. 3.3).
 * logits: DEVICE [B, L, row_stride] of the plan's dtype; B >= 0 (0 is a no-op).
 * workspace: DEVICE, >= caddtree_workspace_bytes(plan, B) bytes, 256-byte aligned
 * (may be NULL when every top-K output pointer is given).
 * The call only enqueues kernels on `stream` (no allocation, memset or
 * synchronisation), so it may be captured in a HIP graph; a replay reads and
 * writes the buffers given at capture. */
caddtree_status_t caddtree_build(caddtree_plan_t plan, const void* logits, int64_t B, int64_t row_stride,
                                 int32_t pos_offset, const int64_t* ctx_len, const caddtree_outputs_t* out,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): caddtree_build with no
 * workspace argument.  The top-K table the caller does not ask for lives in a
 * device array inside the library, CADDTREE_NOALLOC_SCRATCH_BYTES per GPU, held
 * until the process ends; the call allocates and frees nothing and runs the same
 * kernels as caddtree_build, with the same results.
 *   Limit: caddtree_workspace_bytes(plan, B) for the top-K outputs left NULL
 *   must not exceed CADDTREE_NOALLOC_SCRATCH_BYTES (8 MiB: about
 *   2^20 / (L K + L) rounds, 7281 at L = 16, K = 8), else CADDTREE_E_WORKSPACE
 *   and nothing is enqueued.  Passing every top-K output lifts the limit.
 *   Every call on one GPU shares that GPU's array, whatever the plan or stream:
 *   calls that overlap in time on one GPU race (serialise them, e.g. on one
 *   stream).  Each call writes the part it reads before reading it, so nothing
 *   needs clearing between calls.
 *   Other arguments and errors as for caddtree_build; E_HIP if the array's
 *   address could not be taken when the plan was created. */
#define CADDTREE_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)
caddtree_status_t caddtree_build_noalloc(caddtree_plan_t plan, const void* logits, int64_t B, int64_t row_stride,
                                         int32_t pos_offset, const int64_t* ctx_len, const caddtree_outputs_t* out,
                                         hipStream_t stream);

/* Stage 1 (Sec. 3.2): per (round, position) row, LSE in fp64 and the top-K by
 * (value desc, id asc).  topk_ids, topk_logit, lse required; topk_lq optional. */
caddtree_status_t caddtree_reduce_topk(caddtree_plan_t plan, const void* logits, int64_t B, int64_t row_stride,
                                       int32_t* topk_ids, float* topk_logit, float* topk_lq, double* lse,
                                       hipStream_t stream);

/* Stage 2 (Algorithm 1): best-first expansion with the greedy stop, tree in canonical order.
 * Inputs: topk_ids, topk_logit [B, L, K], lse [B, L] (DEVICE); ctx_len as for
 * caddtree_build.  token_ids, parent, depth, n_star required; path_prob, phi,
 * theta optional. */
caddtree_status_t caddtree_expand(caddtree_plan_t plan, const int32_t* topk_ids, const float* topk_logit,
                                  const double* lse, int64_t B, const int64_t* ctx_len,
                                  int32_t* token_ids, int32_t* parent, int32_t* depth, float* path_prob,
                                  int32_t* n_star, float* phi, float* theta, hipStream_t stream);

/* Stage 3 (Sec. 3.3): tree-attention mask and position ids from parent/depth/n_star.
 * mask may be NULL (or the plan's mask NONE) to skip it; pos_ids may be NULL. */
caddtree_status_t caddtree_emit(caddtree_plan_t plan, const int32_t* parent, const int32_t* depth,
                                const int32_t* n_star, int64_t B, int32_t pos_offset,
                                void* mask, int32_t* pos_ids, hipStream_t stream);

/* Synthetic acceptance (tree verification, Sec. 3.3) of B built trees against
 * target continuations drawn from the drafter's factorised distribution
 * (eq. factorized), under which the expected accepted length of a tree is
 * Phi (eq. surrogate).  For a simulated throughput sum (1 + alpha) / sum C
 * (Sec. 4.2) over many rounds.
 *   topk_ids, topk_logit [B, L, K], lse [B, L]: DEVICE, as written by stage 1
 *   token_ids, parent [B, tree_stride], n_star [B]: DEVICE, a tree as written
 *       by caddtree_build / caddtree_expand (tree_stride = the budget cap of
 *       the plan that built it; n_star is clamped to [0, tree_stride])
 *   u [B, L]: DEVICE fp64 uniforms in [0, 1), owned by the caller (the random
 *       numbers are inputs).  Position i draws rank r for the smallest r with
 *       u_i < q^(0) + .. + q^(r), q^(k) = exp(l^(k) - LSE_i), the sum formed
 *       left to right in fp64; u_i at or above the sum of all K draws a token
 *       outside the top-K, which no node carries.
 *   accept_len [B] int32 (required): the length of the longest drawn prefix
 *       that is a path of the tree, 0 .. L.
 *   round_cost [B] fp64 (optional): C_d + C_v(n_star; l) from THIS plan's cost
 *       model (which may differ from the one that built the trees), NaN when
 *       n_star lies outside [0, cap]; ctx_len as for caddtree_build. */
caddtree_status_t caddtree_accept(caddtree_plan_t plan, const int32_t* topk_ids, const float* topk_logit,
                                  const double* lse, int64_t B, const int32_t* token_ids, const int32_t* parent,
                                  int32_t tree_stride, const int32_t* n_star, const double* u,
                                  const int64_t* ctx_len, int32_t* accept_len, double* round_cost,
                                  hipStream_t stream);

/* HOST only (no GPU, no stream): the offline cost model of Sec. 4.6.  Fits a
 * verification-cost profile y_j measured at node counts x_j (x strictly
 * increasing, all finite, 1 <= N <= 2^22) by the least-squares function that
 * is convex and non-decreasing (eq. convex-reg): a piecewise-linear function
 * whose breakpoints the data choose, solved exactly (active-set non-negative
 * least squares on the slope changes).
 *   fit_host [N] (optional): the fitted values at the x_j;
 *   table_host [cap + 1] (optional, 0 <= cap <= CADDTREE_MAX_CAP): the fit at
 *       n = 0 .. cap, interpolated linearly between the x_j and continued
 *       along the end segments outside them, ready to be a plan's
 *       t_verify_host row (one fit per context length, Sec. 4.6).
 * Host memory for the solve is allocated internally.  Returns E_INVALID for
 * bad input and E_UNSUPPORTED if the iteration does not settle. */
caddtree_status_t caddtree_fit_cost(const double* x_host, const double* y_host, int64_t N, double* fit_host,
                                    int32_t cap, double* table_host);

const char* caddtree_status_string(caddtree_status_t status);
const char* caddtree_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* CADDTREE_H */
