// Host side of the C ABI declared in caddtree.h: plan creation and validation,
// workspace sizing, argument checks and launch sequencing on the caller's stream.

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>

#include "internal.h"

struct caddtree_plan {
  int32_t L;
  int64_t V;
  int32_t K;
  int32_t cap;
  caddtree_dtype_t dtype;
  caddtree_mask_t mask;
  uint32_t flags;
  double t_draft;
  int32_t n_ctx;        // cost tables: 1, or one per context-length grid point
  double* d_t_verify;   // device copy, n_ctx x (cap + 1) values
  int64_t* d_ctx_grid;  // device copy of the grid (n_ctx >= 2), else NULL
  bool use_level;       // the batched expansion applies (see plan_create)
  bool use_wide;        // ... in its several-wavefront form
  int num_cu;           // compute units of the plan's device
  bool flat_cost;       // every cost table holds one value up to the cap
  int level_set_cap;    // its threshold-set capacity
  int device;
  int k1_waves;         // 0 = automatic
  int k1_unroll;        // 0 = automatic
  bool noalloc_ready;   // the scratch array of caddtree_build_noalloc has an address on this device
  bool fuse_emit;       // caddtree_build lets the expansion's epilogue write the mask and position ids
  int first_rise;       // the batched expansion's first threshold inputs (ExpandArgs), -2 if per round
  double tau_model;
};

namespace {

thread_local std::string g_last_error;

caddtree_status_t fail(caddtree_status_t st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
caddtree_status_t fail(caddtree_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

caddtree_status_t ok() {
  g_last_error.clear();
  return CADDTREE_OK;
}

caddtree_status_t hip_fail(hipError_t e, const char* what) {
  return fail(CADDTREE_E_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

size_t elem_bytes(caddtree_dtype_t d) { return d == CADDTREE_BF16 ? 2 : 4; }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The value a C caller stored in an enum-typed field or argument, read as the int it is: a C
// caller may pass any int there, which a C++ enum object must not hold.
template <typename E>
int enum_value(const E& e) {
  static_assert(sizeof(E) == sizeof(int), "the C enums of the interface are int-sized");
  int v;
  std::memcpy(&v, &e, sizeof v);
  return v;
}

caddtree_status_t check_plan(const caddtree_plan* p) {
  if (p == nullptr) return fail(CADDTREE_E_INVALID, "plan is NULL");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != p->device)
    return fail(CADDTREE_E_INVALID, "plan was created on device %d but device %d is current", p->device, dev);
  return CADDTREE_OK;
}

struct TopkBuffers {
  int32_t* ids;
  float* logit;
  double* lse;
};

// Carves the top-K table out of the workspace for the pieces the caller did not supply.
size_t topk_workspace(const caddtree_plan* p, int64_t B, const caddtree_outputs_t* out, char* base,
                      TopkBuffers* tb) {
  const size_t rows = (size_t)B * (size_t)p->L;
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    char* r = base ? base + off : nullptr;
    off = align256(off + bytes);
    return r;
  };
  tb->ids = out && out->topk_ids ? out->topk_ids : reinterpret_cast<int32_t*>(take(rows * p->K * 4));
  tb->logit = out && out->topk_logit ? out->topk_logit : reinterpret_cast<float*>(take(rows * p->K * 4));
  tb->lse = out && out->lse ? out->lse : reinterpret_cast<double*>(take(rows * 8));
  return off;
}

caddtree_status_t check_logits(const caddtree_plan* p, const void* logits, int64_t B, int64_t row_stride) {
  if (B < 0) return fail(CADDTREE_E_INVALID, "B = %lld is negative", (long long)B);
  if (B > 0 && logits == nullptr) return fail(CADDTREE_E_INVALID, "logits is NULL");
  if (row_stride < p->V)
    return fail(CADDTREE_E_INVALID, "row_stride %lld < V %lld", (long long)row_stride, (long long)p->V);
  if (B * (int64_t)p->L > (int64_t)INT32_MAX)
    return fail(CADDTREE_E_UNSUPPORTED, "B * L = %lld exceeds 2^31 - 1 rows", (long long)(B * p->L));
  return CADDTREE_OK;
}


caddtree_status_t run_reduce(const caddtree_plan* p, const void* logits, int64_t B, int64_t row_stride,
                             int32_t* ids, float* logit, float* lq, double* lse, hipStream_t stream) {
  caddtree::ReduceArgs a;
  a.logits = logits;
  a.rows = B * p->L;
  a.row_stride = row_stride;
  a.V = (int32_t)p->V;
  a.K = p->K;
  const caddtree::ReduceShape sh = caddtree::reduce_default_shape(a.rows, (int32_t)p->V, p->dtype);
  a.waves_per_row = p->k1_waves > 0 ? p->k1_waves : sh.waves;
  a.unroll = p->k1_unroll > 0 ? p->k1_unroll : sh.unroll;
  const size_t es = elem_bytes(p->dtype);
  a.aligned = (reinterpret_cast<uintptr_t>(logits) % 16 == 0) && ((size_t)row_stride * es) % 16 == 0;
  a.ids = ids;
  a.logit = logit;
  a.lq = lq;
  a.lse = lse;
  hipError_t e = caddtree::launch_reduce_topk(a, p->dtype, stream);
  if (e != hipSuccess) return hip_fail(e, "reduce_topk launch");
  return CADDTREE_OK;
}

caddtree_status_t check_ctx(const caddtree_plan* p, const int64_t* ctx_len) {
  if (p->n_ctx >= 2 && ctx_len == nullptr)
    return fail(CADDTREE_E_INVALID, "ctx_len is required: the plan has %d context-length cost tables", p->n_ctx);
  return CADDTREE_OK;
}

caddtree_status_t run_expand(const caddtree_plan* p, const int32_t* ids, const float* logit, const double* lse,
                             int64_t B, const int64_t* ctx_len, int32_t* token_ids, int32_t* parent,
                             int32_t* depth, float* path_prob, int32_t* n_star, float* phi, float* theta,
                             hipStream_t stream, const caddtree::EmitOut* em = nullptr) {
  caddtree::ExpandArgs a;
  a.em = em ? *em : caddtree::EmitOut{nullptr, nullptr, (int)CADDTREE_MASK_NONE, 0};
  a.topk_ids = ids;
  a.topk_logit = logit;
  a.lse = lse;
  a.B = B;
  a.L = p->L;
  a.K = p->K;
  a.cap = p->cap;
  a.cost.tv = p->d_t_verify;
  a.cost.grid = p->d_ctx_grid;
  a.cost.ctx_len = ctx_len;
  a.cost.J = p->n_ctx;
  a.cost.stride = p->cap + 1;
  a.cost.t_draft = p->t_draft;
  a.token_ids = token_ids;
  a.parent = parent;
  a.depth = depth;
  a.path_prob = path_prob;
  a.n_star = n_star;
  a.phi = phi;
  a.theta = theta;
  a.use_level = p->use_level;
  a.use_wide = p->use_wide;
  a.num_cu = p->num_cu;
  a.level_set_cap = p->level_set_cap;
  a.fixed_budget = (p->flags & CADDTREE_FIXED_BUDGET) != 0;
  a.flat_cost = p->flat_cost;
  a.first_rise = p->first_rise;
  a.tau_model = p->tau_model;
  hipError_t e = caddtree::launch_expand(a, stream);
  if (e != hipSuccess) return hip_fail(e, "expand launch");
  return CADDTREE_OK;
}

caddtree_status_t run_emit(const caddtree_plan* p, const int32_t* parent, const int32_t* depth,
                           const int32_t* n_star, int64_t B, int32_t pos_offset, void* mask, int32_t* pos_ids,
                           hipStream_t stream) {
  caddtree::EmitArgs a;
  a.parent = parent;
  a.depth = depth;
  a.n_star = n_star;
  a.B = B;
  a.cap = p->cap;
  a.pos_offset = pos_offset;
  a.mask_kind = p->mask;
  a.mask = p->mask == CADDTREE_MASK_NONE ? nullptr : mask;
  a.pos_ids = pos_ids;
  a.num_cu = p->num_cu;
  if (a.mask == nullptr && a.pos_ids == nullptr) return CADDTREE_OK;
  hipError_t e = caddtree::launch_emit(a, stream);
  if (e != hipSuccess) return hip_fail(e, "emit launch");
  return CADDTREE_OK;
}

}  // namespace

extern "C" {

const char* caddtree_status_string(caddtree_status_t s) {
  switch (enum_value(s)) {
    case CADDTREE_OK: return "ok";
    case CADDTREE_E_INVALID: return "invalid argument";
    case CADDTREE_E_UNSUPPORTED: return "unsupported configuration";
    case CADDTREE_E_COST: return "cost model rejected";
    case CADDTREE_E_WORKSPACE: return "workspace too small or misaligned";
    case CADDTREE_E_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* caddtree_last_error(void) { return g_last_error.c_str(); }

caddtree_status_t caddtree_plan_create(const caddtree_config_t* cfg, caddtree_plan_t* plan_out) {
  if (plan_out == nullptr) return fail(CADDTREE_E_INVALID, "plan_out is NULL");
  *plan_out = nullptr;
  if (cfg == nullptr) return fail(CADDTREE_E_INVALID, "cfg is NULL");
  if (cfg->L < 1) return fail(CADDTREE_E_INVALID, "L = %d must be >= 1", cfg->L);
  if (cfg->L > CADDTREE_MAX_L) return fail(CADDTREE_E_UNSUPPORTED, "L = %d exceeds %d", cfg->L, CADDTREE_MAX_L);
  if (cfg->K < 1) return fail(CADDTREE_E_INVALID, "K = %d must be >= 1", cfg->K);
  if (cfg->K > CADDTREE_MAX_K) return fail(CADDTREE_E_UNSUPPORTED, "K = %d exceeds %d", cfg->K, CADDTREE_MAX_K);
  if (cfg->V < cfg->K) return fail(CADDTREE_E_INVALID, "V = %lld is smaller than K = %d", (long long)cfg->V, cfg->K);
  if (cfg->V > (int64_t)INT32_MAX - 1)
    return fail(CADDTREE_E_UNSUPPORTED, "V = %lld exceeds 2^31 - 2", (long long)cfg->V);
  if (cfg->budget_cap < 0) return fail(CADDTREE_E_INVALID, "budget_cap = %d is negative", cfg->budget_cap);
  if (cfg->budget_cap > CADDTREE_MAX_CAP)
    return fail(CADDTREE_E_UNSUPPORTED, "budget_cap = %d exceeds %d", cfg->budget_cap, CADDTREE_MAX_CAP);
  const int dtype = enum_value(cfg->dtype), mask = enum_value(cfg->mask);
  if (dtype != CADDTREE_F32 && dtype != CADDTREE_BF16)
    return fail(CADDTREE_E_INVALID, "unknown dtype %d", dtype);
  if (mask != CADDTREE_MASK_NONE && mask != CADDTREE_MASK_U8 && mask != CADDTREE_MASK_BITS32)
    return fail(CADDTREE_E_INVALID, "unknown mask kind %d", mask);
  if (cfg->flags & ~(CADDTREE_ALLOW_NONCONVEX | CADDTREE_FIXED_BUDGET))
    return fail(CADDTREE_E_INVALID, "unknown flags 0x%x", cfg->flags);
  if (!(cfg->t_draft > 0.0) || !std::isfinite(cfg->t_draft))
    return fail(CADDTREE_E_COST, "t_draft = %g must be finite and > 0", cfg->t_draft);
  if (cfg->t_verify_host == nullptr) return fail(CADDTREE_E_INVALID, "t_verify_host is NULL");
  if (cfg->n_ctx < 0) return fail(CADDTREE_E_INVALID, "n_ctx = %d is negative", cfg->n_ctx);
  if (cfg->n_ctx > CADDTREE_MAX_CTX)
    return fail(CADDTREE_E_UNSUPPORTED, "n_ctx = %d exceeds %d", cfg->n_ctx, CADDTREE_MAX_CTX);
  const int J = cfg->n_ctx < 1 ? 1 : cfg->n_ctx;
  if (J >= 2) {
    const int64_t* g = cfg->ctx_grid_host;
    if (g == nullptr) return fail(CADDTREE_E_INVALID, "ctx_grid_host is NULL with n_ctx = %d", J);
    for (int j = 0; j < J; ++j) {
      if (g[j] < 0 || g[j] > ((int64_t)1 << 53))
        return fail(CADDTREE_E_INVALID, "ctx_grid_host[%d] = %lld is outside [0, 2^53]", j, (long long)g[j]);
      if (j > 0 && g[j] <= g[j - 1])
        return fail(CADDTREE_E_INVALID, "ctx_grid_host is not strictly increasing at %d", j);
    }
  }
  const int cap = cfg->budget_cap;
  int flat_start = 0;     // the most leading zero marginal costs over the tables
  bool convex = true;
  bool flat_cost = true;  // every table holds one value (bit for bit) up to the cap
  for (int j = 0; j < J; ++j) {
    const double* tv = cfg->t_verify_host + (size_t)j * (size_t)(cap + 1);
    double scale = 0.0;
    for (int n = 0; n <= cap; ++n) {
      if (!std::isfinite(tv[n])) return fail(CADDTREE_E_COST, "C_v(%d) of table %d is not finite", n, j);
      if (!(cfg->t_draft + tv[n] > 0.0)) return fail(CADDTREE_E_COST, "C_d + C_v(%d) <= 0 in table %d", n, j);
      scale = std::fmax(scale, std::fabs(tv[n]));
    }
    const double slack = 1e-12 * std::fmax(scale, cfg->t_draft);
    for (int n = 1; n <= cap; ++n)
      if (tv[n] - tv[n - 1] < -slack)
        return fail(CADDTREE_E_COST, "C_v of table %d decreases between n = %d and %d", j, n - 1, n);
    for (int n = 2; n <= cap; ++n)
      if ((tv[n] - tv[n - 1]) - (tv[n - 1] - tv[n - 2]) < -slack) {
        if (!(cfg->flags & CADDTREE_ALLOW_NONCONVEX))
          return fail(CADDTREE_E_COST, "C_v of table %d is not convex at n = %d (Assumption 1 needs convex cost)",
                      j, n - 1);
        convex = false;
      }
    int m0 = 0;
    while (m0 < cap && !(tv[m0 + 1] > tv[m0])) ++m0;
    flat_start = std::max(flat_start, m0);
    for (int n = 1; n <= cap && flat_cost; ++n) flat_cost = tv[n] == tv[0];
  }

  caddtree_plan* p = new (std::nothrow) caddtree_plan();
  if (p == nullptr) return fail(CADDTREE_E_INVALID, "out of host memory");
  p->L = cfg->L;
  p->V = cfg->V;
  p->K = cfg->K;
  p->cap = cap;
  p->dtype = (caddtree_dtype_t)dtype;
  p->mask = (caddtree_mask_t)mask;
  p->flags = cfg->flags;
  p->t_draft = cfg->t_draft;
  p->n_ctx = J;
  p->d_t_verify = nullptr;
  p->d_ctx_grid = nullptr;
  // The batched expansion finds the stop by bisection, which needs theta to be
  // unimodal along the pop order (a convex cost, Thm. 1), and a threshold set
  // that holds at least the nodes every tree keeps: the budget with a fixed
  // budget or a cost flat up to the cap, else the nodes before the first
  // positive marginal cost (the most over the tables).  The set is sized to
  // twice that, 512 .. 4096 nodes.  Fixed budgets and flat costs need no cost
  // table in LDS, which leaves room for 5120 nodes (trees of up to 4096).
  const bool fixed = (cfg->flags & CADDTREE_FIXED_BUDGET) != 0;
  const bool lean = fixed || flat_cost;
  const int need = (fixed || flat_start >= cap) ? cap : flat_start + 1;
  p->flat_cost = flat_cost;
  p->use_level = cap >= 1 && (fixed || convex) && need <= caddtree::expand_level_max_need(lean);
  p->level_set_cap = caddtree::expand_level_set_cap(need, lean);
  // With one cost table, where the batched expansion starts its threshold search depends on the
  // plan only: the first position with a positive marginal cost (below the cap and the set
  // capacity) and the cost-model threshold there, found once here instead of by every round.
  // C(n) is formed as the kernels form it for one table, C_d + C_v(n).
  p->first_rise = -2;
  p->tau_model = 0.0;
  if (J == 1 && !lean) {
    const double* tv = cfg->t_verify_host;
    const double td = cfg->t_draft;
    const int mlim = std::min(cap, p->level_set_cap);
    int m0 = -1;
    for (int i = 0; i < mlim && m0 < 0; ++i)
      if (td + tv[i + 1] > td + tv[i]) m0 = i;
    p->first_rise = m0;
    if (m0 >= 0) {
      const int m = std::min(m0 + 32, cap);
      p->tau_model = std::log(2.0 * ((td + tv[m0 + 1]) - (td + tv[m0])) / (td + tv[m])) - 0.5;
    }
  }
  // Large trees of a known size (fixed budgets and costs flat up to the cap, 512 nodes or more) run
  // on eight wavefronts per round; CADDTREE_EXPAND=level keeps them on one, =serial sends every
  // round to the serial kernel.
  p->use_wide = p->use_level && caddtree::expand_wide_applies(cap, lean);
  if (const char* env = std::getenv("CADDTREE_EXPAND")) {
    if (std::strcmp(env, "serial") == 0) p->use_level = false;
    if (std::strcmp(env, "level") == 0) p->use_wide = false;
  }
  // The expansion kernels can write each round's mask and position ids from the tree still in LDS,
  // one wavefront per round, which saves a launch.  That pays for the trees a rising cost keeps small;
  // fixed budgets and costs flat up to the cap (trees of the full cap) and long flat starts keep the
  // emission kernel, whose many workgroups per round write large masks faster.
  p->fuse_emit = !lean && flat_start < 512;
  if (const char* env = std::getenv("CADDTREE_EMIT")) {
    if (std::strcmp(env, "separate") == 0) p->fuse_emit = false;
  }
  p->k1_waves = 0;
  if (const char* env = std::getenv("CADDTREE_K1_WAVES")) {
    const int w = std::atoi(env);
    if (w == 1 || w == 2 || w == 4 || w == 8 || w == 16) p->k1_waves = w;
  }
  p->k1_unroll = 0;
  if (const char* env = std::getenv("CADDTREE_K1_UNROLL")) {
    const int u = std::atoi(env);
    if (u == 4 || u == 8) p->k1_unroll = u;
  }
  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) { delete p; return hip_fail(e, "hipGetDevice"); }
  e = hipDeviceGetAttribute(&p->num_cu, hipDeviceAttributeMultiprocessorCount, p->device);
  if (e != hipSuccess) { delete p; return hip_fail(e, "hipDeviceGetAttribute(multiprocessor count)"); }
  const size_t tv_bytes = sizeof(double) * (size_t)J * (size_t)(cap + 1);
  e = hipMalloc(&p->d_t_verify, tv_bytes);
  if (e != hipSuccess) { delete p; return hip_fail(e, "hipMalloc(cost table)"); }
  e = hipMemcpy(p->d_t_verify, cfg->t_verify_host, tv_bytes, hipMemcpyHostToDevice);
  if (e == hipSuccess && J >= 2) {
    e = hipMalloc(&p->d_ctx_grid, sizeof(int64_t) * (size_t)J);
    if (e == hipSuccess)
      e = hipMemcpy(p->d_ctx_grid, cfg->ctx_grid_host, sizeof(int64_t) * (size_t)J, hipMemcpyHostToDevice);
  }
  // the no-allocation entry point's scratch array: its address on this device, taken once per device
  p->noalloc_ready = caddtree::noalloc_scratch_init(p->device) == hipSuccess;
  (void)hipGetLastError();
  if (e == hipSuccess) e = caddtree::expand_prepare(p->L, p->K, p->cap);
  if (e == hipSuccess) e = caddtree::expand_level_prepare();
  if (e == hipSuccess) e = caddtree::expand_wide_prepare();
  if (e != hipSuccess) {
    (void)hipFree(p->d_t_verify);
    if (p->d_ctx_grid) (void)hipFree(p->d_ctx_grid);
    delete p;
    return hip_fail(e, "plan setup");
  }
  *plan_out = p;
  return ok();
}

void caddtree_plan_destroy(caddtree_plan_t p) {
  if (p == nullptr) return;
  if (p->d_t_verify) (void)hipFree(p->d_t_verify);
  if (p->d_ctx_grid) (void)hipFree(p->d_ctx_grid);
  delete p;
}

size_t caddtree_workspace_bytes(caddtree_plan_t p, int64_t B) {
  if (p == nullptr || B <= 0) return 0;
  TopkBuffers tb;
  return topk_workspace(p, B, nullptr, nullptr, &tb);
}

caddtree_status_t caddtree_reduce_topk(caddtree_plan_t p, const void* logits, int64_t B, int64_t row_stride,
                                       int32_t* topk_ids, float* topk_logit, float* topk_lq, double* lse,
                                       hipStream_t stream) {
  caddtree_status_t st = check_plan(p);
  if (st != CADDTREE_OK) return st;
  if ((st = check_logits(p, logits, B, row_stride)) != CADDTREE_OK) return st;
  if (B > 0 && (topk_ids == nullptr || topk_logit == nullptr || lse == nullptr))
    return fail(CADDTREE_E_INVALID, "topk_ids, topk_logit and lse are required");
  if (B == 0) return ok();
  if ((st = run_reduce(p, logits, B, row_stride, topk_ids, topk_logit, topk_lq, lse, stream)) != CADDTREE_OK)
    return st;
  return ok();
}

caddtree_status_t caddtree_expand(caddtree_plan_t p, const int32_t* topk_ids, const float* topk_logit,
                                  const double* lse, int64_t B, const int64_t* ctx_len, int32_t* token_ids,
                                  int32_t* parent,
                                  int32_t* depth, float* path_prob, int32_t* n_star, float* phi, float* theta,
                                  hipStream_t stream) {
  caddtree_status_t st = check_plan(p);
  if (st != CADDTREE_OK) return st;
  if (B < 0) return fail(CADDTREE_E_INVALID, "B = %lld is negative", (long long)B);
  if (B == 0) return ok();
  if (topk_ids == nullptr || topk_logit == nullptr || lse == nullptr)
    return fail(CADDTREE_E_INVALID, "topk_ids, topk_logit and lse are required");
  if (token_ids == nullptr || parent == nullptr || depth == nullptr || n_star == nullptr)
    return fail(CADDTREE_E_INVALID, "token_ids, parent, depth and n_star are required");
  if (B > (int64_t)INT32_MAX) return fail(CADDTREE_E_UNSUPPORTED, "B exceeds 2^31 - 1");
  if ((st = check_ctx(p, ctx_len)) != CADDTREE_OK) return st;
  if ((st = run_expand(p, topk_ids, topk_logit, lse, B, ctx_len, token_ids, parent, depth, path_prob, n_star,
                       phi, theta, stream)) != CADDTREE_OK)
    return st;
  return ok();
}

caddtree_status_t caddtree_emit(caddtree_plan_t p, const int32_t* parent, const int32_t* depth,
                                const int32_t* n_star, int64_t B, int32_t pos_offset, void* mask,
                                int32_t* pos_ids, hipStream_t stream) {
  caddtree_status_t st = check_plan(p);
  if (st != CADDTREE_OK) return st;
  if (B < 0) return fail(CADDTREE_E_INVALID, "B = %lld is negative", (long long)B);
  if (B == 0) return ok();
  if (B > (int64_t)UINT32_MAX / 2) return fail(CADDTREE_E_UNSUPPORTED, "B too large");
  if (parent == nullptr || n_star == nullptr) return fail(CADDTREE_E_INVALID, "parent and n_star are required");
  if (pos_ids != nullptr && depth == nullptr) return fail(CADDTREE_E_INVALID, "pos_ids needs depth");
  if ((st = run_emit(p, parent, depth, n_star, B, pos_offset, mask, pos_ids, stream)) != CADDTREE_OK) return st;
  return ok();
}

}  // extern "C"

namespace {

// Argument checks shared by caddtree_build and caddtree_build_noalloc; *done is set when B = 0.
caddtree_status_t check_build(const caddtree_plan* p, const void* logits, int64_t B, int64_t row_stride,
                              const int64_t* ctx_len, const caddtree_outputs_t* out, bool* done) {
  *done = false;
  caddtree_status_t st = check_plan(p);
  if (st != CADDTREE_OK) return st;
  if ((st = check_logits(p, logits, B, row_stride)) != CADDTREE_OK) return st;
  if (out == nullptr) return fail(CADDTREE_E_INVALID, "out is NULL");
  if (B == 0) {
    *done = true;
    return CADDTREE_OK;
  }
  if (out->token_ids == nullptr || out->parent == nullptr || out->depth == nullptr || out->n_star == nullptr)
    return fail(CADDTREE_E_INVALID, "out->token_ids, parent, depth and n_star are required");
  if (B > (int64_t)INT32_MAX) return fail(CADDTREE_E_UNSUPPORTED, "B exceeds 2^31 - 1");
  return check_ctx(p, ctx_len);
}

// The three stages on `stream`, the top-K table the caller did not ask for carved from `workspace`.
caddtree_status_t run_build(const caddtree_plan* p, const void* logits, int64_t B, int64_t row_stride,
                            int32_t pos_offset, const int64_t* ctx_len, const caddtree_outputs_t* out,
                            void* workspace, hipStream_t stream) {
  TopkBuffers tb;
  topk_workspace(p, B, out, static_cast<char*>(workspace), &tb);
  caddtree_status_t st;
  if ((st = run_reduce(p, logits, B, row_stride, tb.ids, tb.logit, out->topk_lq, tb.lse, stream)) != CADDTREE_OK)
    return st;
  caddtree::EmitOut em{p->mask == CADDTREE_MASK_NONE ? nullptr : out->mask, out->pos_ids, (int)p->mask, pos_offset};
  const bool fused = p->fuse_emit && p->cap > 0;
  if ((st = run_expand(p, tb.ids, tb.logit, tb.lse, B, ctx_len, out->token_ids, out->parent, out->depth,
                       out->path_prob, out->n_star, out->phi, out->theta, stream, fused ? &em : nullptr)) !=
      CADDTREE_OK)
    return st;
  if (!fused &&
      (st = run_emit(p, out->parent, out->depth, out->n_star, B, pos_offset, out->mask, out->pos_ids, stream)) !=
          CADDTREE_OK)
    return st;
  return ok();
}

}  // namespace

extern "C" {

caddtree_status_t caddtree_build(caddtree_plan_t p, const void* logits, int64_t B, int64_t row_stride,
                                 int32_t pos_offset, const int64_t* ctx_len, const caddtree_outputs_t* out,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream) {
  bool done;
  caddtree_status_t st = check_build(p, logits, B, row_stride, ctx_len, out, &done);
  if (st != CADDTREE_OK) return st;
  if (done) return ok();
  TopkBuffers tb;
  const size_t need = topk_workspace(p, B, out, nullptr, &tb);
  if (need > 0) {
    if (workspace == nullptr) return fail(CADDTREE_E_WORKSPACE, "workspace is NULL, %zu bytes needed", need);
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
      return fail(CADDTREE_E_WORKSPACE, "workspace must be 256-byte aligned");
    if (workspace_bytes < need)
      return fail(CADDTREE_E_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
  }
  return run_build(p, logits, B, row_stride, pos_offset, ctx_len, out, workspace, stream);
}

caddtree_status_t caddtree_build_noalloc(caddtree_plan_t p, const void* logits, int64_t B, int64_t row_stride,
                                         int32_t pos_offset, const int64_t* ctx_len, const caddtree_outputs_t* out,
                                         hipStream_t stream) {
  bool done;
  caddtree_status_t st = check_build(p, logits, B, row_stride, ctx_len, out, &done);
  if (st != CADDTREE_OK) return st;
  if (done) return ok();
  TopkBuffers tb;
  const size_t need = topk_workspace(p, B, out, nullptr, &tb);
  void* scratch = nullptr;
  if (need > 0) {
    if (need > caddtree::kNoAllocScratchBytes)
      return fail(CADDTREE_E_WORKSPACE,
                  "the top-K table of %lld rounds needs %zu bytes, beyond the %zu-byte library scratch; pass the "
                  "top-K outputs or use caddtree_build with a workspace",
                  (long long)B, need, caddtree::kNoAllocScratchBytes);
    if (!p->noalloc_ready || (scratch = caddtree::noalloc_scratch(p->device)) == nullptr)
      return fail(CADDTREE_E_HIP, "the library scratch has no address on device %d", p->device);
  }
  return run_build(p, logits, B, row_stride, pos_offset, ctx_len, out, scratch, stream);
}

caddtree_status_t caddtree_accept(caddtree_plan_t p, const int32_t* topk_ids, const float* topk_logit,
                                  const double* lse, int64_t B, const int32_t* token_ids, const int32_t* parent,
                                  int32_t tree_stride, const int32_t* n_star, const double* u,
                                  const int64_t* ctx_len, int32_t* accept_len, double* round_cost,
                                  hipStream_t stream) {
  caddtree_status_t st = check_plan(p);
  if (st != CADDTREE_OK) return st;
  if (B < 0) return fail(CADDTREE_E_INVALID, "B = %lld is negative", (long long)B);
  if (tree_stride < 0) return fail(CADDTREE_E_INVALID, "tree_stride = %d is negative", tree_stride);
  if (B == 0) return ok();
  if (B > (int64_t)INT32_MAX) return fail(CADDTREE_E_UNSUPPORTED, "B exceeds 2^31 - 1");
  if (topk_ids == nullptr || topk_logit == nullptr || lse == nullptr)
    return fail(CADDTREE_E_INVALID, "topk_ids, topk_logit and lse are required");
  if (token_ids == nullptr || parent == nullptr || n_star == nullptr || u == nullptr || accept_len == nullptr)
    return fail(CADDTREE_E_INVALID, "token_ids, parent, n_star, u and accept_len are required");
  if (round_cost != nullptr && (st = check_ctx(p, ctx_len)) != CADDTREE_OK) return st;
  caddtree::AcceptArgs a;
  a.topk_ids = topk_ids;
  a.topk_logit = topk_logit;
  a.lse = lse;
  a.B = B;
  a.L = p->L;
  a.K = p->K;
  a.token_ids = token_ids;
  a.parent = parent;
  a.tree_stride = tree_stride;
  a.n_star = n_star;
  a.u = u;
  a.cost.tv = p->d_t_verify;
  a.cost.grid = p->d_ctx_grid;
  a.cost.ctx_len = ctx_len;
  a.cost.J = p->n_ctx;
  a.cost.stride = p->cap + 1;
  a.cost.t_draft = p->t_draft;
  a.cap = p->cap;
  a.accept_len = accept_len;
  a.round_cost = round_cost;
  hipError_t e = caddtree::launch_accept(a, stream);
  if (e != hipSuccess) return hip_fail(e, "accept launch");
  return ok();
}

caddtree_status_t caddtree_fit_cost(const double* x_host, const double* y_host, int64_t N, double* fit_host,
                                    int32_t cap, double* table_host) {
  if (x_host == nullptr || y_host == nullptr) return fail(CADDTREE_E_INVALID, "x_host and y_host are required");
  if (N < 1) return fail(CADDTREE_E_INVALID, "N = %lld must be >= 1", (long long)N);
  if (N > ((int64_t)1 << 22)) return fail(CADDTREE_E_UNSUPPORTED, "N = %lld exceeds 2^22", (long long)N);
  if (table_host != nullptr && (cap < 0 || cap > CADDTREE_MAX_CAP))
    return fail(CADDTREE_E_INVALID, "cap = %d must be in [0, %d]", cap, CADDTREE_MAX_CAP);
  for (int64_t j = 0; j < N; ++j) {
    if (!std::isfinite(x_host[j]) || !std::isfinite(y_host[j]))
      return fail(CADDTREE_E_INVALID, "profile point %lld is not finite", (long long)j);
    if (j > 0 && !(x_host[j] > x_host[j - 1]))
      return fail(CADDTREE_E_INVALID, "x_host is not strictly increasing at %lld", (long long)j);
  }
  if (!caddtree::fit_convex_cost(x_host, y_host, (int)N, fit_host, cap, table_host))
    return fail(CADDTREE_E_UNSUPPORTED, "the active-set iteration did not settle");
  return ok();
}

}  // extern "C"
