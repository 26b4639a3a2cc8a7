// Internal launch interface between the host library (api.cpp) and the kernels.  Host-only sources
// include it, so it declares no device code.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#include "caddtree.h"
#include "kargs.h"

namespace caddtree {

// Stage 1: vocabulary reduction + top-K, one workgroup of `waves_per_row`
// wavefronts per logit row.
struct ReduceArgs {
  const void* logits;
  int64_t rows;          // B * L
  int64_t row_stride;    // elements
  int32_t V;
  int32_t K;
  int32_t waves_per_row; // 1 .. 16
  int32_t unroll;        // 16-byte loads in flight per lane: 4 or 8
  bool aligned;          // rows start on 16-byte boundaries
  int32_t* ids;          // [rows, K]
  float* logit;          // [rows, K]
  float* lq;             // [rows, K] or nullptr
  double* lse;           // [rows]
};
hipError_t launch_reduce_topk(const ReduceArgs& a, caddtree_dtype_t dtype, hipStream_t stream);
struct ReduceShape {
  int32_t waves;   // waves per row
  int32_t unroll;  // 16-byte loads in flight per lane
};
ReduceShape reduce_default_shape(int64_t rows, int32_t V, caddtree_dtype_t dtype);

// Stage 2: best-first expansion with the greedy stop, one workgroup per round.
struct ExpandArgs {
  const int32_t* topk_ids;
  const float* topk_logit;
  const double* lse;
  int64_t B;
  int32_t L, K, cap;
  xp::CostTables cost;     // device cost tables, context grid and per-round context lengths
  int32_t* token_ids;
  int32_t* parent;
  int32_t* depth;
  float* path_prob;        // optional
  int32_t* n_star;
  float* phi;              // optional
  float* theta;            // optional
  bool use_level;          // try the batched kernel first
  bool use_wide;           // ... in its several-wavefront form (large trees of a known size)
  int32_t num_cu;          // compute units of the device
  int32_t level_set_cap;   // its threshold-set capacity
  bool fixed_budget;       // no stop rule: keep the top min(cap, #nodes) nodes (DDTree)
  bool flat_cost;          // every table holds one value: C(n) = C(0) up to the cap
  int32_t first_rise;      // one cost table: the first n < min(cap, level_set_cap) with C(n + 1) > C(n),
                           // -1 if none; -2 when the kernel finds it per round (several tables)
  double tau_model;        // with first_rise = m0 >= 0: log(2 (C(m0 + 1) - C(m0)) / C(min(m0 + 32, cap))) - 1/2
  EmitOut em;              // mask and position ids written by the expansion's epilogue (null: not here)
};
size_t expand_lds_bytes(int32_t L, int32_t K, int32_t cap);
hipError_t expand_prepare(int32_t L, int32_t K, int32_t cap);  // raises the dynamic-LDS limit once
hipError_t launch_expand(const ExpandArgs& a, hipStream_t stream);
// in_place_lds > 0: a round the batched kernel cannot settle is run by the serial form in the
// same workgroup, in that many bytes of LDS (the launch reserves the larger of the two layouts);
// 0: such a round is flagged (n_star = -1) for the serial kernel
hipError_t launch_expand_level(const ExpandArgs& a, size_t in_place_lds, hipStream_t stream);
// the largest serial layout that the batched kernel reserves LDS for
constexpr size_t kInPlaceLds = 64 * 1024;
// ... or any serial layout the batched kernels' LDS limit admits, when every round has a CU of its
// own (reserving it then costs no occupancy)
size_t expand_level_lds_limit();
// (lean: fixed budgets and flat costs, which need no cost table and so hold larger sets)
size_t expand_level_lds_bytes(int32_t L, int32_t K, int32_t set_cap, bool lean);
int expand_level_set_cap(int32_t need, bool lean);   // threshold-set capacity for trees of at least `need` nodes
int expand_level_max_need(bool lean);                // the largest `need` the batched kernel takes
hipError_t expand_level_prepare();        // raises the batched kernel's dynamic-LDS limit
// The several-wavefront batched kernel (expand_wide.hip): trees that keep a known number of nodes
// (a fixed budget, or a cost flat up to the cap) of at least 512.
bool expand_wide_applies(int32_t cap, bool lean);
size_t expand_wide_lds_bytes(int32_t L, int32_t K, int32_t set_cap);
hipError_t expand_wide_prepare();
// Rounds it cannot settle are flagged (n_star = -1) for the serial kernel.
hipError_t launch_expand_wide(const ExpandArgs& a, hipStream_t stream);

// Stage 3: mask and position ids.
struct EmitArgs {
  const int32_t* parent;
  const int32_t* depth;
  const int32_t* n_star;
  int64_t B;
  int32_t cap;
  int32_t pos_offset;
  caddtree_mask_t mask_kind;
  void* mask;              // optional
  int32_t* pos_ids;        // optional
  int32_t num_cu;          // compute units of the device
};
hipError_t launch_emit(const EmitArgs& a, hipStream_t stream);

// Synthetic acceptance of built trees against drawn target paths.
struct AcceptArgs {
  const int32_t* topk_ids;
  const float* topk_logit;
  const double* lse;
  int64_t B;
  int32_t L, K;
  const int32_t* token_ids;  // [B, tree_stride]
  const int32_t* parent;     // [B, tree_stride]
  int32_t tree_stride;
  const int32_t* n_star;
  const double* u;           // [B, L] uniforms in [0, 1)
  xp::CostTables cost;
  int32_t cap;               // the plan's cost tables cover n = 0 .. cap
  int32_t* accept_len;
  double* round_cost;        // optional
};
hipError_t launch_accept(const AcceptArgs& a, hipStream_t stream);

// Library-owned scratch for caddtree_build_noalloc (scratch.hip): one array per GPU of this many
// bytes.  noalloc_scratch_init takes its address on `device`, which must be current, once per device;
// noalloc_scratch returns that address (nullptr before a successful init).
constexpr size_t kNoAllocScratchBytes = CADDTREE_NOALLOC_SCRATCH_BYTES;
hipError_t noalloc_scratch_init(int device);
void* noalloc_scratch(int device);

// Host: convex non-decreasing least-squares fit of a cost profile (costfit.cpp); false if the
// active-set iteration did not settle.
bool fit_convex_cost(const double* x_host, const double* y_host, int n, double* fit_host, int32_t cap,
                     double* table_host);

}  // namespace caddtree
