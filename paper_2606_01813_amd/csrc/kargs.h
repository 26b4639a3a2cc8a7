// Plain data the host passes to the kernels: the plan's cost tables and the outputs an expansion
// epilogue writes.  No device code, so host-only sources can include it.
#pragma once

#include <stdint.h>

namespace caddtree {
namespace xp {

// The plan's cost tables as the kernels see them (device pointers).
struct CostTables {
  const double* tv;        // [J, cap + 1]
  const int64_t* grid;     // [J] strictly increasing context lengths (J >= 2), else unused
  const int64_t* ctx_len;  // [B] context length of each round (J >= 2), else unused
  int32_t J;
  int32_t stride;          // cap + 1
  double t_draft;
};

}  // namespace xp

// Mask and position ids written by an expansion kernel's epilogue (device pointers; both null when
// the separate emission kernel writes them).
struct EmitOut {
  void* mask;          // [B, cap, cap] u8 or [B, cap, ceil(cap / 32)] u32, or null
  int32_t* pos_ids;    // [B, cap], or null
  int mask_kind;       // caddtree_mask_t
  int pos_offset;
};

}  // namespace caddtree
