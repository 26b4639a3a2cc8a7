// Device helpers shared by the two expansion kernels (expand.hip, expand_level.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kargs.h"

namespace caddtree {
namespace xp {

// packed node word: parent index + 1 (13 bits), rank (4 bits), depth (6 bits)
__device__ __forceinline__ uint32_t pack(int parent, int rank, int depth) {
  return (uint32_t)(parent + 1) | ((uint32_t)rank << 13) | ((uint32_t)depth << 17);
}
__device__ __forceinline__ int m_parent(uint32_t m) { return (int)(m & 0x1FFFu) - 1; }
__device__ __forceinline__ int m_rank(uint32_t m) { return (int)((m >> 13) & 0xFu); }
__device__ __forceinline__ int m_depth(uint32_t m) { return (int)((m >> 17) & 0x3Fu); }

// min(a, b) that returns a unless b < a (the first argument wins ties, e.g. +0 / -0)
__device__ __forceinline__ double pmin(double a, double b) { return b < a ? b : a; }

// value of lane l (l must be wave-uniform)
__device__ __forceinline__ double rl_d(double v, int l) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ uint32_t rl_u(uint32_t v, int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); }

__host__ __device__ constexpr size_t a16(size_t x) { return (x + 15) & ~(size_t)15; }

// ---- wave scans through DPP (gfx9: row_shr within 16-lane rows, then row_bcast:15 / :31 across rows)
template <int CTRL, int ROW_MASK, bool BOUND>
__device__ __forceinline__ int dpp_i(int old, int v) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, ROW_MASK, 0xF, BOUND);
}
template <int CTRL, int ROW_MASK, bool BOUND>
__device__ __forceinline__ double dpp_d(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)dpp_i<CTRL, ROW_MASK, BOUND>(0, (int)(uint32_t)u);
  const uint32_t hi = (uint32_t)dpp_i<CTRL, ROW_MASK, BOUND>(0, (int)(uint32_t)(u >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// inclusive prefix sum over the 64 lanes (lane order)
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += dpp_i<0x111, 0xF, true>(0, x);
  x += dpp_i<0x112, 0xF, true>(0, x);
  x += dpp_i<0x114, 0xF, true>(0, x);
  x += dpp_i<0x118, 0xF, true>(0, x);
  x += dpp_i<0x142, 0xA, false>(0, x);
  x += dpp_i<0x143, 0xC, false>(0, x);
  return x;
}
__device__ __forceinline__ double wave_incl_scan(double x) {
  x += dpp_d<0x111, 0xF, true>(x);
  x += dpp_d<0x112, 0xF, true>(x);
  x += dpp_d<0x114, 0xF, true>(x);
  x += dpp_d<0x118, 0xF, true>(x);
  x += dpp_d<0x142, 0xA, false>(x);
  x += dpp_d<0x143, 0xC, false>(x);
  return x;
}
// the value of lane - 1 (0 in lane 0)
__device__ __forceinline__ double wave_shr1(double x) { return dpp_d<0x138, 0xF, true>(x); }

// Round cost C(n) = C_d + C_v(n; l) (Sec. 4.2).  With a context-length grid
// L_0 < .. < L_{J-1} and one table C_v(.; L_j) per grid point (Sec. 4.6), a
// round at context length l with L_j <= l < L_{j+1} uses the linear
// interpolation of eq. cv-interp, alpha = (l - L_j) / (L_{j+1} - L_j); l at or
// outside either end of the grid takes that end's table.  Each product and the
// sum are rounded separately (no fused multiply-add), so the value does not
// depend on the compiler's contraction choices.
struct RoundCost {
  const double* lo;   // C_v(.; L_j), cap + 1 values
  const double* hi;   // C_v(.; L_{j+1}) (== lo when alpha == 0)
  double alpha;
  double t_draft;

  // C(n) from the two tables' entries lo[n] and hi[n]
  __device__ __forceinline__ double mix(double l, double h) const {
#pragma clang fp contract(off)
    const double cv = (1.0 - alpha) * l + alpha * h;
    return t_draft + cv;
  }
  __device__ __forceinline__ double operator()(int n) const { return mix(lo[n], hi[n]); }
};

// The cost of round b (CostTables, the plan's tables as the kernels see them, is in kargs.h).
__device__ __forceinline__ RoundCost round_cost(const CostTables& ct, int64_t b) {
  RoundCost c{ct.tv, ct.tv, 0.0, ct.t_draft};
  if (ct.J >= 2) {
    const int64_t ell = ct.ctx_len[b];
    if (ell >= ct.grid[ct.J - 1]) {
      c.lo = c.hi = ct.tv + (int64_t)(ct.J - 1) * ct.stride;
    } else if (ell > ct.grid[0]) {
      int j = 0;
      while (ct.grid[j + 1] <= ell) ++j;
      c.lo = ct.tv + (int64_t)j * ct.stride;
      c.hi = c.lo + ct.stride;
      c.alpha = (double)(ell - ct.grid[j]) / (double)(ct.grid[j + 1] - ct.grid[j]);
    }
  }
  return c;
}

// round_cost computed by a whole wavefront (all 64 lanes call it; J <= 64): the context length and
// every grid point are loaded at once, lane j taking L_j, and the grid points at or below l are
// counted with one ballot, so the search takes one round trip instead of one per grid step.  The
// same table choice and alpha as round_cost.
__device__ __forceinline__ RoundCost round_cost_wave(const CostTables& ct, int64_t b, int lane) {
  RoundCost c{ct.tv, ct.tv, 0.0, ct.t_draft};
  if (ct.J >= 2) {
    const int64_t ell = ct.ctx_len[b];
    const int64_t g = ct.grid[lane < ct.J ? lane : ct.J - 1];
    const int below = __popcll(__ballot(lane < ct.J && g <= ell));   // L_0 .. L_{below - 1} <= l
    auto lane_i64 = [&](int l) -> int64_t {
      const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)g, l);
      const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)g >> 32), l);
      return (int64_t)(((uint64_t)hi << 32) | lo);
    };
    if (below >= ct.J) {                                             // l >= L_{J-1}
      c.lo = c.hi = ct.tv + (int64_t)(ct.J - 1) * ct.stride;
    } else if (below >= 1 && ell > lane_i64(0)) {                    // L_0 < l < L_{J-1}
      const int j = below - 1;                                       // L_j <= l < L_{j+1}
      const int64_t gj = lane_i64(j), gj1 = lane_i64(j + 1);
      c.lo = ct.tv + (int64_t)j * ct.stride;
      c.hi = c.lo + ct.stride;
      c.alpha = (double)(ell - gj) / (double)(gj1 - gj);
    }
  }
  return c;
}

}  // namespace xp
}  // namespace caddtree
