// Synthetic acceptance: tree verification (Sec. 3.3) of each round's draft
// tree against a target continuation drawn from the drafter's factorised
// distribution (eq. factorized), under which the expected accepted length is
// Phi(T) (eq. surrogate).
//
// Position i's target token comes from the caller's uniform u_i by inverse
// transform over the kept tokens in rank order: q^(k) = exp(l^(k) - LSE_i),
// cumulative sums formed left to right in fp64, the first rank whose sum
// exceeds u_i; past the last one the token lies outside the top-K and no node
// carries it.  alpha is the length of the longest drawn prefix that is a path
// of the tree.  The round's cost C(n*) = C_d + C_v(n*; l) (Sec. 4.2) comes
// from the plan's cost model, so that throughput sum (1 + alpha) / sum C can
// be formed over the batch.
//
// One wavefront per round: lane i draws position i; the walk then looks for
// the child of the current node that carries the drawn token, scanning the
// breadth-first node list from just past the current node (children follow
// their parent in that order) with one ballot per 64 nodes.

#include "expand_common.h"
#include "internal.h"

namespace caddtree {
namespace {

constexpr int kW = 64;

__global__ void __launch_bounds__(kW)
accept_kernel(const int32_t* __restrict__ topk_ids, const float* __restrict__ topk_logit,
              const double* __restrict__ lse, int L, int K, const int32_t* __restrict__ token_ids,
              const int32_t* __restrict__ parent, int tree_stride, const int32_t* __restrict__ n_star,
              const double* __restrict__ u, xp::CostTables ct, int cap, int32_t* __restrict__ accept_len,
              double* __restrict__ round_cost) {
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  int tok = -1;
  if (lane < L) {
    const int64_t row = b * L + lane;
    const double ul = u[row];
    const double ls = lse[row];
    double c = 0.0;
    for (int r = 0; r < K; ++r) {
      c = c + exp((double)topk_logit[row * K + r] - ls);
      if (ul < c) {
        tok = topk_ids[row * K + r];
        break;
      }
    }
  }
  const int ns = n_star[b];
  const int n = min(max(ns, 0), tree_stride);
  const int64_t ob = b * tree_stride;
  int cur = -1, alpha = 0, start = 0;
  for (int d = 0; d < L; ++d) {
    const int t = __shfl(tok, d);
    if (t < 0) break;
    int found = -1;
    for (int i0 = start; i0 < n; i0 += kW) {
      const int i = i0 + lane;
      const bool hit = i < n && parent[ob + i] == cur && token_ids[ob + i] == t;
      const unsigned long long m = __ballot(hit);
      if (m) {
        found = i0 + __builtin_ctzll(m);
        break;
      }
    }
    if (found < 0) break;
    cur = found;
    start = found + 1;
    ++alpha;
  }
  if (lane == 0) {
    accept_len[b] = alpha;
    if (round_cost) round_cost[b] = (ns >= 0 && ns <= cap) ? xp::round_cost(ct, b)(ns) : NAN;
  }
}

}  // namespace

hipError_t launch_accept(const AcceptArgs& a, hipStream_t stream) {
  if (a.B == 0) return hipSuccess;
  hipLaunchKernelGGL(accept_kernel, dim3((unsigned)a.B), dim3(kW), 0, stream, a.topk_ids, a.topk_logit, a.lse,
                     a.L, a.K, a.token_ids, a.parent, a.tree_stride, a.n_star, a.u, a.cost, a.cap, a.accept_len,
                     a.round_cost);
  return hipGetLastError();
}

}  // namespace caddtree
