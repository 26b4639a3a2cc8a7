// Stage 2: Algorithm 1 (Sec. 4.5), the serial form as a kernel -- one
// workgroup (one 64-lane wavefront) per round; the algorithm itself is in
// expand_serial.h.  It serves every round of a plan the batched form
// (expand_level.hip) does not take, and the rounds the batched form hands back
// when it cannot run them in place.

#include "expand_serial.h"
#include "internal.h"

namespace caddtree {
namespace {

__global__ void __launch_bounds__(serial::kThreads) expand_kernel(serial::Args a, int only_flagged) {
  const int b = blockIdx.x;
  if (only_flagged && a.n_star_out[b] != -1) return;   // the batched kernel finished this round
  serial::expand_round(a, b);
}

}  // namespace

size_t expand_lds_bytes(int32_t L, int32_t K, int32_t cap) {
  return serial::lds_bytes((size_t)L * K, cap > 0 ? (size_t)cap : 1);
}

hipError_t expand_prepare(int32_t L, int32_t K, int32_t cap) {
  // the attribute is per kernel, not per plan: always allow the largest plan
  (void)L; (void)K; (void)cap;
  const size_t bytes = expand_lds_bytes(CADDTREE_MAX_L, CADDTREE_MAX_K, CADDTREE_MAX_CAP);
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&expand_kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

hipError_t launch_expand(const ExpandArgs& a, hipStream_t stream) {
  if (a.B == 0) return hipSuccess;
  int only_flagged = 0;
  const size_t lds = expand_lds_bytes(a.L, a.K, a.cap);
  if (a.use_level && a.use_wide) {
    // The several-wavefront form flags the rounds it cannot settle; the serial kernel follows.  (A
    // serial form linked into it for in-place use raised its registers to 142-216 per lane: two
    // rounds no longer shared a CU, and fixed 1024 on 1024 rounds took 155 us instead of 113.)
    const hipError_t e = launch_expand_wide(a, stream);
    if (e != hipSuccess) return e;
    only_flagged = 1;
  } else if (a.use_level) {
    // The one-wavefront form runs a round it cannot settle in place when the serial layout needs at
    // most kInPlaceLds bytes, or when every round has a CU of its own and the layout fits the
    // kernel's LDS limit (reserving it then costs no occupancy); otherwise it flags the round and
    // the serial kernel follows, one more launch.
    const bool own_cu = a.B <= (int64_t)a.num_cu && lds <= expand_level_lds_limit();
    const bool in_place = lds <= kInPlaceLds || own_cu;
    const hipError_t e = launch_expand_level(a, in_place ? lds : 0, stream);
    if (e != hipSuccess) return e;
    if (in_place) return hipSuccess;
    only_flagged = 1;
  }
  const serial::Args sa{a.topk_ids, a.topk_logit, a.lse, a.L, a.K, a.cap, a.cost, a.fixed_budget ? 1 : 0,
                        a.token_ids, a.parent, a.depth, a.path_prob, a.n_star, a.phi, a.theta, a.em};
  hipLaunchKernelGGL(expand_kernel, dim3((unsigned)a.B), dim3(serial::kThreads), lds, stream, sa, only_flagged);
  return hipGetLastError();
}

}  // namespace caddtree
