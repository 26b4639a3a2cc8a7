// Stage 3: tree-attention mask and position ids (Sec. 3.3: each node attends to
// the shared context and to its own ancestors).  mask[i][j] = 1 iff node j is
// node i or one of its ancestors, for i, j < n_star; pos[i] = pos_offset +
// depth[i] (the root, the bonus token, sits at pos_offset).
//
// Grid: (round, tile of 64 rows).  The round's parent array (indices < the
// tile's last row) is staged in LDS; each thread produces one 32-column word of
// one row by walking the row's ancestor chain, which is strictly decreasing in
// the breadth-first numbering, so the walk stops as soon as it falls below the
// word.  Packed masks store the word; dense masks expand it to 32 bytes, stored
// as two 16-byte writes where the row allows it.

#include "internal.h"

namespace caddtree {
namespace {

constexpr int kRows = 64;
constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads)
emit_kernel(const int32_t* __restrict__ parent, const int32_t* __restrict__ depth,
            const int32_t* __restrict__ n_star, int cap, int pos_offset, int mask_kind,
            void* __restrict__ mask, int32_t* __restrict__ pos_ids) {
  __shared__ int16_t par[CADDTREE_MAX_CAP];
  const int b = blockIdx.x;
  const int n = min(max(n_star[b], 0), cap);
  const int r0 = blockIdx.y * kRows;
  if (r0 >= n) return;
  const int r1 = min(n, r0 + kRows);
  const int64_t ob = (int64_t)b * cap;
  for (int i = threadIdx.x; i < r1; i += kThreads) par[i] = (int16_t)parent[ob + i];
  if (pos_ids)
    for (int i = r0 + (int)threadIdx.x; i < r1; i += kThreads) pos_ids[ob + i] = pos_offset + depth[ob + i];
  if (mask == nullptr || mask_kind == CADDTREE_MASK_NONE) return;
  __syncthreads();

  const int words = (n + 31) >> 5;
  const int items = (r1 - r0) * words;
  for (int it = threadIdx.x; it < items; it += kThreads) {
    const int i = r0 + it / words;
    const int w = it - (it / words) * words;
    const int lo = w << 5;
    uint32_t bits = 0;
    // the chain is strictly decreasing; a malformed parent array ends the walk
    for (int j = i, steps = 0; j >= lo && steps <= CADDTREE_MAX_L; ++steps) {
      if (j < lo + 32) bits |= 1u << (j - lo);
      const int nj = par[j];
      if (nj >= j) break;
      j = nj;
    }
    if (mask_kind == CADDTREE_MASK_BITS32) {
      const int64_t stride = (cap + 31) >> 5;
      static_cast<uint32_t*>(mask)[(ob + i) * stride + w] = bits;
    } else {
      uint8_t* rowp = static_cast<uint8_t*>(mask) + (ob + i) * cap;
      const int hi = min(n, lo + 32);
      if (hi - lo == 32 && (reinterpret_cast<uintptr_t>(rowp + lo) & 15u) == 0) {
        // 32 bytes as two 16-byte stores; (b * 0x00204081) & 0x01010101 spreads 4 bits over 4 bytes
        uint4 q[2];
        uint32_t* qw = reinterpret_cast<uint32_t*>(q);
#pragma unroll
        for (int k = 0; k < 8; ++k) qw[k] = (((bits >> (4 * k)) & 0xFu) * 0x00204081u) & 0x01010101u;
        reinterpret_cast<uint4*>(rowp + lo)[0] = q[0];
        reinterpret_cast<uint4*>(rowp + lo)[1] = q[1];
      } else {
        for (int j = lo; j < hi; ++j) rowp[j] = (uint8_t)((bits >> (j - lo)) & 1u);
      }
    }
  }
}

}  // namespace

hipError_t launch_emit(const EmitArgs& a, hipStream_t stream) {
  if (a.B == 0 || a.cap == 0) return hipSuccess;
  const dim3 grid((unsigned)a.B, (unsigned)((a.cap + kRows - 1) / kRows));
  hipLaunchKernelGGL(emit_kernel, grid, dim3(kThreads), 0, stream, a.parent, a.depth, a.n_star,
                     a.cap, a.pos_offset, (int)a.mask_kind, a.mask, a.pos_ids);
  return hipGetLastError();
}

}  // namespace caddtree
