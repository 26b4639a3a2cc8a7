// Stage 3: tree-attention mask and position ids (Sec. 3.3: each node attends to
// the shared context and to its own ancestors).  mask[i][j] = 1 iff node j is
// node i or one of its ancestors, for i, j < n_star; pos[i] = pos_offset +
// depth[i] (the root, the bonus token, sits at pos_offset).
//
// Grid: (round, group of 1-4 tiles of 64 rows), 256 threads.  The round's parent
// array (indices below the group's last row) is staged in LDS once per group,
// with 16-byte loads (staging it once per tile cost s1's 4096-row rounds about
// a sixth of the kernel's time).  Then, tile by tile, two phases:
//  1. one thread per row walks the row's ancestor chain (strictly decreasing in
//     the breadth-first numbering) and sets each ancestor's bit in the tile's
//     bit matrix in LDS (64 rows x up to 128 words);
//  2. the tile is written out row by row with consecutive threads on
//     consecutive 4-word groups (packed; single words when rows are not
//     16-byte aligned) or 16-byte column groups (dense, each 16 bits spread to
//     16 bytes), so every store instruction is coalesced.

#include <algorithm>

#include <hip/hip_runtime.h>

#include "internal.h"

namespace caddtree {
namespace {

constexpr int kRows = 64;
constexpr int kThreads = 256;
constexpr int kMaxGroup = 4;                  // tiles per workgroup, at most (the parents are staged once)

// dynamic LDS: the parent array (cap int16, rounded to 16 bytes), then the tile's bit matrix
// (kRows rows of ceil(cap / 32) words)
__host__ __device__ inline size_t par_bytes(int cap) { return ((size_t)cap * 2 + 15) & ~(size_t)15; }
__host__ __device__ inline size_t emit_lds_bytes(int cap) {
  return par_bytes(cap) + (size_t)kRows * (size_t)((cap + 31) >> 5) * 4;
}

__device__ __forceinline__ int log2_pow2_at_least(int x) {   // smallest k with 2^k >= x (x >= 1)
  int k = 0;
  while ((1 << k) < x) ++k;
  return k;
}

// 4 mask bits as 4 bytes of 0/1: (b * 0x00204081) & 0x01010101
__device__ __forceinline__ uint32_t spread4(uint32_t b) { return ((b & 0xFu) * 0x00204081u) & 0x01010101u; }

__global__ void __launch_bounds__(kThreads)
emit_kernel(const int32_t* __restrict__ parent, const int32_t* __restrict__ depth,
            const int32_t* __restrict__ n_star, int cap, int pos_offset, int mask_kind,
            void* __restrict__ mask, int32_t* __restrict__ pos_ids, int group) {
  extern __shared__ __align__(16) unsigned char smem[];
  int16_t* par = reinterpret_cast<int16_t*>(smem);
  uint32_t* tile = reinterpret_cast<uint32_t*>(smem + par_bytes(cap));   // [kRows][tw]
  const int tw = (cap + 31) >> 5;
  const int b = blockIdx.x;
  const int n = min(max(n_star[b], 0), cap);
  const int g0 = blockIdx.y * group * kRows;    // the group's first row
  if (g0 >= n) return;
  const int g1 = min(n, g0 + group * kRows);
  const int64_t ob = (int64_t)b * cap;
  const bool want_mask = mask != nullptr && mask_kind != CADDTREE_MASK_NONE;
  if (pos_ids)
    for (int i = g0 + (int)threadIdx.x; i < g1; i += kThreads) pos_ids[ob + i] = pos_offset + depth[ob + i];
  if (!want_mask) return;
  const int32_t* pr = parent + ob;
  const bool vec = (reinterpret_cast<uintptr_t>(pr) & 15u) == 0;
  // the parents of rows below the group's end, with 16-byte loads of whole 4-entry groups, all of a
  // thread's groups issued at once (indices clamped, so no load waits behind a branch)
  static_assert(4 * 4 * kThreads >= CADDTREE_MAX_CAP, "one pass of 16-byte loads covers the largest cap");
  const int n4 = vec ? g1 >> 2 : 0;
  const int4* p4 = reinterpret_cast<const int4*>(pr);
  if (n4 > 0) {
    int4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = p4[min((int)threadIdx.x + u * kThreads, n4 - 1)];
    uint2* par2 = reinterpret_cast<uint2*>(par);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int g = (int)threadIdx.x + u * kThreads;
      if (g < n4)
        par2[g] = make_uint2(((uint32_t)v[u].x & 0xFFFFu) | ((uint32_t)v[u].y << 16),
                             ((uint32_t)v[u].z & 0xFFFFu) | ((uint32_t)v[u].w << 16));
    }
  }
  for (int i = (n4 << 2) + (int)threadIdx.x; i < g1; i += kThreads) par[i] = (int16_t)pr[i];
  const int words = (n + 31) >> 5;

  for (int r0 = g0; r0 < g1; r0 += kRows) {   // the group's tiles of 64 rows
    const int r1 = min(g1, r0 + kRows);
    const int nr = r1 - r0;
    {                                         // clear the rows in use, 16 bytes at a time
      const int zw = nr * tw;
      uint4* t4 = reinterpret_cast<uint4*>(tile);
      for (int g = threadIdx.x; g < (zw >> 2); g += kThreads) t4[g] = make_uint4(0u, 0u, 0u, 0u);
      for (int w = ((zw >> 2) << 2) + (int)threadIdx.x; w < zw; w += kThreads) tile[w] = 0u;
    }
    __syncthreads();                          // parents staged (first tile), tile cleared

    // 1. ancestor bits, one thread per row; the chain is strictly decreasing, and a malformed
    //    parent array ends the walk
    if ((int)threadIdx.x < nr) {
      const int i = r0 + (int)threadIdx.x;
      for (int j = i, steps = 0; j >= 0 && steps <= CADDTREE_MAX_L; ++steps) {
        atomicOr(&tile[(i - r0) * tw + (j >> 5)], 1u << (j & 31));
        const int nj = par[j];
        if (nj >= j) break;
        j = nj;
      }
    }
    __syncthreads();

    // 2. stores
    if (mask_kind == CADDTREE_MASK_BITS32) {
      const int64_t stride = tw;
      uint32_t* mrow = static_cast<uint32_t*>(mask) + (ob + r0) * stride;
      if ((tw & 3) == 0 && (reinterpret_cast<uintptr_t>(mask) & 15u) == 0) {
        // rows start on 16 bytes in LDS and in the mask: 4-word groups, one 16-byte store each
        // (the group that holds the row's last used word stores only the used words)
        const int gw = (words + 3) >> 2;
        const int lg = log2_pow2_at_least(gw);   // groups per row, padded to a power of two
        for (int t = threadIdx.x; t < (nr << lg); t += kThreads) {
          const int r = t >> lg, g = t & ((1 << lg) - 1);
          if (g >= gw) continue;
          const int w = g << 2;
          const uint4 v = *reinterpret_cast<const uint4*>(tile + r * tw + w);
          uint32_t* dst = mrow + r * stride + w;
          if (w + 4 <= words) {
            *reinterpret_cast<uint4*>(dst) = v;
          } else {
            dst[0] = v.x;
            if (w + 1 < words) dst[1] = v.y;
            if (w + 2 < words) dst[2] = v.z;
          }
        }
      } else {
        const int lw = log2_pow2_at_least(words);   // words per row, padded to a power of two
        for (int t = threadIdx.x; t < (nr << lw); t += kThreads) {
          const int r = t >> lw, w = t & ((1 << lw) - 1);
          if (w < words) mrow[r * stride + w] = tile[r * tw + w];
        }
      }
    } else {
      const int groups = (n + 15) >> 4;
      const int lg = log2_pow2_at_least(groups);
      for (int t = threadIdx.x; t < (nr << lg); t += kThreads) {
        const int r = t >> lg, g = t & ((1 << lg) - 1);
        if (g >= groups) continue;
        const uint32_t bits = (tile[r * tw + (g >> 1)] >> ((g & 1) << 4)) & 0xFFFFu;
        uint8_t* rowp = static_cast<uint8_t*>(mask) + (ob + r0 + r) * cap;
        const int c0 = g << 4, c1 = min(n, c0 + 16);
        if (c1 - c0 == 16 && (reinterpret_cast<uintptr_t>(rowp + c0) & 15u) == 0) {
          uint4 q;
          q.x = spread4(bits);
          q.y = spread4(bits >> 4);
          q.z = spread4(bits >> 8);
          q.w = spread4(bits >> 12);
          *reinterpret_cast<uint4*>(rowp + c0) = q;
        } else {
          for (int c = c0; c < c1; ++c) rowp[c] = (uint8_t)((bits >> (c - c0)) & 1u);
        }
      }
    }
    __syncthreads();                          // the tile is read before the next one clears it
  }
}

}  // namespace

// Tiles per workgroup: as many as keep about four workgroups per CU over the grid (a workgroup of
// the largest cap holds 40 KB of LDS), at most kMaxGroup.
hipError_t launch_emit(const EmitArgs& a, hipStream_t stream) {
  if (a.B == 0 || a.cap == 0) return hipSuccess;
  const int64_t tiles = a.B * (int64_t)((a.cap + kRows - 1) / kRows);
  const int64_t want = 4 * (int64_t)(a.num_cu > 0 ? a.num_cu : 256);
  const int group = (int)std::min<int64_t>(kMaxGroup, std::max<int64_t>(1, tiles / want));
  const dim3 grid((unsigned)a.B, (unsigned)((a.cap + group * kRows - 1) / (group * kRows)));
  hipLaunchKernelGGL(emit_kernel, grid, dim3(kThreads), emit_lds_bytes(a.cap), stream, a.parent, a.depth, a.n_star,
                     a.cap, a.pos_offset, (int)a.mask_kind, a.mask, a.pos_ids, group);
  return hipGetLastError();
}

}  // namespace caddtree
