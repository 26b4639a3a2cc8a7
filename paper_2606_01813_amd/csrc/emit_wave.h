// Tree-attention mask of one round written by one 64-lane wavefront (Sec. 3.3:
// each node attends to the shared context and to its own ancestors), for the
// expansion kernels' epilogues: the round's tree is already in LDS, so its mask
// rows are written without another launch.  mask[i][j] = 1 iff node j is node i
// or one of its ancestors, for i, j < n; only that n x n block is written (for
// packed masks: words below ceil(n / 32), the bits at or beyond n as zero), as
// the stand-alone emission kernel does.
//
// Trees of at most 64 nodes: lane i holds row i as a 64-bit mask and gathers its
// ancestors by pointer jumping (row |= row of the node 2^k levels up, k = 0, 1, ..:
// log2 of the depth rounds of lane permutes instead of a dependent LDS read per
// depth), then writes its own row.  Larger trees go in tiles of 64 rows: lane r
// walks row r's ancestor chain (strictly decreasing indices in breadth-first order,
// at most CADDTREE_MAX_L steps) and sets one bit per ancestor in its own row of an
// LDS bit tile; the tile is then stored with consecutive lanes on consecutive words
// (packed) or 16-byte column groups (dense u8, 16 bits spread to 16 bytes).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "caddtree.h"
#include "kargs.h"

namespace caddtree {

// round b's first mask row of an epilogue's outputs (EmitOut is in kargs.h)
__device__ __forceinline__ void* round_mask(const EmitOut& em, int b, int cap) {
  if (em.mask == nullptr || em.mask_kind == CADDTREE_MASK_NONE) return nullptr;
  if (em.mask_kind == CADDTREE_MASK_BITS32)
    return static_cast<uint32_t*>(em.mask) + (int64_t)b * cap * ((cap + 31) >> 5);
  return static_cast<uint8_t*>(em.mask) + (int64_t)b * cap * cap;
}

// LDS bytes of the bit tile for a tree of n nodes
__host__ __device__ inline size_t emit_tile_bytes(int n) {
  const int rows = n < 64 ? n : 64;
  return (size_t)rows * (size_t)((n + 31) >> 5) * 4;
}

// 4 mask bits as 4 bytes of 0/1
__device__ __forceinline__ uint32_t emit_spread4(uint32_t b) { return ((b & 0xFu) * 0x00204081u) & 0x01010101u; }

// par[i]: parent index of node i (-1 at depth 1), i < n, in LDS.  tile: LDS scratch of
// emit_tile_bytes(n) bytes, 4-byte aligned.  mask: the round's first row ([cap, cap] u8 or
// [cap, ceil(cap / 32)] u32).  Called by all 64 lanes of the wavefront.
__device__ __forceinline__ void emit_mask_wave(const int16_t* par, int n, int cap, int mask_kind, void* mask,
                                               uint32_t* tile, int lane) {
  if (n <= 0 || mask == nullptr || mask_kind == CADDTREE_MASK_NONE) return;
  const int tw = (n + 31) >> 5;                  // words per tile row = words written per mask row
  const int stride = (cap + 31) >> 5;            // words per packed mask row
  if (n <= 64) {
    const bool live = lane < n;
    int p = live ? (int)par[lane] : -1;
    if (p >= lane) p = -1;                       // a malformed parent array ends the chain
    uint64_t row = live ? (1ull << lane) : 0ull;
    // after round k, row holds the node and its 2^(k+1) - 1 nearest ancestors, and p the next one up
    for (int k = 0; k < 8 && __ballot(p >= 0); ++k) {
      const int src = p >= 0 ? p : lane;
      const uint32_t alo = (uint32_t)__shfl((int)(uint32_t)row, src);
      const uint32_t ahi = (uint32_t)__shfl((int)(uint32_t)(row >> 32), src);
      const int ap = __shfl(p, src);
      if (p >= 0) {
        row |= ((uint64_t)ahi << 32) | alo;
        p = ap;
      }
    }
    if (!live) return;
    if (mask_kind == CADDTREE_MASK_BITS32) {
      uint32_t* m = static_cast<uint32_t*>(mask) + (int64_t)lane * stride;
      for (int w = 0; w < tw; ++w) m[w] = (uint32_t)(row >> (32 * w));
    } else {
      uint8_t* rowp = static_cast<uint8_t*>(mask) + (int64_t)lane * cap;
      for (int c0 = 0; c0 < n; c0 += 16) {
        const uint32_t bits = (uint32_t)(row >> c0) & 0xFFFFu;
        const int c1 = c0 + 16 < n ? c0 + 16 : n;
        if (c1 - c0 == 16 && (reinterpret_cast<uintptr_t>(rowp + c0) & 15u) == 0) {
          uint4 q;
          q.x = emit_spread4(bits);
          q.y = emit_spread4(bits >> 4);
          q.z = emit_spread4(bits >> 8);
          q.w = emit_spread4(bits >> 12);
          *reinterpret_cast<uint4*>(rowp + c0) = q;
        } else {
          for (int c = c0; c < c1; ++c) rowp[c] = (uint8_t)((bits >> (c - c0)) & 1u);
        }
      }
    }
    return;
  }
  for (int r0 = 0; r0 < n; r0 += 64) {
    const int nr = n - r0 < 64 ? n - r0 : 64;
    for (int w = lane; w < nr * tw; w += 64) tile[w] = 0u;
    __syncthreads();
    if (lane < nr) {
      uint32_t* row = tile + lane * tw;
      const int i = r0 + lane;
      for (int j = i, steps = 0; j >= 0 && steps <= CADDTREE_MAX_L; ++steps) {
        row[j >> 5] |= 1u << (j & 31);
        const int nj = par[j];
        if (nj >= j) break;                      // a malformed parent array ends the walk
        j = nj;
      }
    }
    __syncthreads();
    if (mask_kind == CADDTREE_MASK_BITS32) {
      uint32_t* m = static_cast<uint32_t*>(mask) + (int64_t)r0 * stride;
      for (int t = lane; t < nr * tw; t += 64) {
        const int r = t / tw, w = t - r * tw;
        m[(int64_t)r * stride + w] = tile[t];
      }
    } else {
      const int groups = (n + 15) >> 4;          // 16-column groups per row
      for (int t = lane; t < nr * groups; t += 64) {
        const int r = t / groups, g = t - r * groups;
        const uint32_t bits = (tile[r * tw + (g >> 1)] >> ((g & 1) << 4)) & 0xFFFFu;
        uint8_t* rowp = static_cast<uint8_t*>(mask) + (int64_t)(r0 + r) * cap;
        const int c0 = g << 4, c1 = c0 + 16 < n ? c0 + 16 : n;
        if (c1 - c0 == 16 && (reinterpret_cast<uintptr_t>(rowp + c0) & 15u) == 0) {
          uint4 q;
          q.x = emit_spread4(bits);
          q.y = emit_spread4(bits >> 4);
          q.z = emit_spread4(bits >> 8);
          q.w = emit_spread4(bits >> 12);
          *reinterpret_cast<uint4*>(rowp + c0) = q;
        } else {
          for (int c = c0; c < c1; ++c) rowp[c] = (uint8_t)((bits >> (c - c0)) & 1u);
        }
      }
    }
    __syncthreads();                             // the tile is reused by the next 64 rows
  }
}

}  // namespace caddtree
