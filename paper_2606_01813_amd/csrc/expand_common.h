// Device helpers shared by the two expansion kernels (expand.hip, expand_level.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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

__host__ __device__ __forceinline__ size_t a16(size_t x) { return (x + 15) & ~(size_t)15; }

}  // namespace xp
}  // namespace caddtree
