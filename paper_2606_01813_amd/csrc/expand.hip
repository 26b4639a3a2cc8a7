// Stage 2: Algorithm 1 (Sec. 4.5) -- best-first expansion of the draft tree
// with the greedy throughput stop -- and the breadth-first layout of the
// result.  One workgroup (one wavefront) per round; the round's state lives in
// LDS.
//
// Keys.  A node s = (s_1 .. s_d) (0-based ranks) has Lambda(s) = sum_{i<=d}
// l_i^(s_i) (raw fp32 logits widened to fp64, summed in depth order) and log
// prefix probability sigma(s) = min(Lambda(s) - A_d, sigma(parent)),
// A_d = sum_{i<=d} LSE_i, sigma(root) = 0 (eq. prefix-prob; the clamp keeps a
// child from ranking above its parent under rounding).  The frontier is a
// binary max-heap under the total order: sigma desc, depth asc, Lambda desc,
// rank tuple lexicographically asc.  Every node's predecessor (previous
// sibling, or the parent for a first child) comes first in that order, so the
// heap pops nodes in exactly that order.
//
// Stop (Algorithm 1; Lemma 1): with C(n) = C_d + C_v(n), the popped node is
// kept iff ((1 + Phi) + delta) / C(n + 1) > theta_prev, delta = exp(sigma);
// the loop also ends at the budget cap or when the heap is empty.
//
// Heap entries hold sigma (fp64) and a packed (parent, rank, depth); Lambda of
// a frontier node is recomputed from its parent when a tie needs it.  Kept
// nodes hold Lambda, sigma and the packed word.  LDS per round is about
// 32 bytes x cap.
//
// Layout: kept nodes are renumbered breadth-first: the children
// of a node are ranks 0 .. c-1 (a kept node's predecessors are kept), so a
// queue walk over a child table gives depth asc, rank tuple lexicographic asc.

#include <cmath>

#include "internal.h"

namespace caddtree {
namespace {

constexpr int kThreads = 64;

// packed node word: parent index + 1 (13 bits), rank (4 bits), depth (6 bits)
__device__ __forceinline__ uint32_t pack(int parent, int rank, int depth) {
  return (uint32_t)(parent + 1) | ((uint32_t)rank << 13) | ((uint32_t)depth << 17);
}
__device__ __forceinline__ int m_parent(uint32_t m) { return (int)(m & 0x1FFFu) - 1; }
__device__ __forceinline__ int m_rank(uint32_t m) { return (int)((m >> 13) & 0xFu); }
__device__ __forceinline__ int m_depth(uint32_t m) { return (int)((m >> 17) & 0x3Fu); }

// min(a, b) that returns a unless b < a (the first argument wins ties, e.g. +0 / -0)
__device__ __forceinline__ double pmin(double a, double b) { return b < a ? b : a; }

struct Round {
  const double* A;       // [L + 1]
  const float* tl;       // [L * K] raw logits
  double* hsig;          // heap keys
  uint32_t* hmeta;
  double* slam;          // kept nodes, pop order
  double* ssig;
  uint32_t* smeta;
  int K;

  __device__ double lam_of(uint32_t m) const {
    const int p = m_parent(m);
    const double base = p >= 0 ? slam[p] : 0.0;
    return base + (double)tl[(m_depth(m) - 1) * K + m_rank(m)];
  }

  // true iff entry a pops before entry b
  __device__ bool before(double sa, uint32_t ma, double sb, uint32_t mb) const {
    if (sa != sb) return sa > sb;
    const int da = m_depth(ma), db = m_depth(mb);
    if (da != db) return da < db;
    const double la = lam_of(ma), lb = lam_of(mb);
    if (la != lb) return la > lb;
    int pa = m_parent(ma), pb = m_parent(mb), ra = m_rank(ma), rb = m_rank(mb);
    while (pa != pb) {   // same depth: walk up to the common ancestor
      const uint32_t xa = smeta[pa], xb = smeta[pb];
      ra = m_rank(xa); rb = m_rank(xb);
      pa = m_parent(xa); pb = m_parent(xb);
    }
    return ra < rb;
  }

  __device__ void sift_down(int i, int f, double s, uint32_t m) const {
    for (;;) {
      int c = 2 * i + 1;
      if (c >= f) break;
      double cs = hsig[c];
      uint32_t cm = hmeta[c];
      if (c + 1 < f) {
        const double s2 = hsig[c + 1];
        const uint32_t m2 = hmeta[c + 1];
        if (before(s2, m2, cs, cm)) { ++c; cs = s2; cm = m2; }
      }
      if (!before(cs, cm, s, m)) break;
      hsig[i] = cs; hmeta[i] = cm;
      i = c;
    }
    hsig[i] = s; hmeta[i] = m;
  }

  __device__ void sift_up(int i, double s, uint32_t m) const {
    while (i > 0) {
      const int p = (i - 1) >> 1;
      const double ps = hsig[p];
      const uint32_t pm = hmeta[p];
      if (!before(s, m, ps, pm)) break;
      hsig[i] = ps; hmeta[i] = pm;
      i = p;
    }
    hsig[i] = s; hmeta[i] = m;
  }
};

__device__ __forceinline__ size_t align16(size_t x) { return (x + 15) & ~(size_t)15; }

__global__ void __launch_bounds__(kThreads)
expand_kernel(const int32_t* __restrict__ topk_ids, const float* __restrict__ topk_logit,
              const double* __restrict__ lse, int L, int K, int cap, double t_draft,
              const double* __restrict__ tv, int32_t* __restrict__ token_ids,
              int32_t* __restrict__ parent_out, int32_t* __restrict__ depth_out,
              float* __restrict__ path_prob, int32_t* __restrict__ n_star_out,
              float* __restrict__ phi_out, float* __restrict__ theta_out) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int LK = L * K;
  const int ncap = cap > 0 ? cap : 1;

  size_t off = 0;
  double* A = reinterpret_cast<double*>(smem + off);      off = align16(off + sizeof(double) * (L + 1));
  float* tl = reinterpret_cast<float*>(smem + off);       off = align16(off + sizeof(float) * LK);
  double* slam = reinterpret_cast<double*>(smem + off);   off = align16(off + sizeof(double) * ncap);
  double* ssig = reinterpret_cast<double*>(smem + off);   off = align16(off + sizeof(double) * ncap);
  uint32_t* smeta = reinterpret_cast<uint32_t*>(smem + off); off = align16(off + sizeof(uint32_t) * ncap);
  double* hsig = reinterpret_cast<double*>(smem + off);   off = align16(off + sizeof(double) * (ncap + 1));
  uint32_t* hmeta = reinterpret_cast<uint32_t*>(smem + off); off = align16(off + sizeof(uint32_t) * (ncap + 1));
  __shared__ int s_n;

  for (int i = lane; i < LK; i += kThreads) tl[i] = topk_logit[(int64_t)b * LK + i];
  if (lane == 0) {
    A[0] = 0.0;
    for (int d = 1; d <= L; ++d) A[d] = A[d - 1] + lse[(int64_t)b * L + d - 1];
  }
  __syncthreads();

  if (lane == 0) {
    Round R{A, tl, hsig, hmeta, slam, ssig, smeta, K};
    int f = 0, n = 0;
    double phi = 0.0;
    double theta_prev = 1.0 / (t_draft + tv[0]);
    {
      const double lam = 0.0 + (double)tl[0];
      R.sift_up(f++, pmin(lam - A[1], 0.0), pack(-1, 0, 1));
    }
    double cnext = cap > 0 ? tv[1] : 0.0;
    while (f > 0 && n < cap) {
      const double sig = hsig[0];
      const uint32_t meta = hmeta[0];
      const double delta = exp(sig);
      const double theta_new = (1.0 + phi + delta) / (t_draft + cnext);
      if (theta_new <= theta_prev) break;
      const int p = m_parent(meta), r = m_rank(meta), d = m_depth(meta);
      const double base_lam = p >= 0 ? slam[p] : 0.0;
      const double base_sig = p >= 0 ? ssig[p] : 0.0;
      const double lam = base_lam + (double)tl[(d - 1) * K + r];
      slam[n] = lam; ssig[n] = sig; smeta[n] = meta;
      phi += delta;
      theta_prev = theta_new;
      const int me = n++;
      if (n < cap) cnext = tv[n + 1];
      const bool has_sib = r + 1 < K;
      bool has_child = d < L;
      double cs = 0.0; uint32_t cm = 0;
      if (has_child) {
        const double lc = lam + (double)tl[d * K];
        cs = pmin(lc - A[d + 1], sig);
        cm = pack(me, 0, d + 1);
      }
      if (has_sib) {
        const double ls = base_lam + (double)tl[(d - 1) * K + r + 1];
        R.sift_down(0, f, pmin(ls - A[d], base_sig), pack(p, r + 1, d));
      } else if (has_child) {
        R.sift_down(0, f, cs, cm);
        has_child = false;
      } else {
        --f;
        if (f > 0) R.sift_down(0, f, hsig[f], hmeta[f]);
      }
      if (has_child) R.sift_up(f++, cs, cm);
    }
    s_n = n;
    n_star_out[b] = n;
    if (phi_out) phi_out[b] = (float)phi;
    if (theta_out) theta_out[b] = (float)theta_prev;

    // breadth-first renumbering; the heap arrays are free now (>= 12 (cap + 1) bytes)
    const int nn = n;
    int16_t* cnt = reinterpret_cast<int16_t*>(hsig);  // [nn + 1], root at nn
    int16_t* cst = cnt + (nn + 1);                    // [nn + 1]
    int16_t* kids = cst + (nn + 1);                   // [nn]
    int16_t* order = kids + nn;                       // [nn]
    int16_t* pos = order + nn;                        // [nn]
    for (int i = 0; i <= nn; ++i) cnt[i] = 0;
    for (int v = 0; v < nn; ++v) {
      const int pp = m_parent(smeta[v]);
      cnt[pp < 0 ? nn : pp]++;
    }
    int acc = 0;
    for (int i = 0; i <= nn; ++i) { cst[i] = (int16_t)acc; acc += cnt[i]; }
    for (int v = 0; v < nn; ++v) {
      const uint32_t m = smeta[v];
      const int pp = m_parent(m);
      kids[cst[pp < 0 ? nn : pp] + m_rank(m)] = (int16_t)v;
    }
    int tail = 0;
    for (int k = 0; k < cnt[nn]; ++k) { const int v = kids[cst[nn] + k]; order[tail] = (int16_t)v; pos[v] = (int16_t)tail++; }
    for (int i = 0; i < nn; ++i) {
      const int u = order[i];
      for (int k = 0; k < cnt[u]; ++k) { const int v = kids[cst[u] + k]; order[tail] = (int16_t)v; pos[v] = (int16_t)tail++; }
    }
  }
  __syncthreads();

  const int n = s_n;
  const int16_t* cnt = reinterpret_cast<const int16_t*>(hsig);
  const int16_t* order = cnt + 2 * (n + 1) + n;
  const int16_t* pos = order + n;
  const int64_t ob = (int64_t)b * cap;
  for (int i = lane; i < n; i += kThreads) {
    const int v = order[i];
    const uint32_t m = smeta[v];
    const int p = m_parent(m), d = m_depth(m), r = m_rank(m);
    token_ids[ob + i] = topk_ids[(int64_t)b * LK + (d - 1) * K + r];
    parent_out[ob + i] = p < 0 ? -1 : (int)pos[p];
    depth_out[ob + i] = d;
    if (path_prob) path_prob[ob + i] = (float)exp(ssig[v]);
  }
}

}  // namespace

size_t expand_lds_bytes(int32_t L, int32_t K, int32_t cap) {
  auto a16 = [](size_t x) { return (x + 15) & ~(size_t)15; };
  const size_t ncap = cap > 0 ? (size_t)cap : 1;
  size_t off = 0;
  off = a16(off + sizeof(double) * (L + 1));
  off = a16(off + sizeof(float) * (size_t)L * K);
  off = a16(off + sizeof(double) * ncap);
  off = a16(off + sizeof(double) * ncap);
  off = a16(off + sizeof(uint32_t) * ncap);
  off = a16(off + sizeof(double) * (ncap + 1));
  off = a16(off + sizeof(uint32_t) * (ncap + 1));
  return off;
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
  const size_t lds = expand_lds_bytes(a.L, a.K, a.cap);
  hipLaunchKernelGGL(expand_kernel, dim3((unsigned)a.B), dim3(kThreads), lds, stream,
                     a.topk_ids, a.topk_logit, a.lse, a.L, a.K, a.cap, a.t_draft, a.t_verify,
                     a.token_ids, a.parent, a.depth, a.path_prob, a.n_star, a.phi, a.theta);
  return hipGetLastError();
}

}  // namespace caddtree
