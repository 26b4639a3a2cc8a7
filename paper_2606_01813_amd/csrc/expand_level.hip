// Stage 2, batched form: Algorithm 1 (Sec. 4.5) evaluated over a threshold set.
//
// Algorithm 1 pops nodes in the order sigma desc, depth asc, Lambda desc, rank
// tuple asc (see expand.hip for the keys) and keeps them while theta rises.
// Every node outside T(tau) = {nodes with sigma >= tau} comes after every node
// inside it, so the first |T(tau)| pops are T(tau) in that order.  One
// workgroup (one wavefront) per round:
//
//  1. build T(tau) level by level from the root.  The children of a node that
//     reach the threshold are a prefix of its ranks (sigma falls with the rank),
//     so each lane counts its node's children, an exclusive scan gives their
//     slots, and the set comes out in breadth-first order (depth, then rank
//     tuple), which is also the tie-break of the pop order within a depth;
//  2. rank the set by the pop order (each lane counts the nodes before its own;
//     exact sigma ties fall back to depth, Lambda and generation order);
//  3. run the stop rule: Phi accumulates in pop order exactly as the sequential
//     loop does (one lane), theta for every position follows in parallel, and
//     the first position whose theta does not rise (or the cap) ends the tree;
//  4. if every node of T(tau) was kept and the tree continues below tau, lower
//     tau and start again; if T(tau) outgrows its LDS capacity, raise tau
//     (bisection between the two).
//
// The initial tau comes from the cost model: a node kept at a position near n
// has delta > (1 + Phi) c_{n+1} / C(n) (Lemma 1), so the stop lies around
// log(2 c_1 / C(32)).  A round that does not settle within kMaxAttempts, or
// whose tree needs more than kSCap nodes, is flagged (n_star = -1) and left to
// the serial kernel, which gives the same result.  Costs with a flat start
// (c_1 = 0) go straight to the serial kernel: the threshold search converges
// slowly there.
//
// The kept nodes are a prefix of the pop order and a prefix-closed set, so
// their breadth-first positions are a running count over generation order.

#include <cmath>

#include "expand_common.h"
#include "internal.h"

namespace caddtree {
namespace {

using namespace xp;

constexpr int kW = 64;
constexpr int kSCap = 256;        // nodes of T(tau) held at once
constexpr int kMaxAttempts = 14;

__device__ __forceinline__ int excl_scan(int v, int lane, int* total) {
  int x = v;
#pragma unroll
  for (int o = 1; o < kW; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  *total = __shfl(x, kW - 1);
  return x - v;
}

struct Lds {
  float* tl;        // [L * K] raw logits
  int32_t* tid;     // [L * K] token ids
  double* cw;       // [W] C(0 .. W - 1) = C_d + C_v
  double* sig;      // T(tau), generation order
  double* lam;
  uint32_t* meta;
  int16_t* rnk;     // pop-order rank of each node of T(tau)
  int16_t* pos;     // breadth-first position of each kept node
  double* dsort;    // delta in pop order
  double* P;        // Phi before each position
  double* th;       // theta_new at each position
};

__host__ __device__ __forceinline__ size_t level_lds_bytes(size_t LK, size_t W) {
  size_t off = 0;
  off = a16(off + 4 * LK);
  off = a16(off + 4 * LK);
  off = a16(off + 8 * W);
  off = a16(off + 8 * kSCap);
  off = a16(off + 8 * kSCap);
  off = a16(off + 4 * kSCap);
  off = a16(off + 2 * kSCap);
  off = a16(off + 2 * kSCap);
  off = a16(off + 8 * kSCap);
  off = a16(off + 8 * (kSCap + 1));
  off = a16(off + 8 * kSCap);
  return off;
}

__device__ Lds carve(unsigned char* smem, size_t LK, size_t W) {
  Lds s;
  size_t off = 0;
  s.tl = reinterpret_cast<float*>(smem + off);      off = a16(off + 4 * LK);
  s.tid = reinterpret_cast<int32_t*>(smem + off);   off = a16(off + 4 * LK);
  s.cw = reinterpret_cast<double*>(smem + off);     off = a16(off + 8 * W);
  s.sig = reinterpret_cast<double*>(smem + off);    off = a16(off + 8 * kSCap);
  s.lam = reinterpret_cast<double*>(smem + off);    off = a16(off + 8 * kSCap);
  s.meta = reinterpret_cast<uint32_t*>(smem + off); off = a16(off + 4 * kSCap);
  s.rnk = reinterpret_cast<int16_t*>(smem + off);   off = a16(off + 2 * kSCap);
  s.pos = reinterpret_cast<int16_t*>(smem + off);   off = a16(off + 2 * kSCap);
  s.dsort = reinterpret_cast<double*>(smem + off);  off = a16(off + 8 * kSCap);
  s.P = reinterpret_cast<double*>(smem + off);      off = a16(off + 8 * (kSCap + 1));
  s.th = reinterpret_cast<double*>(smem + off);
  return s;
}

__global__ void __launch_bounds__(kW)
expand_level_kernel(const int32_t* __restrict__ topk_ids, const float* __restrict__ topk_logit,
                    const double* __restrict__ lse, int L, int K, int cap, CostTables ct, int fixed,
                    int32_t* __restrict__ token_ids,
                    int32_t* __restrict__ parent_out, int32_t* __restrict__ depth_out,
                    float* __restrict__ path_prob, int32_t* __restrict__ n_star_out,
                    float* __restrict__ phi_out, float* __restrict__ theta_out) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int LK = L * K;
  const int W = (cap < kSCap ? cap : kSCap) + 2;
  const Lds s = carve(smem, (size_t)LK, (size_t)W);
  const RoundCost C = ct.round(b);

  for (int i = lane; i < LK; i += kW) {
    s.tl[i] = topk_logit[(int64_t)b * LK + i];
    s.tid[i] = topk_ids[(int64_t)b * LK + i];
  }
  for (int i = lane; i < W; i += kW) s.cw[i] = i <= cap ? C(i) : 1.0;
  // lane d holds A_d = sum_{i<=d} LSE_i, summed in depth order (d = 0 .. L)
  const double lse_l = lane < L ? lse[(int64_t)b * L + lane] : 0.0;
  double Areg = 0.0;
  {
    double acc = 0.0;
    for (int d = 1; d <= L; ++d) {
      acc = acc + rl_d(lse_l, d - 1);
      if (lane == d) Areg = acc;
    }
  }
  __syncthreads();

  const double theta0 = 1.0 / s.cw[0];
  const double A1 = rl_d(Areg, 1);
  const double top = pmin(0.0 + (double)s.tl[0] - A1, 0.0);   // the first node to pop
  double tau = top - 3.0;
  if (!fixed && s.cw[1] - s.cw[0] > 0.0) {
    const int m = cap < 32 ? cap : 32;
    tau = log(2.0 * (s.cw[1] - s.cw[0]) / s.cw[m]) - 0.5;
  }
  tau = fmin(tau, top);

  double lo = -INFINITY, hi = INFINITY;
  int n = 0, ns = 0;
  double phi = 0.0, theta = theta0;
  bool done = cap == 0;
  for (int attempt = 0; attempt < kMaxAttempts && !done; ++attempt) {
    // ---- 1. T(tau), level by level
    bool over = false, cut = false;
    {
      const bool live = lane < K;
      double x = 0.0, l1 = 0.0;
      if (live) { l1 = 0.0 + (double)s.tl[lane]; x = l1 - A1; }
      const bool in = live && x >= tau;     // the ranks that qualify form a prefix
      if (in) { s.sig[lane] = pmin(x, 0.0); s.lam[lane] = l1; s.meta[lane] = pack(-1, lane, 1); }
      ns = __popcll(__ballot(in));
      cut = ns < K;
    }
    int la = 0, lb = ns;                    // the current level is [la, lb)
    for (int d = 1; d < L && la < lb && !over; ++d) {
      __syncthreads();
      const double Ad = __shfl(Areg, d + 1);
      int nb = lb;
      for (int p0 = la; p0 < lb; p0 += kW) {
        const int p = p0 + lane;
        const bool live = p < lb;
        const int pp = live ? p : la;
        const double ps = s.sig[pp], pl = s.lam[pp];
        int c = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r)
          c += (live && r < K && (pl + (double)s.tl[d * K + (r < K ? r : 0)]) - Ad >= tau) ? 1 : 0;
        int tot = 0;
        const int off = excl_scan(c, lane, &tot);
        if (live && c < K) cut = true;
        if (nb + tot > kSCap) { over = true; break; }
        for (int r = 0; r < c; ++r) {
          const int i = nb + off + r;
          const double l = pl + (double)s.tl[d * K + r];
          s.sig[i] = pmin(l - Ad, ps);
          s.lam[i] = l;
          s.meta[i] = pack(p, r, d + 1);
        }
        nb += tot;
      }
      la = lb;
      lb = nb;
    }
    cut = __ballot(cut) != 0;
    if (over) {
      lo = tau;
      tau = hi < INFINITY ? 0.5 * (tau + hi) : tau + 1.0;
      tau = fmin(tau, top);
      if (!(lo < tau)) break;               // the set cannot shrink further
      continue;
    }
    ns = lb;
    __syncthreads();

    // ---- 2. pop-order rank
    for (int i0 = 0; i0 < ns; i0 += kW) {
      const int i = i0 + lane;
      const bool live = i < ns;
      const double si = live ? s.sig[i] : INFINITY;
      int r = 0, ties = 0;
#pragma unroll 8
      for (int j = 0; j < ns; ++j) {
        const double sj = s.sig[j];
        r += sj > si ? 1 : 0;
        ties += sj == si ? 1 : 0;
      }
      if (__ballot(live && ties > 1)) {
        const int di = live ? m_depth(s.meta[i]) : 0;
        const double li = live ? s.lam[i] : 0.0;
        int rt = 0;
#pragma unroll 8
        for (int j = 0; j < ns; ++j) {
          const double sj = s.sig[j], lj = s.lam[j];
          const int dj = m_depth(s.meta[j]);
          rt += (sj == si && j != i && (dj < di || (dj == di && (lj > li || (lj == li && j < i))))) ? 1 : 0;
        }
        r += (live && ties > 1) ? rt : 0;
      }
      if (live) {
        s.rnk[i] = (int16_t)r;
        s.dsort[r] = exp(si);
      }
    }
    __syncthreads();

    // ---- 3. stop rule
    if (lane == 0) {
      double acc = 0.0;
      for (int k = 0; k < ns; ++k) { s.P[k] = acc; acc = acc + s.dsort[k]; }
      s.P[ns] = acc;
    }
    __syncthreads();
    for (int k = lane; k < ns; k += kW) {
      if (k < cap) {
        const int m = k + 1;
        const double c = m < W ? s.cw[m] : C(m);
        s.th[k] = (1.0 + s.P[k] + s.dsort[k]) / c;
      }
    }
    __syncthreads();
    int kk = ns;
    for (int k0 = 0; k0 < ns; k0 += kW) {
      const int k = k0 + lane;
      bool stop = false;
      if (k < ns) stop = k >= cap || (!fixed && s.th[k] <= (k == 0 ? theta0 : s.th[k - 1]));
      const unsigned long long ms = __ballot(stop);
      if (ms) { kk = k0 + __builtin_ctzll(ms); break; }
    }
    if (kk < ns || kk >= cap || !cut) {     // stopped inside, hit the cap, or the whole tree is here
      n = kk;
      phi = s.P[kk];
      theta = kk == 0 ? theta0 : s.th[kk - 1];
      done = true;
    } else {                                // every node kept: the stop lies below tau
      hi = tau;
      tau = lo > -INFINITY ? 0.5 * (tau + lo) : tau - 1.5;
    }
  }
  if (!done) {
    if (lane == 0) n_star_out[b] = -1;      // left to the serial kernel
    return;
  }
  if (lane == 0) {
    n_star_out[b] = n;
    if (phi_out) phi_out[b] = (float)phi;
    if (theta_out) theta_out[b] = (float)theta;
  }
  if (n == 0) return;

  // ---- breadth-first positions: kept nodes before this one in generation order
  int base = 0;
  for (int i0 = 0; i0 < ns; i0 += kW) {
    const int i = i0 + lane;
    const bool kept = i < ns && s.rnk[i] < n;
    const unsigned long long m = __ballot(kept);
    const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
    if (kept) s.pos[i] = (int16_t)(base + below);
    base += __popcll(m);
  }
  __syncthreads();
  const int64_t ob = (int64_t)b * cap;
  for (int i = lane; i < ns; i += kW) {
    if (s.rnk[i] < n) {
      const uint32_t m = s.meta[i];
      const int p = m_parent(m), d = m_depth(m), r = m_rank(m);
      const int o = s.pos[i];
      token_ids[ob + o] = s.tid[(d - 1) * K + r];
      parent_out[ob + o] = p < 0 ? -1 : (int)s.pos[p];
      depth_out[ob + o] = d;
      if (path_prob) path_prob[ob + o] = (float)exp(s.sig[i]);
    }
  }
}

}  // namespace

size_t expand_level_lds_bytes(int32_t L, int32_t K, int32_t cap) {
  const size_t W = (cap < kSCap ? (size_t)cap : kSCap) + 2;
  return level_lds_bytes((size_t)L * K, W);
}

hipError_t launch_expand_level(const ExpandArgs& a, hipStream_t stream) {
  if (a.B == 0) return hipSuccess;
  hipLaunchKernelGGL(expand_level_kernel, dim3((unsigned)a.B), dim3(kW), expand_level_lds_bytes(a.L, a.K, a.cap),
                     stream, a.topk_ids, a.topk_logit, a.lse, a.L, a.K, a.cap, a.cost, a.fixed_budget ? 1 : 0,
                     a.token_ids, a.parent, a.depth, a.path_prob, a.n_star, a.phi, a.theta);
  return hipGetLastError();
}

}  // namespace caddtree
