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
//     so each lane counts its node's children, a prefix sum gives their slots,
//     and the set comes out in breadth-first order (depth, then rank tuple),
//     which is also the tie-break of the pop order within a depth;
//  2. find where the greedy stop falls along the pop order of T(tau):
//     * up to 64 nodes: each lane ranks its node by counting the nodes that
//       pop before it (the full order with its tie-breaks, one pass), the
//       path probabilities are scattered into pop order, a prefix sum gives
//       Phi before every position m, and m is kept iff
//       (1 + Phi_m + delta_m) / C(m + 1) > (1 + Phi_m) / C(m) and m < cap;
//     * larger sets: under a convex cost theta rises and then falls along the
//       pop order (Thm. 1), so "position m is kept" holds below n* and fails
//       from n* on, and a bisection over pivot nodes finds n*: a pivot's
//       position and the Phi before it are a count and a sum over the nodes
//       that pop before it;
//     with a fixed budget m is kept iff m < cap;
//  3. if every node of T(tau) is kept and the tree continues below tau, lower
//     tau and start again; if T(tau) outgrows its capacity, raise tau
//     (bisection between the two).
//
// The initial tau comes from the cost model: a node kept near position n has
// delta > (1 + Phi) c_{n+1} / C(n) (Lemma 1); with c_{m0+1} the first positive
// marginal cost the stop lies past m0, around delta = (1 + Phi) c / C with Phi
// of order one.  A round that does not settle within kMaxAttempts, or whose
// tree needs more nodes than the set holds (512, or up to 4096 for fixed
// budgets and long flat cost starts, sized by the host), is flagged
// (n_star = -1) and left to the serial kernel, which gives the same tree.
//
// The kept nodes are a prefix of the pop order and a prefix-closed set, so
// their breadth-first positions are a running count over generation order.
// Phi here is a prefix sum over the wave rather than a left-to-right sum in
// pop order: it matches the sequential sum to rounding, and the tree does not
// depend on it except at stop margins of that size.

#include <cmath>

#include "expand_common.h"
#include "internal.h"

namespace caddtree {
namespace {

using namespace xp;

constexpr int kW = 64;
constexpr int kSmall = 512;           // sets up to this size are selected in registers
constexpr int kMaxSet = 4096;         // the largest set the LDS layout holds
constexpr int kCW = 66;               // C(0 .. 65) cached in LDS
constexpr int kMaxAttempts = 12;

// One node of T(tau): sigma, Lambda, its packed word (parent, rank, depth) and
// its generation index.
struct Node {
  double s;
  double l;
  uint32_t m;
  int g;
};

// node a pops before node b (sigma desc, depth asc, Lambda desc, generation index asc;
// within a depth the generation order is the rank-tuple order)
// (branch-free: every term is evaluated, so the comparison compiles to selects)
__device__ __forceinline__ bool pops_before(double sa, double la, uint32_t ma, int ga,
                                            double sb, double lb, uint32_t mb, int gb) {
  const int da = m_depth(ma), db = m_depth(mb);
  const int t = (int)(la > lb) | ((int)(la == lb) & (int)(ga < gb));
  const int u = (int)(da < db) | ((int)(da == db) & t);
  return ((int)(sa > sb) | ((int)(sa == sb) & u)) != 0;
}
__device__ __forceinline__ bool pops_before(const Node& a, const Node& b) {
  return pops_before(a.s, a.l, a.m, a.g, b.s, b.l, b.m, b.g);
}

struct Lds {
  float* tl;        // [L * K] raw logits
  int32_t* tid;     // [L * K] token ids
  double* cw;       // [kCW] C(0 .. kCW - 1) = C_d + C_v
  double2* sl;      // T(tau) in generation order: (sigma, Lambda)
  uint32_t* meta;   //   packed word (parent, rank, depth)
  double* dl;       //   path probability (large sets), or in pop order (small sets)
  int16_t* pos;     // kept flag, then breadth-first position, of each node
};

// LDS of a round for a set of S nodes
__host__ __device__ __forceinline__ size_t level_lds_bytes(size_t LK, size_t S) {
  size_t off = 0;
  off = a16(off + 4 * LK);
  off = a16(off + 4 * LK);
  off = a16(off + 8 * kCW);
  off = a16(off + 16 * S);
  off = a16(off + 4 * S);
  off = a16(off + 8 * S);
  off = a16(off + 2 * S);
  return off;
}

__device__ Lds carve(unsigned char* smem, size_t LK, size_t S) {
  Lds s;
  size_t off = 0;
  s.tl = reinterpret_cast<float*>(smem + off);      off = a16(off + 4 * LK);
  s.tid = reinterpret_cast<int32_t*>(smem + off);   off = a16(off + 4 * LK);
  s.cw = reinterpret_cast<double*>(smem + off);     off = a16(off + 8 * kCW);
  s.sl = reinterpret_cast<double2*>(smem + off);    off = a16(off + 16 * S);
  s.meta = reinterpret_cast<uint32_t*>(smem + off); off = a16(off + 4 * S);
  s.dl = reinterpret_cast<double*>(smem + off);     off = a16(off + 8 * S);
  s.pos = reinterpret_cast<int16_t*>(smem + off);
  return s;
}

struct Cost {
  const double* cw;
  RoundCost C;
  __device__ __forceinline__ double operator()(int n) const { return n < kCW ? cw[n] : C(n); }
};

// the next, lower threshold: the target, but never at or below a threshold whose
// set overflowed (then halfway towards it)
__device__ __forceinline__ double lower_tau(double tau, double target, double lo) {
  if (lo > -INFINITY && !(target > lo)) return 0.5 * (tau + lo);
  return target;
}

struct Stop {
  int n;        // first position not kept, or ns when every position is kept
  double phi;   // Phi before position n
};

// up to 64 nodes: rank by counting, Phi by a prefix sum over pop positions;
// on a stop inside the set, the kept flags go to s.pos by generation index
__device__ Stop stop_small(const Lds& s, int ns, int cap, int fixed, const Cost& cost, int lane) {
  const bool live = lane < ns;
  const int i = live ? lane : 0;
  const double2 me = s.sl[i];
  const uint32_t mm = s.meta[i];
  int r = 0;
  int j = 0;
  for (; j + 4 <= ns; j += 4) {               // four nodes' loads in flight, then the compares
    double2 o[4];
    uint32_t om[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) { o[u] = s.sl[j + u]; om[u] = s.meta[j + u]; }
#pragma unroll
    for (int u = 0; u < 4; ++u) r += pops_before(o[u].x, o[u].y, om[u], j + u, me.x, me.y, mm, i) ? 1 : 0;
  }
  for (; j < ns; ++j) {
    const double2 o = s.sl[j];
    r += pops_before(o.x, o.y, s.meta[j], j, me.x, me.y, mm, i) ? 1 : 0;
  }
  if (live) s.dl[r] = exp(me.x);
  __syncthreads();
  const double d = lane < ns ? s.dl[lane] : 0.0;
  const double incl = wave_incl_scan(d);
  const double pe = wave_shr1(incl);          // Phi before position `lane`
  bool keep = lane < cap;
  if (keep && !fixed && lane < ns) keep = (1.0 + pe + d) / cost(lane + 1) > (1.0 + pe) / cost(lane);
  const unsigned long long fm = __ballot(lane < ns && !keep);
  if (!fm) return Stop{ns, rl_d(incl, kW - 1)};
  const int stop = __builtin_ctzll(fm);
  if (live) s.pos[lane] = r < stop ? 1 : 0;
  return Stop{stop, rl_d(pe, stop)};
}

// larger sets: bisection over pivots (P nodes per lane, position e = j * 64 + lane
// in generation order)
template <int P>
__device__ Stop stop_large(const Lds& s, int ns, int cap, int fixed, const Cost& cost, int lane, unsigned seed) {
  Node x[P];
  double dl[P];
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const int e = j * kW + lane;
    if (e < ns) {
      const double2 v = s.sl[e];
      x[j] = Node{v.x, v.y, s.meta[e], e};
      dl[j] = exp(v.x);
    } else {
      x[j] = Node{-INFINITY, 0.0, 63u << 17, e};
      dl[j] = 0.0;
    }
  }
  bool hasA = false, hasB = false;
  Node A{0.0, 0.0, 0u, 0}, B{0.0, 0.0, 0u, 0};
  int posB = 0;
  double phiB = 0.0;
  unsigned rng = seed;
  for (;;) {
    unsigned long long cm[P];
    int total = 0;
#pragma unroll
    for (int j = 0; j < P; ++j) {
      bool c = j * kW + lane < ns;
      if (hasA) c = c && pops_before(A, x[j]);
      if (hasB) c = c && pops_before(x[j], B);
      cm[j] = __ballot(c);
      total += __popcll(cm[j]);
    }
    if (total == 0) break;
    rng = rng * 1664525u + 1013904223u;
    int k = (int)((rng >> 8) % (unsigned)total);
    int pj = 0;
    unsigned long long mk = cm[0];
#pragma unroll
    for (int j = 0; j + 1 < P; ++j) {
      const int c = __popcll(cm[j]);
      if (pj == j && k >= c) { k -= c; pj = j + 1; mk = cm[j + 1]; }
    }
    const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(mk >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mk, 0));
    const int pl = __builtin_ctzll(__ballot(((mk >> lane) & 1ull) && below == k));
    Node pv{0.0, 0.0, 0u, pj * kW + pl};
    double pd = 0.0;
#pragma unroll
    for (int j = 0; j < P; ++j)
      if (j == pj) {
        pv.s = rl_d(x[j].s, pl);
        pv.l = rl_d(x[j].l, pl);
        pv.m = rl_u(x[j].m, pl);
        pd = rl_d(dl[j], pl);
      }
    int cnt = 0;
    double part = 0.0;
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const bool bf = j * kW + lane < ns && pops_before(x[j], pv);
      cnt += __popcll(__ballot(bf));
      part += bf ? dl[j] : 0.0;
    }
    const double ph = rl_d(wave_incl_scan(part), kW - 1);
    bool keep = cnt < cap;
    if (keep && !fixed) keep = (1.0 + ph + pd) / cost(cnt + 1) > (1.0 + ph) / cost(cnt);
    if (keep) { hasA = true; A = pv; }
    else { hasB = true; B = pv; posB = cnt; phiB = ph; }
  }
  if (!hasB) {
    double part = 0.0;
#pragma unroll
    for (int j = 0; j < P; ++j) part += dl[j];
    return Stop{ns, rl_d(wave_incl_scan(part), kW - 1)};
  }
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const int e = j * kW + lane;
    if (e < ns) s.pos[e] = pops_before(x[j], B) ? 1 : 0;
  }
  return Stop{posB, phiB};
}

// sets above kSmall nodes: the same bisection with the nodes read from LDS at
// every step
__device__ Stop stop_lds(const Lds& s, int ns, int cap, int fixed, const Cost& cost, int lane, unsigned seed) {
  for (int e = lane; e < ns; e += kW) s.dl[e] = exp(s.sl[e].x);
  __syncthreads();
  bool hasA = false, hasB = false;
  Node A{0.0, 0.0, 0u, 0}, B{0.0, 0.0, 0u, 0};
  int posB = 0;
  double phiB = 0.0;
  unsigned rng = seed;
  // node e lies strictly between A and B in the pop order
  auto cand = [&](int e) -> bool {
    if (e >= ns) return false;
    const double2 v = s.sl[e];
    const Node x{v.x, v.y, s.meta[e], e};
    return (!hasA || pops_before(A, x)) && (!hasB || pops_before(x, B));
  };
  for (;;) {
    int total = 0;
    for (int e0 = 0; e0 < ns; e0 += kW) total += __popcll(__ballot(cand(e0 + lane)));
    if (total == 0) break;
    rng = rng * 1664525u + 1013904223u;
    int k = (int)((rng >> 8) % (unsigned)total);
    int pe = -1;
    for (int e0 = 0; e0 < ns && pe < 0; e0 += kW) {
      const unsigned long long mk = __ballot(cand(e0 + lane));
      const int c = __popcll(mk);
      if (k < c) {
        const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(mk >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mk, 0));
        pe = e0 + __builtin_ctzll(__ballot(((mk >> lane) & 1ull) && below == k));
      } else {
        k -= c;
      }
    }
    const double2 pvv = s.sl[pe];
    const Node pv{pvv.x, pvv.y, s.meta[pe], pe};
    const double pd = s.dl[pe];
    int cnt = 0;
    double part = 0.0;
    for (int e0 = 0; e0 < ns; e0 += kW) {
      const int e = e0 + lane;
      bool bf = false;
      double de = 0.0;
      if (e < ns) {
        const double2 v = s.sl[e];
        bf = pops_before(Node{v.x, v.y, s.meta[e], e}, pv);
        de = s.dl[e];
      }
      cnt += __popcll(__ballot(bf));
      part += bf ? de : 0.0;
    }
    const double ph = rl_d(wave_incl_scan(part), kW - 1);
    bool keep = cnt < cap;
    if (keep && !fixed) keep = (1.0 + ph + pd) / cost(cnt + 1) > (1.0 + ph) / cost(cnt);
    if (keep) { hasA = true; A = pv; }
    else { hasB = true; B = pv; posB = cnt; phiB = ph; }
  }
  if (!hasB) {
    double part = 0.0;
    for (int e = lane; e < ns; e += kW) part += s.dl[e];
    return Stop{ns, rl_d(wave_incl_scan(part), kW - 1)};
  }
  for (int e = lane; e < ns; e += kW) {
    const double2 v = s.sl[e];
    s.pos[e] = pops_before(Node{v.x, v.y, s.meta[e], e}, B) ? 1 : 0;
  }
  return Stop{posB, phiB};
}

__global__ void __launch_bounds__(kW)
expand_level_kernel(const int32_t* __restrict__ topk_ids, const float* __restrict__ topk_logit,
                    const double* __restrict__ lse, int L, int K, int cap, CostTables ct, int fixed,
                    int setcap, int32_t* __restrict__ token_ids,
                    int32_t* __restrict__ parent_out, int32_t* __restrict__ depth_out,
                    float* __restrict__ path_prob, int32_t* __restrict__ n_star_out,
                    float* __restrict__ phi_out, float* __restrict__ theta_out) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int LK = L * K;
  const Lds s = carve(smem, (size_t)LK, (size_t)setcap);
  const Cost cost{s.cw, ct.round(b)};

  for (int i = lane; i < LK; i += kW) {
    s.tl[i] = topk_logit[(int64_t)b * LK + i];
    s.tid[i] = topk_ids[(int64_t)b * LK + i];
  }
  for (int i = lane; i < kCW; i += kW) s.cw[i] = i <= cap ? cost.C(i) : 1.0;
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
  int need = 1;                              // the tree holds at least this many nodes
  if (!fixed && cap >= 1) {
    // the first positive marginal cost c_{m0 + 1} (the stop lies past m0)
    int m0 = -1;
    for (int i0 = 0; i0 < setcap && i0 < cap && m0 < 0; i0 += kW) {
      const int i = i0 + lane;
      const bool up = i < cap && i < setcap && cost(i + 1) > cost(i);
      const unsigned long long m = __ballot(up);
      if (m) m0 = i0 + __builtin_ctzll(m);
    }
    if (m0 < 0 && cap <= setcap / 2) {
      need = cap;                           // flat up to the cap: every node is kept until the cap
    } else if (m0 < 0 || m0 >= setcap / 2) {
      if (lane == 0) n_star_out[b] = -1;    // flat for longer than the set holds: the serial kernel's case
      return;
    } else {
      need = m0 + 1;
      const int m = m0 + 32 < cap ? m0 + 32 : cap;
      tau = log(2.0 * (cost(m0 + 1) - cost(m0)) / cost(m)) - 0.5;
    }
  } else if (fixed) {
    need = cap;
  }
  tau = fmin(tau, top);

  double lo = -INFINITY, hi = INFINITY;
  int n = 0, ns = 0;
  double phi = 0.0, theta = theta0;
  bool all_kept = false;                    // every node of T(tau) is kept (no flags written)
  bool done = cap == 0;
  for (int attempt = 0; attempt < kMaxAttempts && !done; ++attempt) {
    // ---- 1. T(tau), level by level
    bool over = false, cut = false;
    {
      const bool live = lane < K;
      double x = 0.0, l1 = 0.0;
      if (live) { l1 = 0.0 + (double)s.tl[lane]; x = l1 - A1; }
      const bool in = live && x >= tau;     // the ranks that qualify form a prefix
      if (in) { s.sl[lane] = make_double2(pmin(x, 0.0), l1); s.meta[lane] = pack(-1, lane, 1); }
      ns = __popcll(__ballot(in));
      cut = ns < K;
    }
    int la = 0, lb = ns;                    // the current level is [la, lb)
    for (int d = 1; d < L && la < lb && !over; ++d) {
      __syncthreads();
      const double Ad = rl_d(Areg, d + 1);
      int nb = lb;
      for (int p0 = la; p0 < lb; p0 += kW) {
        const int p = p0 + lane;
        const bool live = p < lb;
        const double2 pv = s.sl[live ? p : la];
        int c = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r)
          c += (int)(r < K) & (int)((pv.y + (double)s.tl[d * K + (r < K ? r : 0)]) - Ad >= tau);
        c = live ? c : 0;
        const int incl = wave_incl_scan(c);
        const int tot = __builtin_amdgcn_readlane(incl, kW - 1);
        const int off = incl - c;
        if (live && c < K) cut = true;
        if (nb + tot > setcap) { over = true; break; }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          if (r < c) {
            const int i = nb + off + r;
            const double l = pv.y + (double)s.tl[d * K + r];
            s.sl[i] = make_double2(pmin(l - Ad, pv.x), l);
            s.meta[i] = pack(p, r, d + 1);
          }
        }
        nb += tot;
      }
      la = lb;
      lb = nb;
    }
    cut = __ballot(cut) != 0;
    if (over) {
      lo = tau;
      tau = hi < INFINITY ? 0.5 * (tau + hi) : tau + 1.5;
      tau = fmin(tau, top);
      if (!(lo < tau)) break;               // the set cannot shrink further
      continue;
    }
    ns = lb;
    if (cut && ns < need && ns < cap) {     // too few nodes to hold the stop: lower tau without selecting
      hi = tau;
      const double step = fmin(fmax(log(1.5 * (double)need / (double)(ns > 0 ? ns : 1)), 0.5), 4.0);
      tau = lower_tau(tau, tau - step, lo);
      continue;
    }
    __syncthreads();

    // ---- 2. where the stop falls
    Stop st;
    const unsigned seed = 0x9E3779B9u ^ (unsigned)b ^ ((unsigned)attempt << 16);
    if (ns <= kW) st = stop_small(s, ns, cap, fixed, cost, lane);
    else if (ns <= 2 * kW) st = stop_large<2>(s, ns, cap, fixed, cost, lane, seed);
    else if (ns <= 4 * kW) st = stop_large<4>(s, ns, cap, fixed, cost, lane, seed);
    else if (ns <= kSmall) st = stop_large<8>(s, ns, cap, fixed, cost, lane, seed);
    else st = stop_lds(s, ns, cap, fixed, cost, lane, seed);

    if (st.n < ns) {                        // the stop (or the cap) falls inside T(tau)
      n = st.n;
      phi = st.phi;
      all_kept = false;
      done = true;
    } else if (!cut || ns >= cap) {         // the whole tree (or the cap) is here and all of it is kept
      n = ns;
      phi = st.phi;
      all_kept = true;
      done = true;
    } else {                                // every node kept: the stop lies below tau
      hi = tau;
      // the next pop is kept only while delta > (1 + Phi) c_{n+1} / C(n) (Lemma 1), a bound that
      // does not fall as n grows under a convex cost: aim a little below it
      double target = tau - 1.5;
      if (!fixed) {
        const double c1 = cost(ns + 1) - cost(ns);
        if (c1 > 0.0) target = fmin(tau - 0.25, log((1.0 + st.phi) * c1 / cost(ns)) - 1.0);
      }
      tau = lower_tau(tau, target, lo);
    }
    if (done) theta = n == 0 ? theta0 : (1.0 + phi) / cost(n);
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
  __syncthreads();                          // the kept flags written by the selection
  int base = 0;
  for (int i0 = 0; i0 < ns; i0 += kW) {
    const int i = i0 + lane;
    const bool kept = i < ns && (all_kept || s.pos[i] != 0);
    const unsigned long long m = __ballot(kept);
    const int below = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
    if (i < ns) s.pos[i] = kept ? (int16_t)(base + below) : (int16_t)-1;
    base += __popcll(m);
  }
  __syncthreads();
  const int64_t ob = (int64_t)b * cap;
  for (int i = lane; i < ns; i += kW) {
    const int o = s.pos[i];
    if (o >= 0) {
      const uint32_t m = s.meta[i];
      const int p = m_parent(m), d = m_depth(m), r = m_rank(m);
      token_ids[ob + o] = s.tid[(d - 1) * K + r];
      parent_out[ob + o] = p < 0 ? -1 : (int)s.pos[p];
      depth_out[ob + o] = d;
      if (path_prob) path_prob[ob + o] = (float)exp(s.sl[i].x);
    }
  }
}

}  // namespace

size_t expand_level_lds_bytes(int32_t L, int32_t K, int32_t set_cap) {
  return level_lds_bytes((size_t)L * K, (size_t)set_cap);
}

int expand_level_set_cap(int32_t need) {
  int S = kSmall;
  while (S < kMaxSet && S < 2 * need) S *= 2;
  return S;
}

int expand_level_max_need() { return kMaxSet / 2; }

hipError_t expand_level_prepare() {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&expand_level_kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)level_lds_bytes((size_t)CADDTREE_MAX_L * CADDTREE_MAX_K, kMaxSet));
}

hipError_t launch_expand_level(const ExpandArgs& a, hipStream_t stream) {
  if (a.B == 0) return hipSuccess;
  hipLaunchKernelGGL(expand_level_kernel, dim3((unsigned)a.B), dim3(kW),
                     expand_level_lds_bytes(a.L, a.K, a.level_set_cap), stream, a.topk_ids, a.topk_logit, a.lse,
                     a.L, a.K, a.cap, a.cost, a.fixed_budget ? 1 : 0, a.level_set_cap, a.token_ids, a.parent,
                     a.depth, a.path_prob, a.n_star, a.phi, a.theta);
  return hipGetLastError();
}

}  // namespace caddtree
