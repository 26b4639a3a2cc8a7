// Stage 2, batched form: Algorithm 1 (Sec. 4.5) evaluated over a threshold set.
//
// Algorithm 1 pops nodes in the order sigma desc, depth asc, Lambda desc, rank
// tuple asc (see expand.hip for the keys) and keeps them while theta rises.
// Every node outside T(tau) = {nodes with sigma >= tau} comes after every node
// inside it, so the first |T(tau)| pops are T(tau) in that order.  One
// workgroup (one wavefront) per round:
//
//  1. build T(tau) level by level from the root.  The children of a node that
//     reach the threshold are a prefix of its ranks (sigma falls with the rank).
//     A level of few parents (at most 256 (parent, rank) pairs) is tested one
//     pair a lane, kW / K parents a pass and four passes at once; lane order is
//     (parent, rank) order, so a qualifying child's slot is the count of
//     qualifying lanes below it.  A wider level takes one parent a lane, each
//     lane counting its node's children up to the first rank that no lane
//     takes, and a prefix sum gives their slots.  Either way the set comes out
//     in breadth-first order (depth, then rank tuple), which is also the
//     tie-break of the pop order within a depth.  When a level would not fit
//     in the set, tau is raised in place: a histogram of sigma over the levels
//     built and the candidates of the next one picks the new threshold, the
//     set is compacted (order kept, parents renumbered), and the level is built
//     again.  A parent's sigma is at least its children's, so what remains is
//     T(tau') so far;
//  2. find where the greedy stop falls along the pop order of T(tau).  Nodes
//     that tie on sigma have the same path probability delta = exp(sigma), so
//     Phi before every position, and with it the stop test at every position,
//     depends only on the sigma values in descending order.  The rest of the
//     order decides only which members are kept of a tie group that the stop
//     cuts:
//     * up to 128 nodes: a bitonic network across the wave sorts the sigma
//       values (one or two a lane), a prefix sum of their path probabilities
//       gives Phi before every position m, and m is kept iff
//       (1 + Phi_m + delta_m) / C(m + 1) > (1 + Phi_m) / C(m) and m < cap;
//     * larger sets: under a convex cost theta rises and then falls along the
//       pop order (Thm. 1), so the stop test fails from n* on.  A 64-bin
//       histogram of sigma gives the position of each bin's first node and
//       Phi before it, the test runs at every bin's first node at once, and
//       the bin that holds the stop is ranked node by node (or split again by
//       a histogram of its own range when it holds more than 64 nodes);
//     with a fixed budget m is kept iff m < cap;
//  3. if every node of T(tau) is kept and the tree continues below tau, test
//     the next pop, the frontier node of largest sigma: if it is not kept the
//     stop falls right after T(tau); else lower tau and start again.  Lower
//     tau likewise when T(tau) holds fewer nodes than every tree keeps (a flat
//     start of the cost, or a fixed budget).
//
// The initial tau comes from the cost model: a node kept near position n has
// delta > (1 + Phi) c_{n+1} / C(n) (Lemma 1); with c_{m0+1} the first positive
// marginal cost the stop lies past m0, around delta = (1 + Phi) c / C with Phi
// of order one.  Flat starts and fixed budgets, which keep a known number of
// nodes, start well below and let the in-place raise bring the set to size.
// A round that does not settle within kMaxAttempts (or kMaxRaises raises in
// one attempt), or whose tree needs more nodes than the set holds (512, or up
// to 4096 for fixed budgets and long flat cost starts, sized by the host), goes
// to the serial form (expand_serial.h), which gives the same tree: run in place
// by the same workgroup when the launch reserved LDS for the serial layout,
// else flagged (n_star = -1) for the serial kernel.
//
// The kept nodes are a prefix of the pop order and a prefix-closed set, so
// their breadth-first positions are a running count over generation order.
// Phi here is a prefix sum over the wave rather than a left-to-right sum in
// pop order: it matches the sequential sum to rounding, and the tree does not
// depend on it except at stop margins of that size.
//
// The workgroup is a single wavefront, whose LDS operations complete in issue
// order, so what one step writes to LDS the next step reads without a barrier.

#include "expand_level.h"
#include "expand_serial.h"

namespace caddtree {
namespace {

// A round the batched form cannot settle, run by the serial form in the same workgroup (the
// launch reserved LDS for the serial layout).  Out of line: it is rare, and inlined it would
// crowd the batched kernel's registers.
__device__ __attribute__((noinline)) void serial_in_place(serial::Args a, int b) { serial::expand_round(a, b); }

__global__ void __launch_bounds__(kW)
expand_level_kernel(const int32_t* __restrict__ topk_ids, const float* __restrict__ topk_logit,
                    const double* __restrict__ lse, int L, int K, int cap, CostTables ct, int fixed,
                    int flat, int setcap, int32_t* __restrict__ token_ids,
                    int32_t* __restrict__ parent_out, int32_t* __restrict__ depth_out,
                    float* __restrict__ path_prob, int32_t* __restrict__ n_star_out,
                    float* __restrict__ phi_out, float* __restrict__ theta_out, int in_place, EmitOut em,
                    int first_rise, double tau_model) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int LK = L * K;
  const bool lean = fixed || flat;          // no cost table
  const Lds s = carve(smem, (size_t)LK, (size_t)setcap, lean);
  const RoundCost rc = round_cost_wave(ct, b, lane);
  // the level build's lane split: group grp of K lanes takes one parent, lane rk of it one rank
  constexpr int kPasses = 4;               // passes a step
  constexpr int kPairsFew = 256;           // levels of at most this many (parent, rank) pairs go by pairs
  constexpr int kSoftMul = 2;              // soft set limit of a round of known size, in keep_hi
  const int ppass = kW / K;                 // parents a pass (K <= 16: at least 4)
  const int grp = lane / K;
  const int rk = lane - grp * K;
  const bool in_pass = grp < ppass;

  // setup: the round's global loads are issued together, then stored to LDS.  Indices are
  // clamped rather than guarded (a clamped lane loads and stores the same value as the last
  // valid one), so neither loads nor stores sit behind branches.
  const double c0 = rc(0);
  const double lse_l = lse[(int64_t)b * L + (lane < L ? lane : L - 1)];
  CostCache cc{rc, s.cw, cap, lean ? 0 : (cap < setcap ? cap : setcap) + 2, 0};   // C(0 .. ncw - 1)
  {
    constexpr int kT = CADDTREE_MAX_L * CADDTREE_MAX_K / kW;        // top-K entries per lane, at most
    float lv[kT];
    int32_t iv[kT];
#pragma unroll
    for (int u = 0; u < kT; ++u) {          // clamped like the cost table
      const int i = u * kW + lane < LK ? u * kW + lane : LK - 1;
      lv[u] = topk_logit[(int64_t)b * LK + i];
      iv[u] = topk_ids[(int64_t)b * LK + i];
    }
    cc.ensure(kW + 2, lane);
#pragma unroll
    for (int u = 0; u < kT; ++u) {
      const int i = u * kW + lane < LK ? u * kW + lane : LK - 1;
      s.tl[i] = lv[u];
      s.tid[i] = iv[u];
    }
  }
  // lane d holds A_d = sum_{i<=d} LSE_i, summed in depth order (d = 0 .. L)
  double Areg = 0.0;
  {
    double acc = 0.0;
    for (int d = 1; d <= L; ++d) {
      acc = acc + rl_d(lse_l, d - 1);
      if (lane == d) Areg = acc;
    }
  }
  __syncthreads();

  const double theta0 = 1.0 / c0;
  const double A1 = rl_d(Areg, 1);
  const double top = pmin(0.0 + (double)s.tl[0] - A1, 0.0);   // the first node to pop
  double tau = top - 3.0;
  int need = 1;                              // the tree holds at least this many nodes
  bool tight = false;                        // need is what the tree keeps before any stop test
  if (lean) {                                // fixed budget, or a cost flat up to the cap
    need = cap;
    tight = true;
    tau = top - drop_fixed(need);
  } else if (cap >= 1) {
    // the first positive marginal cost c_{m0 + 1} (the stop lies past m0), and the cost-model
    // threshold there: from the host for a plan with one cost table, else searched here
    int m0 = first_rise;
    double tau_cm = tau_model;
    if (m0 < -1) {
      m0 = -1;
      const int mlim = cap < setcap ? cap : setcap;
      for (int i0 = 0; i0 < mlim && m0 < 0; i0 += kW) {
        const int i = i0 + lane;
        cc.ensure(i0 + kW + 1, lane);
        const unsigned long long m = __ballot(i < mlim && s.cw[i + 1] > s.cw[i]);
        if (m) m0 = i0 + __builtin_ctzll(m);
      }
      if (m0 >= 0 && m0 < setcap / 2) {
        const int m = m0 + 32 < cap ? m0 + 32 : cap;
        cc.ensure(m + 1, lane);
        tau_cm = log(2.0 * (s.cw[m0 + 1] - s.cw[m0]) / s.cw[m]) - 0.5;
      }
    }
    if (m0 < 0 && cap <= setcap / 2) {
      need = cap;                           // flat up to the cap: every node is kept until the cap
      tight = true;
      tau = top - drop_fixed(need);
    } else if (m0 < 0 || m0 >= setcap / 2) {
      // flat for longer than the set holds: the serial form's case
      if (in_place)
        serial_in_place(serial::Args{topk_ids, topk_logit, lse, L, K, cap, ct, fixed, token_ids, parent_out,
                                     depth_out, path_prob, n_star_out, phi_out, theta_out, em}, b);
      else if (lane == 0)
        n_star_out[b] = -1;
      return;
    } else {
      need = m0 + 1;
      tau = tau_cm;
      if (need > 1) {
        tau -= kDropFlat;
        tight = true;
      }
    }
  }
  tau = fmin(tau, top);
  const StopTest tst{cap, fixed, flat, c0, s.cw};

  int n = 0, ns = 0;
  double phi = 0.0;
  bool all_kept = false;                    // every node of T(tau) is kept (no flags written)
  bool done = cap == 0;
  bool failed = false;
  for (int attempt = 0; attempt < kMaxAttempts && !done && !failed; ++attempt) {
    // what a raise keeps at most: a little above need when need is what the tree keeps
    // before any stop test, else room for a stop past need
    int keep_hi;
    if (tight) {
      keep_hi = need + need / 8 + 16;
    } else {
      const int half = setcap / 2, mid = (need + setcap) / 2;
      keep_hi = need <= 1 || half > mid ? half : mid;
    }
    if (keep_hi > setcap) keep_hi = setcap;
    // a flat start (a round that keeps a known number of nodes before any stop test) raises tau
    // as soon as the set passes soft, well above keep_hi, rather than when it would overflow:
    // building and selecting in a set many times the tree costs more than the raise.  A raise from
    // there that finds no threshold drops the limit.
    int soft = setcap;
    if (tight && !lean && kSoftMul * keep_hi + kW < setcap) soft = kSoftMul * keep_hi + kW;
    // ---- 1. T(tau), level by level
    bool cut = false;
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
    int raises = 0;
    for (int d = 1; d < L && la < lb;) {
      const double Ad = rl_d(Areg, d + 1);
      const int tli = d * K + (lane < K ? lane : K - 1);
      const double tr = (double)s.tl[d * K + rk];     // rank rk at depth d + 1
      int nb = lb;
      bool over = false;
      if ((lb - la) * K <= kPairsFew) {
        // ppass parents a pass, one lane per (parent, rank): a child's place in the level is the count
        // of qualifying lanes below it, since lane order is (parent, rank) order.  Four passes go
        // together, their parents read at once.  Lanes past the level's end (and past ppass K)
        // compute on a valid node and take no child.
        for (int q0 = la; q0 < lb; q0 += kPasses * ppass) {
          double2 pv[kPasses];
          int p[kPasses];
          bool live[kPasses];
#pragma unroll
          for (int u = 0; u < kPasses; ++u) {
            p[u] = q0 + u * ppass + grp;
            live[u] = in_pass && p[u] < lb;
            pv[u] = s.sl[live[u] ? p[u] : la];
          }
          bool q[kPasses];
          double x[kPasses], l[kPasses];
          unsigned long long m[kPasses];
          int tot = 0;
#pragma unroll
          for (int u = 0; u < kPasses; ++u) {
            l[u] = pv[u].y + tr;
            x[u] = l[u] - Ad;
            q[u] = live[u] && x[u] >= tau;
            if (live[u] && !q[u]) cut = true;  // a child of a node of the set is left out
            m[u] = __ballot(q[u]);
            tot += __popcll(m[u]);
          }
          if (nb + tot > soft) { over = true; break; }
#pragma unroll
          for (int u = 0; u < kPasses; ++u) {
            if (q[u]) {
              const int at = nb + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m[u] >> 32),
                                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)m[u], 0u));
              s.sl[at] = make_double2(pmin(x[u], pv[u].x), l[u]);
              s.meta[at] = pack(p[u], rk, d + 1);
            }
            nb += __popcll(m[u]);
          }
        }
      } else {
        // one lane per parent: the ranks that qualify form a prefix, counted rank by rank until no
        // lane takes one (dead lanes compute too, on a valid node, and are masked out of the count)
        for (int p0 = la; p0 < lb; p0 += kW) {
          const int p = p0 + lane;
          const bool live = p < lb;
          const double2 pv = s.sl[live ? p : la];
          const double tlv = lane < K ? (double)s.tl[tli] : 0.0;   // lane r: rank r at depth d + 1
          int c = 0, rmax = 0;
          for (; rmax < K; ++rmax) {
            const double x = (pv.y + rl_d(tlv, rmax)) - Ad;
            const int q = (int)(x >= tau) & (int)live;
            if (__ballot(q != 0) == 0) break;
            c += q;
          }
          const int incl = wave_incl_scan(c);
          const int tot = __builtin_amdgcn_readlane(incl, kW - 1);
          const int off = incl - c;
          if (live && c < K) cut = true;
          if (nb + tot > soft) { over = true; break; }
          for (int r = 0; r < rmax; ++r) {
            const double l = pv.y + rl_d(tlv, r);
            const double2 v = make_double2(pmin(l - Ad, pv.x), l);
            const uint32_t m = pack(p, r, d + 1);
            if (r < c) {
              s.sl[nb + off + r] = v;
              s.meta[nb + off + r] = m;
            }
          }
          nb += tot;
        }
      }
      if (over) {
        const double tlv = lane < K ? (double)s.tl[tli] : 0.0;
        const double t2 = ++raises > kMaxRaises ? NAN : raise_tau(s, la, lb, K, Ad, tlv, tau, top, keep_hi, need, lane);
        if (!(t2 > tau)) {
          if (soft < setcap) {                 // nothing changed: build the level again up to setcap
            soft = setcap;
            raises = 0;
            continue;
          }
          failed = true;
          break;
        }
        tau = t2;
        cut = true;                          // nodes were dropped: the tree continues below tau
        continue;                            // build depth d + 1 again
      }
      la = lb;
      lb = nb;
      ++d;
    }
    if (failed) break;
    cut = __ballot(cut) != 0;
    ns = lb;
    if (cut && ns < need && ns < cap) {     // too few nodes to hold the stop: lower tau without selecting
      tau -= fmax(log(4.0 * (double)need / (double)(ns > 0 ? ns : 1)), 1.0);
      continue;
    }

    // ---- 2. where the stop falls
    cc.ensure((ns < cap ? ns : cap) + 2, lane);   // C(m), C(m + 1) at every position, and C(ns + 1)
    Stop st;
    const unsigned seed = 0x9E3779B9u ^ (unsigned)b ^ ((unsigned)attempt << 16);
    if (ns <= kW) st = stop_small(s, ns, tst, lane);
    else if (ns <= 2 * kW) st = stop_rank<2>(s, ns, tst, lane);
    else st = stop_hist(s, ns, tst, tau, top, lane, seed);

    if (!st.all) {                          // the stop (or the cap) falls inside T(tau)
      n = st.n;
      phi = st.phi;
      all_kept = false;
      done = true;
    } else if (!cut || ns >= cap ||
               !kept_at(ns, st.phi, exp(rl_d(frontier_max(s, ns, L, K, Areg, lane), 0)), tst)) {
      // the whole tree (or the cap) is here and all of it is kept, or the next pop (the frontier
      // node of largest sigma) is not kept: the stop falls right after the set
      n = ns;
      phi = st.phi;
      all_kept = true;
      done = true;
    } else {                                // every node kept: the stop lies below tau
      need = ns + 1;                        // and the tree holds more nodes than this set
      tight = false;
      if (need > setcap) { failed = true; break; }
      // the next pop is kept only while delta > (1 + Phi) c_{n+1} / C(n) (Lemma 1), a bound that
      // does not fall as n grows under a convex cost: aim a little below it
      double target = tau - 1.5;
      if (!lean) {
        const double c1 = s.cw[ns + 1] - s.cw[ns];
        if (c1 > 0.0) target = fmin(tau - 0.25, log((1.0 + st.phi) * c1 / s.cw[ns]) - 1.5);
      }
      tau = target;
    }
  }
  if (!done) {                              // left to the serial form
    if (in_place)
      serial_in_place(serial::Args{topk_ids, topk_logit, lse, L, K, cap, ct, fixed, token_ids, parent_out,
                                   depth_out, path_prob, n_star_out, phi_out, theta_out, em}, b);
    else if (lane == 0)
      n_star_out[b] = -1;
    return;
  }
  // theta = (1 + Phi) / C(n): C(n) from the LDS table when the plan has one (every position up to
  // min(ns, cap) + 1 is there), else from memory, a load whose wait falls at the end of the epilogue
  const double cn = n == 0 ? c0 : (lean ? rc(n) : s.cw[n]);
  if (lane == 0) {
    n_star_out[b] = n;
    if (phi_out) phi_out[b] = (float)phi;
  }
  if (n == 0) {
    if (lane == 0 && theta_out) theta_out[b] = (float)theta0;
    return;
  }

  // ---- breadth-first positions: kept nodes before this one in generation order
  int base = 0;
  for (int i0 = 0; i0 < ns; i0 += kW) {
    const int i = i0 + lane;
    const bool kept = i < ns && (all_kept || s.pos[i] != 0);
    const unsigned long long m = __ballot(kept);
    if (i < ns) s.pos[i] = kept ? (int16_t)(base + lane_below(m)) : (int16_t)-1;
    base += __popcll(m);
  }
  const int64_t ob = (int64_t)b * cap;
  int16_t* par = reinterpret_cast<int16_t*>(s.dl);       // output parents, for the mask (dl is done)
  for (int i = lane; i < ns; i += kW) {
    const int o = s.pos[i];
    if (o >= 0) {
      const uint32_t m = s.meta[i];
      const int p = m_parent(m), d = m_depth(m), r = m_rank(m);
      const int po = p < 0 ? -1 : (int)s.pos[p];
      token_ids[ob + o] = s.tid[(d - 1) * K + r];
      parent_out[ob + o] = po;
      depth_out[ob + o] = d;
      if (path_prob) path_prob[ob + o] = (float)exp(s.sl[i].x);
      if (em.pos_ids) em.pos_ids[ob + o] = em.pos_offset + d;
      par[o] = (int16_t)po;
    }
  }
  __syncthreads();
  // the mask, in the set's (sigma, Lambda) region (free now; emit_tile_bytes(n) <= 16 setcap bytes)
  emit_mask_wave(par, n, cap, em.mask_kind, round_mask(em, b, cap), reinterpret_cast<uint32_t*>(s.sl), lane);
  if (lane == 0 && theta_out) theta_out[b] = (float)((1.0 + phi) / cn);
}

}  // namespace

size_t expand_level_lds_bytes(int32_t L, int32_t K, int32_t set_cap, bool lean) {
  return level_lds_bytes((size_t)L * K, (size_t)set_cap, lean);
}

int expand_level_set_cap(int32_t need, bool lean) {
  if (lean && need > kMaxSet / 2) return kMaxLeanSet;
  int S = kSmall;
  while (S < kMaxSet && S < 2 * need) S *= 2;
  return S;
}

int expand_level_max_need(bool lean) { return lean ? kMaxLeanSet * 4 / 5 : kMaxSet / 2; }

size_t expand_level_lds_limit() { return kMaxLds; }

hipError_t expand_level_prepare() {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&expand_level_kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
}

hipError_t launch_expand_level(const ExpandArgs& a, size_t in_place_lds, hipStream_t stream) {
  if (a.B == 0) return hipSuccess;
  const bool lean = a.fixed_budget || a.flat_cost;
  size_t lds = expand_level_lds_bytes(a.L, a.K, a.level_set_cap, lean);
  if (in_place_lds > lds) lds = in_place_lds;
  hipLaunchKernelGGL(expand_level_kernel, dim3((unsigned)a.B), dim3(kW), lds, stream, a.topk_ids, a.topk_logit,
                     a.lse, a.L, a.K, a.cap, a.cost, a.fixed_budget ? 1 : 0, (!a.fixed_budget && a.flat_cost) ? 1 : 0,
                     a.level_set_cap, a.token_ids, a.parent, a.depth, a.path_prob, a.n_star, a.phi, a.theta,
                     in_place_lds > 0 ? 1 : 0, a.em, a.first_rise, a.tau_model);
  return hipGetLastError();
}

}  // namespace caddtree
