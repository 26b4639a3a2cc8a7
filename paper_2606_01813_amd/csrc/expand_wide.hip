// Stage 2 for large trees of a known size: Algorithm 1 over a threshold set
// (Sec. 4.5), one workgroup of several wavefronts per round.  It serves the
// plans whose trees keep a known number of nodes before any stop test -- fixed
// budgets (the DDTree construction, Sec. 3.4) and costs flat up to the cap --
// when that number is 512 or more.  A one-wavefront round of 4096 nodes keeps
// one SIMD of its CU busy and leaves the rest idle; here 8 or 16 wavefronts
// share each pass over a level or over the set.
//
// The steps are those of the one-wavefront kernel (expand_level.hip): build
// T(tau) level by level, raise tau in place when a level overflows the set,
// lower it when the set is too small, find the stop by a histogram of sigma,
// then lay the kept nodes out in breadth-first order.  Each pass is split into
// 64-node chunks, chunk k going to wavefront k mod NW; the steps that need the
// whole set or level (slot offsets of a level's children, histogram totals,
// new indices after a compaction, breadth-first positions) meet at workgroup
// barriers, with per-chunk counts in LDS.
//
// Every branch that decides a barrier's reach is taken by all wavefronts
// alike: each decision is computed by every wavefront from the same LDS values
// after a barrier (or from values every wavefront computes identically), and a
// shared LDS value is rewritten only after a barrier that follows its last
// read.  The steps that act on a handful of nodes (the stop inside its bin,
// small sets, the frontier test, the bisection fallback) run on wavefront 0
// with the one-wavefront routines while the others wait at the next barrier.

#include "expand_level.h"

namespace caddtree {
namespace {

constexpr int kWideMinNodes = 512;         // trees of at least this many nodes
constexpr int kMaxChunks = 2 * kW;          // chunk counts held by two lanes' worth per wavefront
constexpr int kWideBins = 1024;             // histogram bins of the in-place raise
static_assert((kMaxLeanSet + kW - 1) / kW <= kMaxChunks, "a set's chunk counts fit the prefix");
static_assert(kWideBins == 16 * kW, "16 raise bins per lane");

// LDS past the one-wavefront layout: values the wavefronts exchange
struct WideShared {
  int ctot[kMaxChunks];        // per-chunk counts
  int members[kW];             // the stop bin's nodes, generation order
  double A[CADDTREE_MAX_L + 1];
  double res_phi;
  int res_n;
  int res_all;
  int res_flag;
  int cut;                     // some node of the set has a child outside it
  int la_part;                 // compaction: kept nodes of la's chunk below la
};

__host__ __device__ constexpr size_t wide_lds_bytes(size_t LK, size_t S) {
  return a16(level_lds_bytes(LK, S, true)) + a16(sizeof(WideShared));
}
constexpr size_t kWideMaxLds = wide_lds_bytes((size_t)CADDTREE_MAX_L * CADDTREE_MAX_K, kMaxLeanSet);
static_assert(kWideMaxLds <= 160 * 1024, "the largest lean set and the exchange area fit in the LDS of one CU");

// Exclusive prefix of the chunk counts x.ctot[0 .. nchk) (nchk <= 128), read by every wavefront:
// lane i returns the offsets of chunks i (e0) and 64 + i (e1); tot is the sum.
struct ChunkPrefix {
  int e0, e1, tot;
  __device__ __forceinline__ int base(int k) const {
    return k < kW ? __builtin_amdgcn_readlane(e0, k) : __builtin_amdgcn_readlane(e1, k - kW);
  }
};
__device__ __forceinline__ ChunkPrefix chunk_prefix(const WideShared& x, int nchk, int lane) {
  const int c0 = lane < nchk ? x.ctot[lane] : 0;
  const int c1 = kW + lane < nchk ? x.ctot[kW + lane] : 0;
  const int i0 = wave_incl_scan(c0);
  const int s0 = __builtin_amdgcn_readlane(i0, kW - 1);
  const int i1 = wave_incl_scan(c1);
  return ChunkPrefix{i0 - c0, s0 + i1 - c1, s0 + __builtin_amdgcn_readlane(i1, kW - 1)};
}

// Raise tau in place at depth d, as raise_tau does for one wavefront: the lowest threshold of a
// 1024-bin histogram (refined in the straddling bin, up to kRefine passes) that keeps at most
// keep_hi nodes over depths 1 .. d + 1 and, as far as the histogram resolves, at least need;
// then the order-preserving compaction of s[0, lb) to the nodes that reach it, with parents
// renumbered.  Called by every thread of the workgroup; returns tau' (NaN: none found).
template <int NW>
__device__ double wide_raise(const Lds& s, WideShared& x, int& la, int& lb, int K, int d, double Ad, double tau,
                             double top, int keep_hi, int need, int lane, int w, int tid) {
  int* hb = reinterpret_cast<int*>(s.dl);   // free while the set is built: 1024 bins
  const int tli = d * K + (lane < K ? lane : K - 1);
  double lo_e = tau, hi_e = top;
  int above = 0;                             // nodes above the histogram's range
  double t2 = NAN;
  for (int pass = 0; pass < kRefine; ++pass) {
    if (!(hi_e > lo_e)) break;
    const double scale = (double)kWideBins / (hi_e - lo_e);
    const bool first = pass == 0;            // the first pass also takes the values at hi_e
    auto bin = [&](double v) -> int {
      const int b = (int)((v - lo_e) * scale);
      return b < kWideBins - 1 ? b : kWideBins - 1;
    };
    __syncthreads();                         // the previous pass's readers are done with the bins
    for (int i = tid; i < kWideBins; i += (NW * kW)) hb[i] = 0;
    __syncthreads();
    for (int i = tid; i < lb; i += (NW * kW)) {
      const double v = s.sl[i].x;
      if (v >= lo_e && (first || v < hi_e)) atomicAdd(&hb[bin(v)], 1);
    }
    const int nchk = (lb - la + kW - 1) / kW;
    for (int k = w; k < nchk; k += NW) {   // the next level's candidates
      const int p = la + k * kW + lane;
      const bool live = p < lb;
      const double2 pv = s.sl[live ? p : la];
      const double tlv = lane < K ? (double)s.tl[tli] : 0.0;
      for (int r = 0; r < K; ++r) {
        const double xx = (pv.y + rl_d(tlv, r)) - Ad;
        const bool q = live && xx >= tau;
        if (__ballot(q) == 0) break;
        if (q) {
          const double v = pmin(xx, pv.x);
          if (v >= lo_e && (first || v < hi_e)) atomicAdd(&hb[bin(v)], 1);
        }
      }
    }
    __syncthreads();
    // S(b) = above + values in bins >= b; lane l holds bins 16 l .. 16 l + 15
    int h[16];
    int own = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) { h[j] = hb[16 * lane + j]; own += h[j]; }
    const int incl = wave_incl_scan(own);
    const int tot = __builtin_amdgcn_readlane(incl, kW - 1);
    int S = above + tot - incl;              // values in the bins of higher lanes
    int jb = 16;                             // this lane's lowest bin with S(b) <= keep_hi (16: none)
    int Sj = 0;
#pragma unroll
    for (int j = 15; j >= 0; --j) {
      S += h[j];
      if (S <= keep_hi) { jb = j; Sj = S; }
    }
    const unsigned long long okm = __ballot(jb < 16);
    int b1 = kWideBins, S1 = above;
    if (okm) {
      const int l = __builtin_ctzll(okm);
      b1 = 16 * l + __builtin_amdgcn_readlane(jb, l);
      S1 = __builtin_amdgcn_readlane(Sj, l);
    }
    if (b1 == 0) break;                      // everything fits: nothing to raise
    if (S1 >= need) {
      t2 = lo_e + (hi_e - lo_e) * ((double)b1 / (double)kWideBins);
      break;
    }
    above = S1;                              // bin b1 - 1 holds both bounds: split it
    const double wd = (hi_e - lo_e) / (double)kWideBins;
    hi_e = lo_e + wd * (double)b1;
    lo_e = lo_e + wd * (double)(b1 - 1);
  }
  if (!(t2 > tau)) return NAN;

  // compaction: new indices from per-chunk counts of kept nodes, then the moves
  const int n0 = lb;
  const int nchk = (n0 + kW - 1) / kW;
  __syncthreads();                           // every reader of the bins and chunk counts is done
  for (int k = w; k < nchk; k += NW) {
    const int i = k * kW + lane;
    const bool keep = i < n0 && s.sl[i < n0 ? i : 0].x >= t2;
    const unsigned long long km = __ballot(keep);
    if (lane == 0) {
      x.ctot[k] = __popcll(km);
      if (la >= k * kW && la < k * kW + kW) x.la_part = __popcll(km & ((1ull << (la - k * kW)) - 1ull));
    }
  }
  __syncthreads();
  const ChunkPrefix pre = chunk_prefix(x, nchk, lane);
  for (int k = w; k < nchk; k += NW) {
    const int i = k * kW + lane;
    const bool live = i < n0;
    const bool keep = live && s.sl[live ? i : 0].x >= t2;
    const unsigned long long km = __ballot(keep);
    if (live) s.pos[i] = keep ? (int16_t)(pre.base(k) + lane_below(km)) : (int16_t)-1;
  }
  const int la2 = pre.base(la / kW) + x.la_part;
  __syncthreads();                           // every new index is written
  // a kept node moves from i to j <= i: each round reads one chunk per wavefront, then writes it;
  // a later round reads only indices above every index an earlier round wrote
  for (int q0 = 0; q0 < nchk; q0 += NW) {
    const int k = q0 + w;
    const int i = k * kW + lane;
    int j = -1, np = -1;
    double2 v = make_double2(0.0, 0.0);
    uint32_t m = 0u;
    if (k < nchk && i < n0) {
      j = s.pos[i];
      if (j >= 0) {
        v = s.sl[i];
        m = s.meta[i];
        const int par = m_parent(m);
        np = par >= 0 ? (int)s.pos[par] : -1;   // parents come first and are kept
      }
    }
    __syncthreads();
    if (j >= 0) {
      s.sl[j] = v;
      s.meta[j] = pack(np, m_rank(m), m_depth(m));
    }
  }
  __syncthreads();
  la = la2;
  lb = pre.tot;
  return t2;
}

// Where the stop falls in a set of more than 128 nodes: the histogram search of stop_hist, with
// the histograms and the classification passes split over the wavefronts and the stop inside
// its bin found by wavefront 0.  Returns false (fallback) when no bin of at most 64 nodes holds
// the stop within kLevels splits; then the caller runs the bisection on wavefront 0.
template <int NW>
__device__ bool wide_hist(const Lds& s, WideShared& x, int ns, const StopTest& tst, double lo, double hi, int lane,
                          int w, int tid, Stop& out) {
  int base_m = 0;
  double base_p = 0.0;
  for (int level = 0; level < kLevels; ++level) {
    if (!(hi > lo)) break;
    const double scale = (double)kBins / (hi - lo);
    auto bin = [&](double v) -> int {
      const int b = (int)((v - lo) * scale);
      return b < 0 ? 0 : (b < kBins - 1 ? b : kBins - 1);
    };
    auto open = [&](int e) -> bool { return level == 0 || s.pos[e] == 2; };
    __syncthreads();                         // the previous level's readers are done with the bins
    if (w == 0) {
      s.hist[lane] = 0;
      s.hmax[lane] = 0ull;
      s.hmin[lane] = ~0ull;
      s.hsum[lane] = 0ull;
    }
    __syncthreads();
    for (int e = tid; e < ns; e += (NW * kW)) {
      if (open(e)) {
        const double v = s.sl[e].x;
        double dd;
        if (level == 0) {
          dd = exp(v);
          s.dl[e] = dd;
        } else {
          dd = s.dl[e];
        }
        const int b = bin(v);
        atomicAdd(&s.hist[b], 1);
        atomicMax(&s.hmax[b], dkey(v));
        atomicMin(&s.hmin[b], dkey(v));
        atomicAdd(&s.hsum[b], (unsigned long long)(dd * kFix));
      }
    }
    __syncthreads();
    // every wavefront reads the same bins: lane b holds bin b (as in stop_hist)
    const int cnt = s.hist[lane];
    const double fs = (double)s.hsum[lane] / kFix;
    const double vmax = cnt ? dkey_inv(s.hmax[lane]) : 0.0;
    const double vmin = cnt ? dkey_inv(s.hmin[lane]) : 0.0;
    const int rl = kW - 1 - lane;
    const int cr = __shfl(cnt, rl);
    const double fr = __shfl(fs, rl);
    const int ce = wave_incl_scan(cr) - cr;
    const double fe = wave_shr1(wave_incl_scan(fr));
    const int mb = base_m + __shfl(ce, rl);
    const double pb = base_p + __shfl(fe, rl);
    const bool keep_b = cnt == 0 || kept_at(mb, pb, exp(vmax), tst);
    const unsigned long long fails = __ballot(!keep_b);
    const unsigned long long full = __ballot(cnt > 0);
    const unsigned long long above = fails ? full & ~((2ull << (63 - __builtin_clzll(fails))) - 1ull) : full;
    if (above == 0) {                        // the open range's first node is not kept (level 0 only)
      for (int e = tid; e < ns; e += (NW * kW))
        if (open(e)) s.pos[e] = 0;
      out = Stop{base_m, base_p, false};
      return true;
    }
    const int bk = __builtin_ctzll(above);
    const int t = __builtin_amdgcn_readlane(cnt, bk);
    const int mk = __builtin_amdgcn_readlane(mb, bk);
    const double pk = rl_d(pb, bk);
    const double nlo = rl_d(vmin, bk), nhi = rl_d(vmax, bk);
    for (int e = tid; e < ns; e += (NW * kW))
      if (open(e)) {
        const int b = bin(s.sl[e].x);
        s.pos[e] = b > bk ? 1 : (b < bk ? 0 : 2);
      }
    if (t > kW) {                            // split the bin by a histogram of its own range
      lo = nlo;
      hi = nhi;
      base_m = mk;
      base_p = pk;
      continue;
    }
    // the bin's nodes in generation order: per-chunk counts, then a scatter
    const int nchk = (ns + kW - 1) / kW;
    __syncthreads();                         // classification done; chunk counts free
    for (int k = w; k < nchk; k += NW) {
      const int e = k * kW + lane;
      const unsigned long long gm = __ballot(e < ns && s.pos[e < ns ? e : 0] == 2);
      if (lane == 0) x.ctot[k] = __popcll(gm);
    }
    __syncthreads();
    const ChunkPrefix pre = chunk_prefix(x, nchk, lane);
    for (int k = w; k < nchk; k += NW) {
      const int e = k * kW + lane;
      const bool g = e < ns && s.pos[e < ns ? e : 0] == 2;
      const unsigned long long gm = __ballot(g);
      if (g) x.members[pre.base(k) + lane_below(gm)] = e;
    }
    __syncthreads();
    if (w == 0) {
      const Stop st = stop_in_bin(s, x.members, t, mk, pk, ns, tst, lane);
      if (lane == 0) {
        x.res_n = st.n;
        x.res_phi = st.phi;
        x.res_all = st.all ? 1 : 0;
      }
    }
    __syncthreads();
    out = Stop{x.res_n, x.res_phi, x.res_all != 0};
    return true;
  }
  return false;
}

template <int NW>
__global__ void __launch_bounds__(NW * kW)
expand_wide_kernel(const int32_t* __restrict__ topk_ids, const float* __restrict__ topk_logit,
                   const double* __restrict__ lse, int L, int K, int cap, CostTables ct, int fixed, int setcap,
                   int32_t* __restrict__ token_ids, int32_t* __restrict__ parent_out,
                   int32_t* __restrict__ depth_out, float* __restrict__ path_prob, int32_t* __restrict__ n_star_out,
                   float* __restrict__ phi_out, float* __restrict__ theta_out) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kW - 1);
  const int w = tid / kW;
  const int LK = L * K;
  const Lds s = carve(smem, (size_t)LK, (size_t)setcap, true);
  WideShared& x = *reinterpret_cast<WideShared*>(smem + a16(level_lds_bytes((size_t)LK, (size_t)setcap, true)));
  const RoundCost rc = round_cost(ct, b);

  // setup: the top-K table to LDS; A_d = sum_{i<=d} LSE_i in depth order, by wavefront 0
  for (int i = tid; i < LK; i += (NW * kW)) {
    s.tl[i] = topk_logit[(int64_t)b * LK + i];
    s.tid[i] = topk_ids[(int64_t)b * LK + i];
  }
  if (w == 0) {
    const double lse_l = lse[(int64_t)b * L + (lane < L ? lane : L - 1)];
    double acc = 0.0;
    if (lane == 0) x.A[0] = 0.0;
    for (int d = 1; d <= L; ++d) {
      acc = acc + rl_d(lse_l, d - 1);
      if (lane == d) x.A[d] = acc;
    }
  }
  const double c0 = rc(0);
  __syncthreads();

  const double theta0 = 1.0 / c0;
  const double A1 = x.A[1];
  const double top = pmin(0.0 + (double)s.tl[0] - A1, 0.0);   // the first node to pop
  int need = cap;                            // the tree keeps cap nodes before any stop test
  bool tight = true;
  double tau = fmin(top - drop_fixed(need), top);
  const StopTest tst{cap, fixed, fixed ? 0 : 1, c0, nullptr};

  int n = 0, ns = 0;
  double phi = 0.0;
  bool all_kept = false;
  bool done = cap == 0;
  bool failed = false;
  for (int attempt = 0; attempt < kMaxAttempts && !done && !failed; ++attempt) {
    int keep_hi;
    if (tight) {
      keep_hi = need + need / 8 + 16;
    } else {
      const int half = setcap / 2, mid = (need + setcap) / 2;
      keep_hi = need <= 1 || half > mid ? half : mid;
    }
    if (keep_hi > setcap) keep_hi = setcap;
    __syncthreads();                         // the last attempt's readers of the shared values are done
    // ---- 1. T(tau), level by level; depth 1 is counted by every wavefront, written by wavefront 0
    {
      const bool live = lane < K;
      double xx = 0.0, l1 = 0.0;
      if (live) { l1 = 0.0 + (double)s.tl[lane]; xx = l1 - A1; }
      const bool in = live && xx >= tau;
      if (w == 0 && in) { s.sl[lane] = make_double2(pmin(xx, 0.0), l1); s.meta[lane] = pack(-1, lane, 1); }
      ns = __popcll(__ballot(in));
      if (tid == 0) x.cut = ns < K ? 1 : 0;
    }
    __syncthreads();
    bool dropped = false;                    // a raise dropped nodes: the tree continues below tau
    int la = 0, lb = ns;
    int raises = 0;
    for (int d = 1; d < L && la < lb;) {
      const double Ad = x.A[d + 1];
      const int tli = d * K + (lane < K ? lane : K - 1);
      const int nchk = (lb - la + kW - 1) / kW;
      // a. each parent's children that reach tau (a prefix of its ranks), and the chunk totals
      int mycut = 0;
      for (int k = w; k < nchk; k += NW) {
        const int p = la + k * kW + lane;
        const bool live = p < lb;
        const double2 pv = s.sl[live ? p : la];
        const double tlv = lane < K ? (double)s.tl[tli] : 0.0;
        int c = 0;
        for (int r = 0; r < K; ++r) {
          const double xx = (pv.y + rl_d(tlv, r)) - Ad;
          const int q = (int)(xx >= tau) & (int)live;
          if (__ballot(q != 0) == 0) break;
          c += q;
        }
        if (live) s.pos[p] = (int16_t)c;
        mycut |= (int)(live && c < K);
        const int tot = __builtin_amdgcn_readlane(wave_incl_scan(c), kW - 1);
        if (lane == 0) x.ctot[k] = tot;
      }
      if (__ballot(mycut != 0) != 0 && lane == 0) x.cut = 1;
      __syncthreads();
      const ChunkPrefix pre = chunk_prefix(x, nchk, lane);
      const int nb = lb;
      if (nb + pre.tot > setcap) {           // the level would overflow the set: raise tau in place
        if (++raises > kMaxRaises) { failed = true; break; }
        const double t2 = wide_raise<NW>(s, x, la, lb, K, d, Ad, tau, top, keep_hi, need, lane, w, tid);
        if (!(t2 > tau)) { failed = true; break; }
        tau = t2;
        dropped = true;
        continue;                            // build depth d + 1 again
      }
      // b. the children, at their chunk's offset plus the prefix within the chunk
      for (int k = w; k < nchk; k += NW) {
        const int p = la + k * kW + lane;
        const bool live = p < lb;
        const double2 pv = s.sl[live ? p : la];
        const double tlv = lane < K ? (double)s.tl[tli] : 0.0;
        const int c = live ? (int)s.pos[p] : 0;
        const int at = nb + pre.base(k) + wave_incl_scan(c) - c;
        for (int r = 0; __ballot(r < c) != 0; ++r) {
          const double l = pv.y + rl_d(tlv, r);
          const double2 v = make_double2(pmin(l - Ad, pv.x), l);
          const uint32_t m = pack(p, r, d + 1);
          if (r < c) {
            s.sl[at + r] = v;
            s.meta[at + r] = m;
          }
        }
      }
      __syncthreads();
      la = lb;
      lb = nb + pre.tot;
      ++d;
    }
    if (failed) break;
    __syncthreads();
    const bool cut = x.cut != 0 || dropped;
    ns = lb;
    if (cut && ns < need && ns < cap) {     // too few nodes to hold the stop: lower tau without selecting
      tau -= fmax(log(4.0 * (double)need / (double)(ns > 0 ? ns : 1)), 1.0);
      continue;
    }

    // ---- 2. where the stop falls
    Stop st;
    const unsigned seed = 0x9E3779B9u ^ (unsigned)b ^ ((unsigned)attempt << 16);
    bool have = false;
    if (ns > 2 * kW) have = wide_hist<NW>(s, x, ns, tst, tau, top, lane, w, tid, st);
    if (!have) {                             // small sets, and the bisection fallback: wavefront 0
      __syncthreads();
      if (w == 0) {
        Stop r;
        if (ns <= kW) r = stop_small(s, ns, tst, lane);
        else if (ns <= 2 * kW) r = stop_rank<2>(s, ns, tst, lane);
        else r = stop_lds(s, ns, tst, lane, seed);
        if (lane == 0) {
          x.res_n = r.n;
          x.res_phi = r.phi;
          x.res_all = r.all ? 1 : 0;
        }
      }
      __syncthreads();
      st = Stop{x.res_n, x.res_phi, x.res_all != 0};
    }

    if (!st.all) {                          // the stop (or the cap) falls inside T(tau)
      n = st.n;
      phi = st.phi;
      all_kept = false;
      done = true;
      continue;
    }
    bool stop_after = !cut || ns >= cap;
    if (!stop_after && !fixed) {            // a flat cost: test the next pop, the frontier's best node
      __syncthreads();
      if (w == 0) {
        const double Areg = lane <= L ? x.A[lane <= L ? lane : 0] : 0.0;   // lane d: A_d
        const double fm = rl_d(frontier_max(s, ns, L, K, Areg, lane), 0);
        if (lane == 0) x.res_flag = kept_at(ns, st.phi, exp(fm), tst) ? 0 : 1;
      }
      __syncthreads();
      stop_after = x.res_flag != 0;
    }
    if (stop_after) {                       // the whole tree (or the cap) is here, all of it kept
      n = ns;
      phi = st.phi;
      all_kept = true;
      done = true;
    } else {                                // every node kept: the stop lies below tau
      need = ns + 1;
      tight = false;
      if (need > setcap) { failed = true; break; }
      tau = tau - 1.5;
    }
  }
  if (!done) {                              // left to the serial kernel
    if (tid == 0) n_star_out[b] = -1;
    return;
  }
  if (tid == 0) {
    n_star_out[b] = n;
    if (phi_out) phi_out[b] = (float)phi;
    if (theta_out) theta_out[b] = (float)(n == 0 ? theta0 : (1.0 + phi) / rc(n));
  }
  if (n == 0) return;

  // ---- breadth-first positions: kept nodes before each one in generation order
  const int nchk = (ns + kW - 1) / kW;
  __syncthreads();                          // the selection's flags are written
  for (int k = w; k < nchk; k += NW) {
    const int i = k * kW + lane;
    const bool kept = i < ns && (all_kept || s.pos[i < ns ? i : 0] != 0);
    const unsigned long long km = __ballot(kept);
    if (lane == 0) x.ctot[k] = __popcll(km);
  }
  __syncthreads();
  const ChunkPrefix pre = chunk_prefix(x, nchk, lane);
  for (int k = w; k < nchk; k += NW) {
    const int i = k * kW + lane;
    const bool live = i < ns;
    const bool kept = live && (all_kept || s.pos[live ? i : 0] != 0);
    const unsigned long long km = __ballot(kept);
    if (live) s.pos[i] = kept ? (int16_t)(pre.base(k) + lane_below(km)) : (int16_t)-1;
  }
  __syncthreads();
  const int64_t ob = (int64_t)b * cap;
  for (int i = tid; i < ns; i += (NW * kW)) {
    const int o = s.pos[i];
    if (o >= 0) {
      const uint32_t m = s.meta[i];
      const int p = m_parent(m), dd = m_depth(m), r = m_rank(m);
      token_ids[ob + o] = s.tid[(dd - 1) * K + r];
      parent_out[ob + o] = p < 0 ? -1 : (int)s.pos[p];
      depth_out[ob + o] = dd;
      if (path_prob) path_prob[ob + o] = (float)exp(s.sl[i].x);
    }
  }
}

}  // namespace

bool expand_wide_applies(int32_t cap, bool lean) { return lean && cap >= kWideMinNodes; }

size_t expand_wide_lds_bytes(int32_t L, int32_t K, int32_t set_cap) {
  return wide_lds_bytes((size_t)L * K, (size_t)set_cap);
}

hipError_t expand_wide_prepare() {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&expand_wide_kernel<8>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)kWideMaxLds);
  if (e == hipSuccess)
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&expand_wide_kernel<16>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)kWideMaxLds);
  return e;
}

// Sixteen wavefronts per round (at most 128 VGPRs each, so one round per CU) when every round has
// a CU of its own or the set's LDS allows only one round per CU anyway; else eight, so that two
// rounds share a CU.
hipError_t launch_expand_wide(const ExpandArgs& a, hipStream_t stream) {
  if (a.B == 0) return hipSuccess;
  const size_t lds = expand_wide_lds_bytes(a.L, a.K, a.level_set_cap);
  const bool sixteen = a.B <= (int64_t)a.num_cu || 2 * lds > (size_t)160 * 1024;
  if (sixteen)
    hipLaunchKernelGGL(expand_wide_kernel<16>, dim3((unsigned)a.B), dim3(16 * kW), lds, stream, a.topk_ids,
                       a.topk_logit, a.lse, a.L, a.K, a.cap, a.cost, a.fixed_budget ? 1 : 0, a.level_set_cap,
                       a.token_ids, a.parent, a.depth, a.path_prob, a.n_star, a.phi, a.theta);
  else
    hipLaunchKernelGGL(expand_wide_kernel<8>, dim3((unsigned)a.B), dim3(8 * kW), lds, stream, a.topk_ids,
                       a.topk_logit, a.lse, a.L, a.K, a.cap, a.cost, a.fixed_budget ? 1 : 0, a.level_set_cap,
                       a.token_ids, a.parent, a.depth, a.path_prob, a.n_star, a.phi, a.theta);
  return hipGetLastError();
}

}  // namespace caddtree
