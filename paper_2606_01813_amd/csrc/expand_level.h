// The threshold-set machinery of the batched expansion (Algorithm 1 over T(tau) = {sigma >= tau},
// Sec. 4.5): constants, the LDS layout of a round, the stop test, the selection of the stop
// position in a set (by rank, by histogram, by bisection), the in-place raise of tau and the
// frontier maximum.  Single-wavefront routines: every call is made by all 64 lanes of one
// wavefront.  Shared by the one-wavefront kernel (expand_level.hip) and the routines of the
// several-wavefront kernel for large fixed-size trees (expand_wide.hip).
#pragma once

#include <cmath>

#include "expand_common.h"
#include "internal.h"

namespace caddtree {
namespace {

using namespace xp;

constexpr int kW = 64;
constexpr int kSmall = 512;           // sets up to this size are selected in registers
constexpr int kMaxSet = 4096;         // the largest set the LDS layout holds
constexpr int kMaxLeanSet = 5120;     // the same without the cost table (fixed budgets, flat costs)
constexpr int kMaxAttempts = 12;
constexpr int kBins = kW;             // histogram bins of the in-place raise (one per lane)
constexpr int kRefine = 4;            // histogram passes per raise
constexpr int kMaxRaises = 32;        // raises per attempt
constexpr double kDropFlat = 2.0;     // a flat start begins this far (nats) below the cost-model threshold

// Fixed budgets and costs flat up to the cap keep `need` nodes: the first threshold lies this far
// (nats) below the top node, further for larger trees.
__device__ __forceinline__ double drop_fixed(int need) {
  const double d = 6.0 + 2.0 * log2((double)(need > 128 ? need : 128) / 128.0);
  return d < 12.0 ? d : 12.0;
}

__device__ __forceinline__ int lane_below(unsigned long long m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

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

struct Lds {
  float* tl;        // [L * K] raw logits
  int32_t* tid;     // [L * K] token ids
  double* cw;       // [S + 2] C(n) = C_d + C_v(min(n, cap)), for costs other than fixed budgets
  double2* sl;      // [S] T(tau) in generation order: (sigma, Lambda)
  uint32_t* meta;   // [S]   packed word (parent, rank, depth)
  double* dl;       // [S]   path probability (sets above kSmall), or in sigma order (small sets)
  int16_t* pos;     // [S]   new index (raise), kept flag, then breadth-first position
  unsigned long long* hsum;   // [kBins] fixed-point delta sums (selection)
  unsigned long long* hmax;   // [kBins] largest sigma, as an ordered key (selection)
  unsigned long long* hmin;   // [kBins] smallest sigma, as an ordered key (selection)
  int* hist;                  // [kBins] node counts (raise, selection)
};

// LDS of a round for a set of S nodes
// (lean: no cost table, for fixed budgets and costs flat up to the cap)
__host__ __device__ constexpr size_t cost_entries(size_t S, bool lean) { return lean ? 0 : S + 2; }
__host__ __device__ constexpr size_t level_lds_bytes(size_t LK, size_t S, bool lean) {
  return a16(a16(a16(a16(a16(a16(a16(a16(4 * LK) + 4 * LK) + 8 * cost_entries(S, lean)) + 16 * S) + 4 * S) + 8 * S) +
                 2 * S) +
             32 * (size_t)kBins);
}
constexpr size_t kMaxLds = level_lds_bytes((size_t)CADDTREE_MAX_L * CADDTREE_MAX_K, kMaxSet, false) >
                                   level_lds_bytes((size_t)CADDTREE_MAX_L * CADDTREE_MAX_K, kMaxLeanSet, true)
                               ? level_lds_bytes((size_t)CADDTREE_MAX_L * CADDTREE_MAX_K, kMaxSet, false)
                               : level_lds_bytes((size_t)CADDTREE_MAX_L * CADDTREE_MAX_K, kMaxLeanSet, true);
static_assert(kMaxLds <= 160 * 1024, "the largest set must fit in the LDS of one CU");

__device__ Lds carve(unsigned char* smem, size_t LK, size_t S, bool lean) {
  Lds s;
  size_t off = 0;
  s.tl = reinterpret_cast<float*>(smem + off);      off = a16(off + 4 * LK);
  s.tid = reinterpret_cast<int32_t*>(smem + off);   off = a16(off + 4 * LK);
  s.cw = reinterpret_cast<double*>(smem + off);     off = a16(off + 8 * cost_entries(S, lean));
  s.sl = reinterpret_cast<double2*>(smem + off);    off = a16(off + 16 * S);
  s.meta = reinterpret_cast<uint32_t*>(smem + off); off = a16(off + 4 * S);
  s.dl = reinterpret_cast<double*>(smem + off);     off = a16(off + 8 * S);
  s.pos = reinterpret_cast<int16_t*>(smem + off);   off = a16(off + 2 * S);
  s.hsum = reinterpret_cast<unsigned long long*>(smem + off);
  s.hmax = s.hsum + kBins;
  s.hmin = s.hmax + kBins;
  s.hist = reinterpret_cast<int*>(s.hmin + kBins);
  return s;
}

// The cost table C(0 .. ncw - 1) in LDS is filled on demand, 64 entries at a time, so a round
// reads from memory only the part of the table that its positions reach (each distinct line
// read adds to the round's latency).
struct CostCache {
  const RoundCost rc;
  double* cw;
  int cap;
  int ncw;       // entries the table holds at most
  int filled;    // entries written so far (wave-uniform)

  // make C(0 .. k - 1) available
  __device__ __forceinline__ void ensure(int k, int lane) {
    if (k > ncw) k = ncw;
    if (k <= filled) return;
    constexpr int kC = 8;                    // entries per lane and batch
    const int hi = ((k + kW - 1) / kW) * kW < ncw ? ((k + kW - 1) / kW) * kW : ncw;
    for (int i0 = filled; i0 < hi; i0 += kC * kW) {
      double lv[kC], hv[kC];
      int ci[kC];
#pragma unroll
      for (int u = 0; u < kC; ++u) {        // clamped, not guarded, so the loads go out together;
        ci[u] = i0 + u * kW + lane < hi ? i0 + u * kW + lane : hi - 1;   // past the end, every
        const int n = ci[u] < cap ? ci[u] : cap;                           // lane reads one entry
        lv[u] = rc.lo[n];
        hv[u] = rc.hi[n];
      }
      // every load is issued before the first use: a use waits for all loads issued before it
      // (and for the caller's, e.g. the top-K table's), so an interleaved use would cost a round trip
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < kC; ++u) cw[ci[u]] = rc.mix(lv[u], hv[u]);
    }
    filled = hi;
  }
};

// The stop test of a round: a fixed budget keeps every position below the cap; a cost flat up
// to the cap has C(m) = C(0) at every position (no table); else C(m) comes from the LDS table.
struct StopTest {
  int cap;
  int fixed;
  int flat;
  double c0;         // C(0)
  const double* cw;  // C(0 ..), costs that are neither fixed budgets nor flat
};

// position m of the pop order is kept, with Phi before it and delta at it
__device__ __forceinline__ bool kept_at(int m, double phi, double delta, const StopTest& t) {
  if (m >= t.cap) return false;
  if (t.fixed) return true;
  if (t.flat) return (1.0 + phi + delta) / t.c0 > (1.0 + phi) / t.c0;
  return (1.0 + phi + delta) / t.cw[m + 1] > (1.0 + phi) / t.cw[m];
}

struct Stop {
  int n;        // first position not kept, or ns when every position is kept
  double phi;   // Phi before position n
  bool all;     // every position is kept (no flags written)
};

// Kept flags when the stop cuts a tie group: the group (sigma == v) fills pop positions
// [g0, g0 + t), and its members at positions below `stop` are kept.  A member's position
// is g0 plus the number of members that pop before it; the members are walked one by
// one (as many steps as the group has members), each against every lane's nodes.
template <int P>
__device__ void cut_group_flags(const Lds& s, int ns, const double (&sg)[P], double v, int g0, int stop, int lane) {
  int rt[P];
  double lam[P];
  uint32_t mm[P];
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const int e = j * kW + lane;
    rt[j] = 0;
    lam[j] = e < ns ? s.sl[e].y : 0.0;
    mm[j] = e < ns ? s.meta[e] : 0u;
  }
#pragma unroll
  for (int jo = 0; jo < P; ++jo) {
    unsigned long long gm = __ballot(jo * kW + lane < ns && sg[jo] == v);
    while (gm) {
      const int ol = __builtin_ctzll(gm);
      gm &= gm - 1;
      const int o = jo * kW + ol;
      const double lo = rl_d(lam[jo], ol);
      const uint32_t mo = rl_u(mm[jo], ol);
#pragma unroll
      for (int j = 0; j < P; ++j)
        rt[j] += (sg[j] == v && pops_before(v, lo, mo, o, v, lam[j], mm[j], j * kW + lane)) ? 1 : 0;
    }
  }
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const int e = j * kW + lane;
    if (e < ns) s.pos[e] = (sg[j] > v || (sg[j] == v && g0 + rt[j] < stop)) ? 1 : 0;
  }
}

// ---- sigma values in pop order by a bitonic network across the wave: the delta at a pop position, and
// with it Phi and the stop test there, depend only on the sigma values in descending order (nodes that
// tie on sigma have equal deltas), so the network sorts the values alone.

// the value of lane `lane ^ J`: DPP within a row of 16 lanes (XOR 4 and 8 as two permutations each),
// an LDS permute across rows
template <int J>
__device__ __forceinline__ int xor_lane_i(int v) {
  if constexpr (J == 1) return dpp_i<0xB1, 0xF, false>(0, v);                       // quad_perm [1,0,3,2]
  else if constexpr (J == 2) return dpp_i<0x4E, 0xF, false>(0, v);                  // quad_perm [2,3,0,1]
  else if constexpr (J == 4) return dpp_i<0x141, 0xF, false>(0, dpp_i<0x1B, 0xF, false>(0, v));  // half mirror o [3,2,1,0]
  else if constexpr (J == 8) return dpp_i<0x141, 0xF, false>(0, dpp_i<0x140, 0xF, false>(0, v)); // half mirror o mirror
  else return __shfl_xor(v, J);
}
template <int J>
__device__ __forceinline__ double xor_lane(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)xor_lane_i<J>((int)(uint32_t)u);
  const uint32_t hi = (uint32_t)xor_lane_i<J>((int)(uint32_t)(u >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// one compare-exchange stage (block size KB, distance J) over element e = r * 64 + lane of v[r]
template <int P, int KB, int J>
__device__ __forceinline__ void sort_stage(double (&v)[P], int lane) {
  if constexpr (J >= kW) {
    constexpr int jr = J / kW;
#pragma unroll
    for (int r = 0; r < P; ++r) {
      if ((r ^ jr) > r) {
        const bool desc = ((r * kW + lane) & KB) == 0;
        const double a = v[r], b = v[r ^ jr];
        const double hi = fmax(a, b), lo = fmin(a, b);
        v[r] = desc ? hi : lo;
        v[r ^ jr] = desc ? lo : hi;
      }
    }
  } else {
#pragma unroll
    for (int r = 0; r < P; ++r) {
      const double o = xor_lane<J>(v[r]);
      const bool keep_max = ((lane & J) == 0) == (((r * kW + lane) & KB) == 0);
      v[r] = keep_max ? fmax(v[r], o) : fmin(v[r], o);
    }
  }
}
template <int P, int KB, int J>
__device__ __forceinline__ void sort_merge(double (&v)[P], int lane) {
  sort_stage<P, KB, J>(v, lane);
  if constexpr (J > 1) sort_merge<P, KB, J / 2>(v, lane);
}
template <int P, int KB = 2>
__device__ __forceinline__ void sort_desc(double (&v)[P], int lane) {
  sort_merge<P, KB, KB / 2>(v, lane);
  if constexpr (KB < P * kW) sort_desc<P, KB * 2>(v, lane);
}

// up to 64 nodes: the sigma values in pop order, Phi by a prefix sum over those positions; on a stop
// inside the set, the kept flags go to s.pos by generation index
__device__ Stop stop_small(const Lds& s, int ns, const StopTest& tst, int lane) {
  const bool live = lane < ns;
  double sg[1];
  sg[0] = live ? s.sl[lane].x : -INFINITY;
  const double me = sg[0];
  double srt[1] = {me};
  sort_desc<1>(srt, lane);                    // lane p: sigma at pop position p (padding last)
  const double d = live ? exp(srt[0]) : 0.0;  // delta at position `lane`
  const double incl = wave_incl_scan(d);
  const double pe = wave_shr1(incl);          // Phi before position `lane`
  const bool keep = live && kept_at(lane, pe, d, tst);
  const unsigned long long fm = __ballot(live && !keep);
  if (!fm) return Stop{ns, rl_d(incl, kW - 1), true};
  const int stop = __builtin_ctzll(fm);
  // the tie group at the stop position
  const double v = rl_d(srt[0], stop);
  const int g0 = __popcll(__ballot(live && me > v));
  if (g0 < stop) {
    cut_group_flags<1>(s, ns, sg, v, g0, stop, lane);
  } else if (live) {
    s.pos[lane] = me > v ? 1 : 0;
  }
  return Stop{stop, rl_d(pe, stop), false};
}

// The stop inside the tie group of value vA (first position mA, Phi before it phA, delta dA,
// tA members): the offset of the first member position that is not kept, or tA.
__device__ __forceinline__ int group_stop(int mA, double phA, double dA, int tA, const StopTest& tst, int lane) {
  for (int k0 = 1; k0 < tA; k0 += kW) {
    const int k = k0 + lane;
    const bool bad = k < tA && !kept_at(mA + k, phA + (double)k * dA, dA, tst);
    const unsigned long long bm = __ballot(bad);
    if (bm) return k0 + __builtin_ctzll(bm);
  }
  return tA;
}

// Sets of 65 .. 64 P nodes held in registers (node e = j * 64 + lane): the sigma values in pop order by
// the network over 64 P positions (position p = j * 64 + lane in register j), and the stop test at
// every position in parallel, 64 positions at a time, with Phi carried across them.
template <int P>
__device__ Stop stop_rank(const Lds& s, int ns, const StopTest& tst, int lane) {
  double sg[P], srt[P];
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const int e = j * kW + lane;
    sg[j] = e < ns ? s.sl[e].x : -INFINITY;
    srt[j] = sg[j];
  }
  sort_desc<P>(srt, lane);
  double carry = 0.0;                         // Phi before the current 64 positions
  int stop = ns;
  double phi = 0.0;
#pragma unroll
  for (int j = 0; j < P; ++j) {
    const int p0 = j * kW;
    if (p0 < ns && stop == ns) {              // wave-uniform
      const int p = p0 + lane;
      const bool live = p < ns;
      const double d = live ? exp(srt[j]) : 0.0;
      const double incl = wave_incl_scan(d);
      const double pe = carry + wave_shr1(incl);  // Phi before position p
      const bool keep = live && kept_at(p, pe, d, tst);
      const unsigned long long fm = __ballot(live && !keep);
      if (fm) {
        const int l = __builtin_ctzll(fm);
        stop = p0 + l;
        phi = rl_d(pe, l);
      } else {
        carry += rl_d(incl, kW - 1);
      }
    }
  }
  if (stop == ns) return Stop{ns, carry, true};
  // the tie group at the stop position
  double v = 0.0;
#pragma unroll
  for (int j = 0; j < P; ++j)
    if (stop / kW == j) v = rl_d(srt[j], stop % kW);
  int g0 = 0;
#pragma unroll
  for (int j = 0; j < P; ++j) g0 += __popcll(__ballot(sg[j] > v));
  if (g0 < stop) {
    cut_group_flags<P>(s, ns, sg, v, g0, stop, lane);
  } else {
#pragma unroll
    for (int j = 0; j < P; ++j)
      if (j * kW + lane < ns) s.pos[j * kW + lane] = sg[j] > v ? 1 : 0;
  }
  return Stop{stop, phi, false};
}

// sets above kSmall nodes: the same bisection with the values read from LDS at every step
__device__ Stop stop_lds(const Lds& s, int ns, const StopTest& tst, int lane, unsigned seed) {
  for (int e = lane; e < ns; e += kW) s.dl[e] = exp(s.sl[e].x);
  bool hasA = false, hasB = false;
  double vA = 0.0, vB = 0.0, dA = 0.0, phA = 0.0;
  int mA = 0;
  unsigned rng = seed;
  auto cand = [&](int e) -> bool {
    if (e >= ns) return false;
    const double x = s.sl[e].x;
    return (!hasA || x < vA) && (!hasB || x > vB);
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
      if (k < c) pe = e0 + __builtin_ctzll(__ballot(((mk >> lane) & 1ull) && lane_below(mk) == k));
      else k -= c;
    }
    const double v = s.sl[pe].x;
    const double pd = s.dl[pe];
    int cnt = 0;
    double part = 0.0;
    for (int e0 = 0; e0 < ns; e0 += kW) {
      const int e = e0 + lane;
      const bool bf = e < ns && s.sl[e].x > v;
      cnt += __popcll(__ballot(bf));
      part += bf ? s.dl[e] : 0.0;
    }
    const double ph = rl_d(wave_incl_scan(part), kW - 1);
    if (kept_at(cnt, ph, pd, tst)) { hasA = true; vA = v; dA = pd; mA = cnt; phA = ph; }
    else { hasB = true; vB = v; }
  }
  if (!hasA) {
    for (int e = lane; e < ns; e += kW) s.pos[e] = 0;
    return Stop{0, 0.0, false};
  }
  int tA = 0;
  for (int e0 = 0; e0 < ns; e0 += kW) {
    const int e = e0 + lane;
    tA += __popcll(__ballot(e < ns && s.sl[e < ns ? e : 0].x == vA));
  }
  const int ks = group_stop(mA, phA, dA, tA, tst, lane);
  const int n = mA + ks;
  const double phi = phA + (double)ks * dA;
  if (n == ns) return Stop{ns, phi, true};
  if (ks == tA) {
    for (int e = lane; e < ns; e += kW) s.pos[e] = s.sl[e].x >= vA ? 1 : 0;
    return Stop{n, phi, false};
  }
  // the stop cuts the group of vA: list its members (generation order) in the dl array, which
  // the bisection no longer needs, then rank each member by the members that pop before it
  int* mem = reinterpret_cast<int*>(s.dl);
  int t = 0;
  for (int e0 = 0; e0 < ns; e0 += kW) {
    const int e = e0 + lane;
    const bool g = e < ns && s.sl[e < ns ? e : 0].x == vA;
    const unsigned long long gm = __ballot(g);
    if (g) mem[t + lane_below(gm)] = e;
    t += __popcll(gm);
  }
  for (int e = lane; e < ns; e += kW) s.pos[e] = s.sl[e].x > vA ? 1 : 0;
  for (int j0 = 0; j0 < t; j0 += kW) {         // 64 members at a time ...
    const int j = j0 + lane;
    const bool live = j < t;
    const int e = mem[live ? j : 0];
    const double lam = s.sl[e].y;
    const uint32_t mme = s.meta[e];
    int rt = 0;
    for (int q0 = 0; q0 < t; q0 += kW) {        // ... against every member, 64 at a time
      const int q = q0 + lane;
      const int eo = mem[q < t ? q : 0];
      const double lo = s.sl[eo].y;
      const uint32_t mo = s.meta[eo];
      const int nq = t - q0 < kW ? t - q0 : kW;
      for (int k = 0; k < nq; ++k)
        rt += pops_before(vA, rl_d(lo, k), rl_u(mo, k), __builtin_amdgcn_readlane(eo, k), vA, lam, mme, e) ? 1 : 0;
    }
    if (live) s.pos[e] = mA + rt < n ? 1 : 0;
  }
  return Stop{n, phi, false};
}

// order-preserving 64-bit key of a double, and back
__device__ __forceinline__ unsigned long long dkey(double x) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(x);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}
__device__ __forceinline__ double dkey_inv(unsigned long long k) {
  const unsigned long long b = (k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k;
  return __longlong_as_double((long long)b);
}
constexpr double kFix = 0x1p50;   // fixed-point scale of delta in the bin sums (at most 4096 * 2^50 < 2^63)

// The stop inside the bin that holds it, of t <= 64 nodes: mem[0 .. t) are the bin's nodes in
// generation order, mk the position of its first node in the pop order and pk Phi before it.
// Ranks them by sigma (ties by index), tests every position, and marks each of them kept (1) or
// not (0) in s.pos; a tie group cut by the stop is ordered by the full pop order.  Uses s.hsum as
// scratch.
__device__ __forceinline__ Stop stop_in_bin(const Lds& s, const int* mem, int t, int mk, double pk, int ns,
                                            const StopTest& tst, int lane) {
  const bool live = lane < t;
  const int me = mem[live ? lane : 0];
  const double sg = live ? s.sl[me].x : -INFINITY;
  int r = 0;
  for (int o = 0; o < t; ++o) {
    const double so = rl_d(sg, o);
    r += (int)(so > sg) | ((int)(so == sg) & (int)(o < lane));
  }
  double* ds = reinterpret_cast<double*>(s.hsum);   // delta of the bin's nodes in sigma order
  if (live) ds[r] = s.dl[me];
  const double d = live ? ds[lane] : 0.0;
  const double incl = wave_incl_scan(d);
  const double pe = pk + wave_shr1(incl);           // Phi before position mk + lane
  const bool keep = live && kept_at(mk + lane, pe, d, tst);
  const unsigned long long fm = __ballot(live && !keep);
  const int ks = fm ? __builtin_ctzll(fm) : t;
  const int n = mk + ks;
  const double phi = fm ? rl_d(pe, ks) : pk + rl_d(incl, kW - 1);
  if (n == ns) return Stop{ns, phi, true};
  int kept = 1;
  if (ks < t) {
    const double v = rl_d(sg, __builtin_ctzll(__ballot(live && r == ks)));   // sigma at the stop
    const int g0 = __popcll(__ballot(live && sg > v));
    kept = r < ks;
    if (g0 < ks) {                      // the stop cuts a tie group: its full pop order decides
      const double lam = live ? s.sl[me].y : 0.0;
      const uint32_t mm = live ? s.meta[me] : 0u;
      int rt = 0;
      for (int o = 0; o < t; ++o) {
        const double so = rl_d(sg, o);
        if (so == v)
          rt += (live && sg == v &&
                 pops_before(v, rl_d(lam, o), rl_u(mm, o), __builtin_amdgcn_readlane(me, o), v, lam, mm, me))
                    ? 1 : 0;
      }
      kept = sg > v || (sg == v && g0 + rt < ks);
    }
  }
  if (live) s.pos[me] = kept ? 1 : 0;
  return Stop{n, phi, false};
}

// Sets above 128 nodes, in LDS.  A 64-bin histogram over the range of sigma gives, per bin,
// the node count, the largest and smallest sigma and the sum of delta in fixed point
// (integer atomics, so the sums do not depend on the order of the additions; their error,
// below ns * 2^-50, is far under the stop margins the inputs keep).  Bins are monotone in
// sigma, so the first node of every bin sits at a known position with a known Phi before
// it, and the stop test at the first node of every bin runs in parallel.  The stop lies in
// the last bin whose first node passes.  A bin of at most 64 nodes is ranked by sigma (ties
// by index) and tested one node per lane; a larger one is split by a histogram of its own
// range, up to kLevels deep.  s.pos marks each node kept (1), not kept (0) or still open (2).
// A bin of more than 64 equal values, or deeper nesting, falls back to the bisection.
constexpr int kLevels = 4;

__device__ Stop stop_hist(const Lds& s, int ns, const StopTest& tst, double lo, double hi, int lane, unsigned seed) {
  int base_m = 0;                         // position of the open range's first node
  double base_p = 0.0;                    // Phi before it
  for (int level = 0; level < kLevels; ++level) {
    if (!(hi > lo)) break;
    const double scale = (double)kBins / (hi - lo);
    auto bin = [&](double v) -> int {
      const int b = (int)((v - lo) * scale);
      return b < 0 ? 0 : (b < kBins - 1 ? b : kBins - 1);
    };
    auto open = [&](int e) -> bool { return level == 0 || s.pos[e] == 2; };
    s.hist[lane] = 0;
    s.hmax[lane] = 0ull;
    s.hmin[lane] = ~0ull;
    s.hsum[lane] = 0ull;
    for (int e0 = 0; e0 < ns; e0 += kW) {
      const int e = e0 + lane;
      if (e < ns && open(e)) {
        const double v = s.sl[e].x;
        double d;
        if (level == 0) {
          d = exp(v);
          s.dl[e] = d;
        } else {
          d = s.dl[e];
        }
        const int b = bin(v);
        atomicAdd(&s.hist[b], 1);
        atomicMax(&s.hmax[b], dkey(v));
        atomicMin(&s.hmin[b], dkey(v));
        atomicAdd(&s.hsum[b], (unsigned long long)(d * kFix));
      }
    }
    // lane b holds bin b; in reversed lane order the prefix sums run from the top bin down
    const int cnt = s.hist[lane];
    const double fs = (double)s.hsum[lane] / kFix;
    const double vmax = cnt ? dkey_inv(s.hmax[lane]) : 0.0;
    const double vmin = cnt ? dkey_inv(s.hmin[lane]) : 0.0;
    const int rl = kW - 1 - lane;
    const int cr = __shfl(cnt, rl);
    const double fr = __shfl(fs, rl);
    const int ce = wave_incl_scan(cr) - cr;
    const double fe = wave_shr1(wave_incl_scan(fr));
    const int mb = base_m + __shfl(ce, rl);     // position of bin `lane`'s first node
    const double pb = base_p + __shfl(fe, rl);  // Phi before it
    const bool keep_b = cnt == 0 || kept_at(mb, pb, exp(vmax), tst);
    const unsigned long long fails = __ballot(!keep_b);
    const unsigned long long full = __ballot(cnt > 0);
    const unsigned long long above = fails ? full & ~((2ull << (63 - __builtin_clzll(fails))) - 1ull) : full;
    if (above == 0) {                     // the open range's first node is not kept (level 0 only)
      for (int e = lane; e < ns; e += kW)
        if (open(e)) s.pos[e] = 0;
      return Stop{base_m, base_p, false};
    }
    const int bk = __builtin_ctzll(above);      // the stop lies in this bin or right after it
    const int t = __builtin_amdgcn_readlane(cnt, bk);
    const int mk = __builtin_amdgcn_readlane(mb, bk);
    const double pk = rl_d(pb, bk);
    for (int e = lane; e < ns; e += kW)
      if (open(e)) {
        const int b = bin(s.sl[e].x);
        s.pos[e] = b > bk ? 1 : (b < bk ? 0 : 2);
      }
    if (t > kW) {                         // split the bin by a histogram of its own range
      lo = rl_d(vmin, bk);
      hi = rl_d(vmax, bk);
      base_m = mk;
      base_p = pk;
      continue;
    }
    // the bin's nodes, one per lane, in generation order
    int* mem = s.hist;                    // the counts are in registers now
    {
      int nb = 0;
      for (int e0 = 0; e0 < ns; e0 += kW) {
        const int e = e0 + lane;
        const bool g = e < ns && s.pos[e < ns ? e : 0] == 2;
        const unsigned long long gm = __ballot(g);
        if (g) mem[nb + lane_below(gm)] = e;
        nb += __popcll(gm);
      }
    }
    return stop_in_bin(s, mem, t, mk, pk, ns, tst, lane);
  }
  return stop_lds(s, ns, tst, lane, seed);
}

// Raise tau in place at depth d.  Depths 1 .. d are s[0, lb) (depth d at [la, lb)); the
// children of depth d that reach tau are the candidates at depth d + 1.  Picks tau' > tau
// such that T(tau') over depths 1 .. d + 1 holds at most keep_hi nodes and, as far as the
// histogram resolves, at least `need`; compacts s[0, lb) to the nodes that reach tau'
// (order kept, parents renumbered) and updates la, lb.  Returns tau', or NaN when no such
// threshold is found.
__device__ double raise_tau(const Lds& s, int& la, int& lb, int K, double Ad, double tlv, double tau, double top,
                            int keep_hi, int need, int lane) {
  double lo_e = tau, hi_e = top;
  int above = 0;                             // nodes above the histogram's range
  double t2 = NAN;
  for (int pass = 0; pass < kRefine; ++pass) {
    if (!(hi_e > lo_e)) break;
    const double scale = (double)kBins / (hi_e - lo_e);
    const bool first = pass == 0;            // the first pass also takes the values at hi_e
    auto bin = [&](double v) -> int {
      const int b = (int)((v - lo_e) * scale);
      return b < kBins - 1 ? b : kBins - 1;
    };
    s.hist[lane] = 0;
    for (int i0 = 0; i0 < lb; i0 += kW) {
      const int i = i0 + lane;
      if (i < lb) {
        const double v = s.sl[i].x;
        if (v >= lo_e && (first || v < hi_e)) atomicAdd(&s.hist[bin(v)], 1);
      }
    }
    for (int p0 = la; p0 < lb; p0 += kW) {
      const int p = p0 + lane;
      const bool live = p < lb;
      const double2 pv = s.sl[live ? p : la];
      for (int r = 0; r < K; ++r) {
        const double x = (pv.y + rl_d(tlv, r)) - Ad;
        const bool q = live && x >= tau;
        if (__ballot(q) == 0) break;
        if (q) {
          const double v = pmin(x, pv.x);
          if (v >= lo_e && (first || v < hi_e)) atomicAdd(&s.hist[bin(v)], 1);
        }
      }
    }
    const int h = s.hist[lane];
    const int incl = wave_incl_scan(h);
    const int tot = __builtin_amdgcn_readlane(incl, kW - 1);
    const int S = above + tot - (incl - h);   // nodes in bins >= lane, and above the range
    const unsigned long long okm = __ballot(S <= keep_hi);
    const int b1 = okm ? __builtin_ctzll(okm) : kBins;
    const int S1 = b1 < kBins ? __builtin_amdgcn_readlane(S, b1) : above;
    if (b1 == 0) break;                       // everything fits: nothing to raise
    if (S1 >= need) {
      t2 = lo_e + (hi_e - lo_e) * ((double)b1 / (double)kBins);
      break;
    }
    // bin b1 - 1 holds both bounds: split it
    above = S1;
    const double w = (hi_e - lo_e) / (double)kBins;
    hi_e = lo_e + w * (double)b1;
    lo_e = lo_e + w * (double)(b1 - 1);
  }
  if (!(t2 > tau)) return NAN;
  // compact s[0, lb) to the nodes with sigma >= t2
  int base = 0, la2 = 0;
  for (int i0 = 0; i0 < lb; i0 += kW) {
    const int i = i0 + lane;
    const bool live = i < lb;
    const double2 v = s.sl[live ? i : 0];
    const uint32_t m = s.meta[live ? i : 0];
    const bool keep = live && v.x >= t2;
    const unsigned long long km = __ballot(keep);
    const int j = base + lane_below(km);
    if (live) s.pos[i] = keep ? (int16_t)j : (int16_t)-1;
    const int par = m_parent(m);
    const int np = (keep && par >= 0) ? (int)s.pos[par] : -1;   // parents come first and are kept
    if (keep) {
      s.sl[j] = v;
      s.meta[j] = pack(np, m_rank(m), m_depth(m));
    }
    if (la >= i0 && la < i0 + kW) la2 = base + __popcll(km & ((1ull << (la - i0)) - 1ull));
    base += __popcll(km);
  }
  la = la2;
  lb = base;
  return t2;
}

// The largest sigma among the nodes outside the set s[0, ns) = T(tau), where every node of the set is
// kept and the tree continues: the next pop, whose delta decides whether the stop falls right after
// the set.  Every node outside T(tau) descends from, or is a later sibling of, a frontier node (the
// first child of a node with no child in the set, or the next sibling of a node that is its
// parent's last child in the set; siblings are contiguous in generation order), and sigma does not
// rise along either step, so the largest sigma outside is the largest over the frontier.  Each
// frontier node's sigma is formed as the build forms a child's.  Uses s.pos as scratch.  The
// caller reads the result through readlane: the compiler cannot see that the butterfly leaves it
// wave-uniform, and a value it takes for divergent would make the attempt loop's control
// divergent after it.
__device__ double frontier_max(const Lds& s, int ns, int L, int K, double Areg, int lane) {
  for (int i = lane; i < ns; i += kW) s.pos[i] = 0;
  for (int i = lane; i < ns; i += kW) {
    const int p = m_parent(s.meta[i]);
    if (p >= 0) s.pos[p] = 1;               // p has a child in the set
  }
  double best = -INFINITY;
  for (int i0 = 0; i0 < ns; i0 += kW) {
    const int i = i0 + lane;
    const bool live = i < ns;
    const int ii = live ? i : 0;
    const uint32_t m = s.meta[ii];
    const int p = m_parent(m), r = m_rank(m), d = m_depth(m);
    const double2 v = s.sl[ii];
    const double Ad = __shfl(Areg, d);            // A_d
    const double Ad1 = __shfl(Areg, d < L ? d + 1 : d);
    if (live && d < L && s.pos[ii] == 0) {        // first child: rank 0 at depth d + 1
      const double l = v.y + (double)s.tl[d * K];
      best = fmax(best, pmin(l - Ad1, v.x));
    }
    const bool last = i + 1 >= ns || m_parent(s.meta[i + 1 < ns ? i + 1 : ii]) != p;
    if (live && last && r + 1 < K) {              // next sibling: rank r + 1 at depth d
      const double2 pv = p < 0 ? make_double2(0.0, 0.0) : s.sl[p];   // the root: sigma 0, Lambda 0
      const double l = pv.y + (double)s.tl[(d - 1) * K + r + 1];
      best = fmax(best, pmin(l - Ad, pv.x));
    }
  }
  for (int k = 1; k < kW; k <<= 1) best = fmax(best, __shfl_xor(best, k));
  return best;   // the same in every lane (the caller reads it as a wave-uniform value)
}

}  // namespace
}  // namespace caddtree
