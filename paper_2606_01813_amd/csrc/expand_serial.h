// Stage 2, serial form: Algorithm 1 (Sec. 4.5) -- best-first expansion of the
// draft tree with the greedy throughput stop -- and the breadth-first layout of
// the result, for one round, by one workgroup (one 64-lane wavefront), in the
// dynamic LDS.  One pop at a time, exactly as Algorithm 1 runs.
//
// expand.hip runs it as a kernel (every round of a plan the batched form does
// not serve, or the rounds the batched form hands back); expand_level.hip calls
// it in place for a round it cannot settle when the plan's LDS allows.
//
// Keys.  A node s = (s_1 .. s_d) (0-based ranks) has Lambda(s) = sum_{i<=d}
// l_i^(s_i) (raw fp32 logits widened to fp64, summed in depth order) and log
// prefix probability sigma(s) = min(Lambda(s) - A_d, sigma(parent)),
// A_d = sum_{i<=d} LSE_i, sigma(root) = 0 (eq. prefix-prob; the clamp keeps a
// child from ranking above its parent under rounding).  Nodes pop in the total
// order: sigma desc, depth asc, Lambda desc, rank tuple lexicographically asc.
// Every node's predecessor (previous sibling, or the parent for a first child)
// comes first in that order, so a priority queue pops nodes in exactly that
// order and any correct priority queue gives the same tree.
//
// Stop (Algorithm 1; Lemma 1): with C(n) = C_d + C_v(n), the popped node is
// kept iff ((1 + Phi) + delta) / C(n + 1) > theta_prev, delta = exp(sigma);
// the loop also ends at the budget cap or when the queue is empty.
//
// Frontier.  The queue is a sorted list held in registers across the wave:
// position p = 64 * slot + lane, ascending towards the next node to pop, up to
// kSlots * 64 entries.  Popping reads the top position; a push counts, with one
// ballot per slot, the entries that pop after the new node and shifts the ones
// above it up by one lane (DPP wave_shr).  Neither touches LDS.  A round whose
// frontier outgrows the register list moves it into an LDS binary heap and
// continues there (same order, same results, slower).
//
// Per-round values live in registers too: lane d holds A_d, and the lanes hold
// 64 consecutive values of C(n + 1) (the next 64 are prefetched from HBM).
// Kept nodes (Lambda, sigma, packed parent/rank/depth, 128-bit rank-tuple key)
// go to LDS.
//
// Layout.  The breadth-first position of a kept node is the number of kept
// nodes before it in (depth, rank tuple); with the packed keys every lane
// counts for its nodes in parallel.  Rounds that used the heap, or kept more
// than 512 nodes, renumber with a serial walk over a child table instead (the
// children of a kept node are ranks 0 .. c-1, since a kept node's
// predecessors are kept).

#pragma once

#include <cmath>
#include <type_traits>

#include "emit_wave.h"
#include "expand_common.h"

namespace caddtree {
namespace serial {

constexpr int kThreads = 64;
constexpr int kSlots = 4;                  // register frontier capacity = 256 entries
constexpr int kRegCap = kSlots * kThreads;
constexpr int kParallelLayoutMax = 512;

using namespace xp;

// lane i <- lane i - 1 across the whole wave (lane 0 keeps its own value)
__device__ __forceinline__ uint32_t wshr_u(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x138, 0xF, 0xF, false);
}
__device__ __forceinline__ double wshr_d(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = wshr_u((uint32_t)u), hi = wshr_u((uint32_t)(u >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Rank tuples of two distinct same-depth nodes given as (parent, rank): walk
// both parent chains up to the common ancestor and compare the ranks below it.
__device__ __forceinline__ bool rank_tuple_less(const uint32_t* smeta, int pa, int ra, int pb, int rb) {
  while (pa != pb) {
    const uint32_t xa = smeta[pa], xb = smeta[pb];
    ra = m_rank(xa); rb = m_rank(xb);
    pa = m_parent(xa); pb = m_parent(xb);
  }
  return ra < rb;
}

// true iff node a pops before node b
__device__ __forceinline__ bool pops_before(double sa, double la, uint32_t ma, double sb, double lb, uint32_t mb,
                                            const uint32_t* smeta) {
  if (sa != sb) return sa > sb;
  const int da = m_depth(ma), db = m_depth(mb);
  if (da != db) return da < db;
  if (la != lb) return la > lb;
  return rank_tuple_less(smeta, m_parent(ma), m_rank(ma), m_parent(mb), m_rank(mb));
}

// ---------------------------------------------------------------- LDS heap (overflow path)
struct Heap {
  const float* tl;
  const double* slam;
  const uint32_t* smeta;
  double* hsig;
  uint32_t* hmeta;
  int K;

  __device__ double lam_of(uint32_t m) const {
    const int p = m_parent(m);
    const double base = p >= 0 ? slam[p] : 0.0;
    return base + (double)tl[(m_depth(m) - 1) * K + m_rank(m)];
  }
  __device__ bool before(double sa, uint32_t ma, double sb, uint32_t mb) const {
    if (sa != sb) return sa > sb;
    if (m_depth(ma) != m_depth(mb)) return m_depth(ma) < m_depth(mb);
    const double la = lam_of(ma), lb = lam_of(mb);
    if (la != lb) return la > lb;
    return rank_tuple_less(smeta, m_parent(ma), m_rank(ma), m_parent(mb), m_rank(mb));
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

// ---------------------------------------------------------------- LDS layout
// The union region holds, one at a time: the kept nodes' rank-tuple keys, the
// overflow heap, and the serial layout's scratch.
__host__ __device__ __forceinline__ size_t union_bytes(size_t ncap) {
  const size_t keys = 16 * ncap;
  const size_t heap = a16(8 * (ncap + 1)) + 4 * (ncap + 1);
  const size_t serial = 10 * ncap + 4;
  const size_t m = keys > heap ? keys : heap;
  return a16(m > serial ? m : serial);
}

struct Lds {
  float* tl;          // [L * K] raw logits
  int32_t* tid;       // [L * K] token ids
  double* slam;       // kept nodes, pop order
  double* ssig;
  uint32_t* smeta;
  uint64_t* key;      // [2 * cap]: (hi, lo) rank-tuple key per kept node   } union
  double* hsig;       // overflow heap keys                                  }
  uint32_t* hmeta;    //                                                     }
  int16_t* pos;       // [cap] breadth-first position of each kept node
};

__device__ Lds carve(unsigned char* smem, size_t LK, size_t ncap) {
  Lds s;
  size_t off = 0;
  s.tl = reinterpret_cast<float*>(smem + off);        off = a16(off + sizeof(float) * LK);
  s.tid = reinterpret_cast<int32_t*>(smem + off);     off = a16(off + sizeof(int32_t) * LK);
  s.slam = reinterpret_cast<double*>(smem + off);     off = a16(off + sizeof(double) * ncap);
  s.ssig = reinterpret_cast<double*>(smem + off);     off = a16(off + sizeof(double) * ncap);
  s.smeta = reinterpret_cast<uint32_t*>(smem + off);  off = a16(off + sizeof(uint32_t) * ncap);
  unsigned char* u = smem + off;
  s.key = reinterpret_cast<uint64_t*>(u);
  s.hsig = reinterpret_cast<double*>(u);
  s.hmeta = reinterpret_cast<uint32_t*>(u + a16(8 * (ncap + 1)));
  off += union_bytes(ncap);
  s.pos = reinterpret_cast<int16_t*>(smem + off);
  return s;
}

inline size_t lds_bytes(size_t LK, size_t ncap) {
  size_t off = 0;
  off = a16(off + sizeof(float) * LK);
  off = a16(off + sizeof(int32_t) * LK);
  off = a16(off + sizeof(double) * ncap);
  off = a16(off + sizeof(double) * ncap);
  off = a16(off + sizeof(uint32_t) * ncap);
  off += union_bytes(ncap);
  off = a16(off + sizeof(int16_t) * ncap);
  return off;
}

// What a round reads and writes (device pointers; the optional outputs may be null).
struct Args {
  const int32_t* topk_ids;
  const float* topk_logit;
  const double* lse;
  int L, K, cap;
  CostTables ct;
  int fixed;
  int32_t* token_ids;
  int32_t* parent_out;
  int32_t* depth_out;
  float* path_prob;
  int32_t* n_star_out;
  float* phi_out;
  float* theta_out;
  EmitOut em;          // mask and position ids, when this epilogue writes them
};

// Round b, by the calling 64-lane workgroup, in the dynamic LDS (lds_bytes(L * K, cap) bytes).
__device__ __forceinline__ void expand_round(const Args& a, int b) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int32_t* __restrict__ topk_ids = a.topk_ids;
  const float* __restrict__ topk_logit = a.topk_logit;
  const double* __restrict__ lse = a.lse;
  const int L = a.L, K = a.K, cap = a.cap, fixed = a.fixed;
  const CostTables ct = a.ct;
  int32_t* __restrict__ token_ids = a.token_ids;
  int32_t* __restrict__ parent_out = a.parent_out;
  int32_t* __restrict__ depth_out = a.depth_out;
  float* __restrict__ path_prob = a.path_prob;
  int32_t* __restrict__ n_star_out = a.n_star_out;
  float* __restrict__ phi_out = a.phi_out;
  float* __restrict__ theta_out = a.theta_out;
  const int lane = threadIdx.x;
  const int LK = L * K;
  const Lds s = carve(smem, (size_t)LK, cap > 0 ? (size_t)cap : 1);
  const RoundCost C = round_cost(ct, b);

  for (int i = lane; i < LK; i += kThreads) {
    s.tl[i] = topk_logit[(int64_t)b * LK + i];
    s.tid[i] = topk_ids[(int64_t)b * LK + i];
  }
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
  // the lanes hold C(64 k + 1 + lane) for the current block k and prefetch block k + 1
  double cblk = lane + 1 <= cap ? C(lane + 1) : 1.0;
  double cnxt = 64 + lane + 1 <= cap ? C(64 + lane + 1) : 1.0;
  const double c0 = C(0);
  __syncthreads();

  // register frontier: positions [0, f), ascending towards the next pop
  double fs[kSlots], fl[kSlots];
  uint32_t fm[kSlots];
#pragma unroll
  for (int j = 0; j < kSlots; ++j) { fs[j] = -INFINITY; fl[j] = 0.0; fm[j] = 0; }
  int f = 0, n = 0;
  double phi = 0.0;
  double theta_prev = 1.0 / c0;
  bool used_heap = false;

  // insert x into the sorted register list; NS = slots in use (compile time)
  auto push = [&](auto ns_tag, double xs, double xl, uint32_t xm) {
    constexpr int NS = decltype(ns_tag)::value;
    int q = 0;   // entries that pop after x
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      const int p = j * kThreads + lane;
      const bool valid = p < f;
      bool w = valid && xs > fs[j];
      const bool tie = valid && xs == fs[j];
      if (__ballot(tie)) {
        if (tie) w = pops_before(xs, xl, xm, fs[j], fl[j], fm[j], s.smeta);
      }
      q += __popcll(__ballot(w));
    }
#pragma unroll
    for (int j = NS - 1; j >= 0; --j) {
      const int p = j * kThreads + lane;
      double ss = wshr_d(fs[j]), sl = wshr_d(fl[j]);
      uint32_t sm = wshr_u(fm[j]);
      if (j > 0) {
        const double cs = rl_d(fs[j - 1], 63), cl = rl_d(fl[j - 1], 63);
        const uint32_t cm = rl_u(fm[j - 1], 63);
        if (lane == 0) { ss = cs; sl = cl; sm = cm; }
      }
      const bool up = p > q, at = p == q;
      fs[j] = up ? ss : (at ? xs : fs[j]);
      fl[j] = up ? sl : (at ? xl : fl[j]);
      fm[j] = up ? sm : (at ? xm : fm[j]);
    }
    ++f;
  };

  {
    const double lam = 0.0 + (double)s.tl[0];
    push(std::integral_constant<int, 1>{}, pmin(lam - rl_d(Areg, 1), 0.0), lam, pack(-1, 0, 1));
  }

  // one pop of Algorithm 1 with NS register slots; returns false when the loop ends
  auto step = [&](auto ns_tag) -> bool {
    constexpr int NS = decltype(ns_tag)::value;
    const int top = f - 1;
    const int tlane = top & 63;
    double sig = 0.0, lam = 0.0;
    uint32_t meta = 0;
    if (NS == 1) {
      sig = rl_d(fs[0], tlane); lam = rl_d(fl[0], tlane); meta = rl_u(fm[0], tlane);
    } else {
      const int tj = top >> 6;
#pragma unroll
      for (int j = 0; j < NS; ++j)
        if (j == tj) { sig = rl_d(fs[j], tlane); lam = rl_d(fl[j], tlane); meta = rl_u(fm[j], tlane); }
    }
    const int p = m_parent(meta), r = m_rank(meta), d = m_depth(meta);
    // issue every LDS read of this pop up front (clamped indices, selected later)
    const int pc = p >= 0 ? p : 0;
    const double raw_lam = s.slam[pc], raw_sig = s.ssig[pc];
    const uint64_t raw_hi = s.key[2 * pc], raw_lo = s.key[2 * pc + 1];
    const float raw_sib = s.tl[(d - 1) * K + (r + 1 < K ? r + 1 : r)];
    const float raw_child = s.tl[(d < L ? d : d - 1) * K];
    const double delta = exp(sig);
    const double theta_new = (1.0 + phi + delta) / rl_d(cblk, n & 63);
    if (!fixed && theta_new <= theta_prev) return false;
    --f;
    const double base_lam = p >= 0 ? raw_lam : 0.0;
    const double base_sig = p >= 0 ? raw_sig : 0.0;
    const uint64_t pk_hi = p >= 0 ? raw_hi : 0, pk_lo = p >= 0 ? raw_lo : 0;
    phi += delta;
    theta_prev = theta_new;
    const int me = n++;
    if ((n & 63) == 0) {
      cblk = cnxt;
      const int idx = n + 64 + lane + 1;
      cnxt = idx <= cap ? C(idx) : 1.0;
    }
    if (lane == 0) {   // before the pushes: their tie-breaks may walk through this node
      s.slam[me] = lam; s.ssig[me] = sig; s.smeta[me] = meta;
      s.key[2 * me] = (pk_hi << 4) | (pk_lo >> 60);
      s.key[2 * me + 1] = (pk_lo << 4) | (uint64_t)r;
    }
    if (r + 1 < K) {
      const double ls = base_lam + (double)raw_sib;
      push(ns_tag, pmin(ls - rl_d(Areg, d), base_sig), ls, pack(p, r + 1, d));
    }
    if (d < L) {
      const double lc = lam + (double)raw_child;
      push(ns_tag, pmin(lc - rl_d(Areg, d + 1), sig), lc, pack(me, 0, d + 1));
    }
    return true;
  };

  bool go = true;
  while (go && f > 0 && n < cap && f < kThreads) go = step(std::integral_constant<int, 1>{});
  while (go && f > 0 && n < cap && f < kRegCap) go = step(std::integral_constant<int, kSlots>{});
  if (go && f > 0 && n < cap) used_heap = true;

  if (used_heap) {
    // move the register list into an LDS max-heap (descending order is a valid heap)
#pragma unroll
    for (int j = 0; j < kSlots; ++j) {
      const int p = j * kThreads + lane;
      if (p < f) { s.hsig[f - 1 - p] = fs[j]; s.hmeta[f - 1 - p] = fm[j]; }
    }
    __syncthreads();
    if (lane == 0) {
      const Heap H{s.tl, s.slam, s.smeta, s.hsig, s.hmeta, K};
      double cnext = n < cap ? C(n + 1) : 0.0;
      while (f > 0 && n < cap) {
        const double sig = s.hsig[0];
        const uint32_t meta = s.hmeta[0];
        const double delta = exp(sig);
        const double theta_new = (1.0 + phi + delta) / cnext;
        if (!fixed && theta_new <= theta_prev) break;
        const int p = m_parent(meta), r = m_rank(meta), d = m_depth(meta);
        const double base_lam = p >= 0 ? s.slam[p] : 0.0;
        const double base_sig = p >= 0 ? s.ssig[p] : 0.0;
        const double lam = base_lam + (double)s.tl[(d - 1) * K + r];
        s.slam[n] = lam; s.ssig[n] = sig; s.smeta[n] = meta;
        phi += delta;
        theta_prev = theta_new;
        const int me = n++;
        if (n < cap) cnext = C(n + 1);
        bool has_child = d < L;
        double cs = 0.0;
        uint32_t cm = 0;
        if (has_child) {
          const double lc = lam + (double)s.tl[d * K];
          cs = pmin(lc - rl_d(Areg, d + 1), sig);
          cm = pack(me, 0, d + 1);
        }
        if (r + 1 < K) {
          const double ls = base_lam + (double)s.tl[(d - 1) * K + r + 1];
          H.sift_down(0, f, pmin(ls - rl_d(Areg, d), base_sig), pack(p, r + 1, d));
        } else if (has_child) {
          H.sift_down(0, f, cs, cm);
          has_child = false;
        } else {
          --f;
          if (f > 0) H.sift_down(0, f, s.hsig[f], s.hmeta[f]);
        }
        if (has_child) H.sift_up(f++, cs, cm);
      }
      // hand the final scalars to the other lanes
      s.hsig[0] = phi;
      s.hsig[1] = theta_prev;
      s.hmeta[0] = (uint32_t)n;
    }
    __syncthreads();
    phi = s.hsig[0];
    theta_prev = s.hsig[1];
    n = (int)s.hmeta[0];
    __syncthreads();
  }

  if (lane == 0) {
    n_star_out[b] = n;
    if (phi_out) phi_out[b] = (float)phi;
    if (theta_out) theta_out[b] = (float)theta_prev;
  }

  if (!used_heap && n <= kParallelLayoutMax) {
    // position = number of kept nodes before this one in (depth, rank tuple)
    for (int v = lane; v < n; v += kThreads) {
      const int dv = m_depth(s.smeta[v]);
      const uint64_t hv = s.key[2 * v], lv = s.key[2 * v + 1];
      int cnt = 0;
      for (int u = 0; u < n; ++u) {
        const int du = m_depth(s.smeta[u]);
        const uint64_t hu = s.key[2 * u], lu = s.key[2 * u + 1];
        cnt += (du < dv || (du == dv && (hu < hv || (hu == hv && lu < lv)))) ? 1 : 0;
      }
      s.pos[v] = (int16_t)cnt;
    }
  } else if (lane == 0) {
    // serial breadth-first walk over a child table
    int16_t* cnt = reinterpret_cast<int16_t*>(s.key);  // [n + 1], the root at n
    int16_t* cst = cnt + (n + 1);                       // [n + 1]
    int16_t* kids = cst + (n + 1);                      // [n]
    int16_t* order = kids + n;                          // [n]
    for (int i = 0; i <= n; ++i) cnt[i] = 0;
    for (int v = 0; v < n; ++v) {
      const int pp = m_parent(s.smeta[v]);
      cnt[pp < 0 ? n : pp]++;
    }
    int acc = 0;
    for (int i = 0; i <= n; ++i) { cst[i] = (int16_t)acc; acc += cnt[i]; }
    for (int v = 0; v < n; ++v) {
      const uint32_t m = s.smeta[v];
      const int pp = m_parent(m);
      kids[cst[pp < 0 ? n : pp] + m_rank(m)] = (int16_t)v;
    }
    int tail = 0;
    for (int k = 0; k < cnt[n]; ++k) {
      const int v = kids[cst[n] + k];
      order[tail] = (int16_t)v;
      s.pos[v] = (int16_t)tail++;
    }
    for (int i = 0; i < n; ++i) {
      const int u = order[i];
      for (int k = 0; k < cnt[u]; ++k) {
        const int v = kids[cst[u] + k];
        order[tail] = (int16_t)v;
        s.pos[v] = (int16_t)tail++;
      }
    }
  }
  __syncthreads();

  const int64_t ob = (int64_t)b * cap;
  int16_t* par = reinterpret_cast<int16_t*>(s.slam);     // output parents, for the mask (slam is done)
  for (int v = lane; v < n; v += kThreads) {
    const uint32_t m = s.smeta[v];
    const int p = m_parent(m), d = m_depth(m), r = m_rank(m);
    const int i = s.pos[v];
    const int pi = p < 0 ? -1 : (int)s.pos[p];
    token_ids[ob + i] = s.tid[(d - 1) * K + r];
    parent_out[ob + i] = pi;
    depth_out[ob + i] = d;
    if (path_prob) path_prob[ob + i] = (float)exp(s.ssig[v]);
    if (a.em.pos_ids) a.em.pos_ids[ob + i] = a.em.pos_offset + d;
    par[i] = (int16_t)pi;
  }
  __syncthreads();
  // the mask, in the key/heap region (free now; it holds emit_tile_bytes(n) <= 16 cap bytes)
  emit_mask_wave(par, n, cap, a.em.mask_kind, round_mask(a.em, b, cap), reinterpret_cast<uint32_t*>(s.key), lane);
}

}  // namespace serial
}  // namespace caddtree
