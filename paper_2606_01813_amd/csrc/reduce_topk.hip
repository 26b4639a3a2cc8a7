// Stage 1: per (round, position) row, the full-vocabulary log-normaliser
// LSE = log sum_v exp(l_v) and the top-K tokens by (logit desc, id asc)
// (Sec. 3.2, eq. marginals; the Require line of Algorithm 1).
//
// One HBM pass per row.  A row is cut into `waves_per_row` contiguous
// segments, one wavefront each, all in one workgroup.  A wavefront streams
// 16-byte loads (8 bf16 or 4 fp32 per lane, 1 KiB per wave per load) and
// keeps, per lane, an fp64 sum of 2^(x log2 e - r) where r is a wave-uniform
// integer exponent that only grows: when it moves, the sums are rescaled by an
// exact power of two.  The exponent argument is formed with a two-part log2 e
// (two fmas), so the only per-term error is the hardware exp2.
//
// Top-K: the wave keeps a sorted list of 16 slots in lanes 0..15 of its first
// DPP row.  An element is a candidate when it is >= the wave threshold (the
// K-th slot, or an initial lower bound); the fast path is one compare of the
// lane's chunk maximum per 8 elements, and the rare path inserts candidates one
// at a time with a DPP row shift.  The initial bound is the minimum over K'
// (>= K) disjoint lane groups of the group maximum over the first chunks, which
// is <= the K-th largest element, so no top-K element is ever filtered out.
//
// At the end, wave 0 merges the waves' lists (when their K best fit in one wave, each
// candidate, as a 64-bit key, is ranked against all of them in one pass), combines the
// per-wave sums,
// and replaces the top-K terms' fp32 exp2 values (recomputed bit-identically
// from the exponent recorded at insertion) by fp64 values, which removes the
// error of the largest terms from the normaliser.

#include <climits>
#include <cmath>

#include "expand_common.h"
#include "internal.h"

namespace caddtree {
namespace {

constexpr int kWave = 64;
constexpr float kLog2eHi = 0x1.715476p+0f;     // log2(e) rounded to fp32
constexpr float kLog2eLo = 0x1.4ae0c0p-26f;    // log2(e) - kLog2eHi, rounded to fp32
constexpr double kLog2eD = 0x1.71547652b82fep+0;
constexpr double kLn2D = 0x1.62e42fefa39efp-1;
constexpr float kNoExp = -1.0e30f;             // "no reference exponent yet"

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// streaming 16-byte load with the non-temporal hint: each byte of the logits is read once
__device__ __forceinline__ uint4 stream_load(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

template <typename T> struct Vec;
template <> struct Vec<float> { static constexpr int n = 4; };
template <> struct Vec<uint16_t> { static constexpr int n = 8; };

__device__ __forceinline__ float readlane_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ int readlane_i(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

// lane k <- lane k-1 inside each row of 16 lanes; lane 0 of a row gets 0
__device__ __forceinline__ int shr1(int v) { return __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true); }
__device__ __forceinline__ float shr1f(float v) { return __int_as_float(shr1(__float_as_int(v))); }

// the maximum over the wave, wave-uniform: a DPP max-scan (row shifts, then row broadcasts; a lane
// with no source keeps its own value), whose last lane holds the total
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_keep(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, ROW_MASK, 0xF, false));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_keep<0x111, 0xF>(v));
  v = fmaxf(v, dpp_keep<0x112, 0xF>(v));
  v = fmaxf(v, dpp_keep<0x114, 0xF>(v));
  v = fmaxf(v, dpp_keep<0x118, 0xF>(v));
  v = fmaxf(v, dpp_keep<0x142, 0xA>(v));
  v = fmaxf(v, dpp_keep<0x143, 0xC>(v));
  return readlane_f(v, kWave - 1);
}

// (v, id) goes before (w, wid) in the order value desc, id asc
__device__ __forceinline__ bool before(float v, int id, float w, int wid) {
  return v > w || (v == w && id < wid);
}

__device__ __forceinline__ float term(float x, float r) {
  float a = fmaf(x, kLog2eHi, -r);
  a = fmaf(x, kLog2eLo, a);
  return __builtin_amdgcn_exp2f(a);
}

struct WaveState {
  double acc;     // per lane
  float r;        // wave-uniform reference exponent (integral value)
  float mx;       // wave-uniform running maximum
  float thr;      // wave-uniform candidate threshold
  int thr_id;
  float lv;       // list slot (lanes 0..15): value, id, exponent at insertion
  int lid;
  float lr;
};

__device__ __forceinline__ void list_insert(WaveState& s, float v, int id, float r, int K) {
  const bool b = before(v, id, s.lv, s.lid);
  const float pv = shr1f(s.lv);
  const int pid = shr1(s.lid);
  const float pr = shr1f(s.lr);
  const int pb = shr1(b ? 1 : 0);
  if (b) {
    if (pb) { s.lv = pv; s.lid = pid; s.lr = pr; }
    else    { s.lv = v;  s.lid = id;  s.lr = r; }
  }
  const int kid = readlane_i(s.lid, K - 1);
  if (kid != INT_MAX) { s.thr = readlane_f(s.lv, K - 1); s.thr_id = kid; }
}

// Rare path of one chunk: move the reference exponent, then insert candidates.
// x[j] is element base + lane * VEC + j; valid elements have bit j set in ok.
template <int VEC>
__device__ __forceinline__ void rare(WaveState& s, const float (&x)[VEC], unsigned ok, float cmax, int base, int K) {
  if (__ballot(cmax > s.mx)) {
    const float m = wave_max(cmax);
    s.mx = m;
    const float nr = ceilf(m * kLog2eHi);
    if (nr > s.r) {
      s.acc = ldexp(s.acc, (int)fmaxf(s.r - nr, -2000.f));
      s.r = nr;
    }
  }
#pragma unroll
  for (int j = 0; j < VEC; ++j) {
    unsigned long long m = __ballot(((ok >> j) & 1u) && x[j] >= s.thr);
    while (m) {
      const int l = __builtin_ctzll(m);
      m &= m - 1;
      const float v = readlane_f(x[j], l);
      const int id = base + l * VEC + j;
      if (before(v, id, s.thr, s.thr_id)) list_insert(s, v, id, s.r, K);
    }
  }
}

template <int VEC>
__device__ __forceinline__ void chunk(WaveState& s, const float (&x)[VEC], unsigned ok, int base, int K) {
  float cmax = -INFINITY;
#pragma unroll
  for (int j = 0; j < VEC; ++j) cmax = ((ok >> j) & 1u) ? fmaxf(cmax, x[j]) : cmax;
  if (__builtin_expect(__ballot(cmax >= s.thr) != 0, 0)) rare<VEC>(s, x, ok, cmax, base, K);
#pragma unroll
  for (int j = 0; j < VEC; ++j) {
    const float t = term(x[j], s.r);
    s.acc += ((ok >> j) & 1u) ? (double)t : 0.0;
  }
}

// A full chunk.  Every lane adds its terms pairwise in fp32 and the result once in
// fp64.  A lane whose elements include a top-K candidate (the rare path) then adds the
// fp64 difference between its terms summed one by one and that fp32 sum, so its
// contribution is the fp64 sum of its fp32 terms and the final fp64 correction of the
// top-K terms removes their whole error.
template <int VEC>
__device__ __forceinline__ void chunk_full(WaveState& s, const float (&x)[VEC], int base, int K) {
  float cmax = x[0];
#pragma unroll
  for (int j = 1; j < VEC; ++j) cmax = fmaxf(cmax, x[j]);
  const bool cand = cmax >= s.thr;
  const bool any = __ballot(cand) != 0;
  if (__builtin_expect(any, 0)) rare<VEC>(s, x, (1u << VEC) - 1u, cmax, base, K);
  float t[VEC], p[VEC];
#pragma unroll
  for (int j = 0; j < VEC; ++j) p[j] = t[j] = term(x[j], s.r);
#pragma unroll
  for (int w = 1; w < VEC; w <<= 1)
#pragma unroll
    for (int j = 0; j + w < VEC; j += 2 * w) p[j] += p[j + w];
  s.acc += (double)p[0];
  if (__builtin_expect(any, 0) && cand) {
    double e = 0.0;
#pragma unroll
    for (int j = 0; j < VEC; ++j) e += (double)t[j];
    s.acc += e - (double)p[0];
  }
}

__device__ __forceinline__ void unpack(const uint4& q, float (&x)[8]) {
  x[0] = __uint_as_float(q.x << 16); x[1] = __uint_as_float(q.x & 0xffff0000u);
  x[2] = __uint_as_float(q.y << 16); x[3] = __uint_as_float(q.y & 0xffff0000u);
  x[4] = __uint_as_float(q.z << 16); x[5] = __uint_as_float(q.z & 0xffff0000u);
  x[6] = __uint_as_float(q.w << 16); x[7] = __uint_as_float(q.w & 0xffff0000u);
}
__device__ __forceinline__ void unpack(const uint4& q, float (&x)[4]) {
  x[0] = __uint_as_float(q.x); x[1] = __uint_as_float(q.y);
  x[2] = __uint_as_float(q.z); x[3] = __uint_as_float(q.w);
}

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }

// guarded element-wise load of one lane's VEC elements starting at element e
template <typename T, int VEC>
__device__ __forceinline__ unsigned load_guarded(const T* rowp, int e, int V, float (&x)[VEC]) {
  unsigned ok = 0;
#pragma unroll
  for (int j = 0; j < VEC; ++j) {
    if (e + j < V) { x[j] = to_f32(rowp[e + j]); ok |= 1u << j; }
    else x[j] = -INFINITY;
  }
  return ok;
}

// (value, id) as one unsigned 64-bit key whose order is the top-K order: the value's bits mapped
// to an unsigned integer that grows with the value (-0 taken as +0, which compares equal to it),
// then INT_MAX - id (smaller ids first)
__device__ __forceinline__ uint64_t order_key(float v, int id) {
  uint32_t b = (uint32_t)__float_as_int(v);
  if (b == 0x80000000u) b = 0u;
  const uint32_t u = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((uint64_t)u << 32) | (uint32_t)(INT_MAX - id);
}
__device__ __forceinline__ int key_id(uint64_t k) { return INT_MAX - (int)(uint32_t)k; }

// kUnroll: 16-byte loads in flight per lane (4 or 8); kS: wavefronts per row (1 .. 16)
template <typename T, bool kAligned, int kUnroll, int kS>
__global__ void __launch_bounds__(1024)
reduce_topk_kernel(const T* __restrict__ logits, int64_t row_stride, int V, int K,
                   int32_t* __restrict__ out_ids, float* __restrict__ out_logit,
                   float* __restrict__ out_lq, double* __restrict__ out_lse) {
  constexpr int VEC = Vec<T>::n;
  constexpr int CH = kWave * VEC;
  __shared__ double s_acc[16];
  __shared__ float s_r[16];
  __shared__ float s_lv[16][16];
  __shared__ int s_lid[16][16];
  __shared__ float s_lr[16][16];
  __shared__ uint64_t s_key[kWave];     // the waves' K best as keys, wave w's at w K .. w K + K - 1
  __shared__ float s_kv[kWave];         // ... their values as read (the sign of a zero included)
  __shared__ float s_kr[kWave];
  __shared__ int s_sel[16];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  constexpr int S = kS;
  const int64_t row = blockIdx.x;
  const T* rowp = logits + row * row_stride;
  const int nch = (V + CH - 1) / CH;
  const int nfull = V / CH;
  const int c0 = (int)((int64_t)wave * nch / S);
  const int c1 = (int)((int64_t)(wave + 1) * nch / S);
  const int cfull = c1 < nfull ? c1 : nfull;

  WaveState s;
  s.acc = 0.0; s.r = kNoExp; s.mx = -INFINITY; s.thr = -INFINITY; s.thr_id = INT_MAX;
  s.lv = -INFINITY; s.lid = INT_MAX; s.lr = 0.f;

  int c = c0;
  if (kAligned) {
    const uint4* p4 = reinterpret_cast<const uint4*>(rowp);
    if (c + kUnroll <= cfull) {
      const uint4* lp = p4 + lane + (int64_t)c * (CH / VEC);   // chunk c of this lane
      uint4 q[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) q[u] = stream_load(lp + u * (CH / VEC));
      // the first group sets the reference exponent and the initial threshold
      float g = -INFINITY;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {   // unpacked twice: keeps the live registers to one chunk
        float x[VEC];
        unpack(q[u], x);
#pragma unroll
        for (int j = 0; j < VEC; ++j) g = fmaxf(g, x[j]);
      }
      s.mx = wave_max(g);
      s.r = ceilf(s.mx * kLog2eHi);
      int kp = 1;
      while (kp < K) kp <<= 1;
      const int grp = kWave / kp;           // lanes per group; kp groups
      float gm = g;
      for (int o = 1; o < grp; o <<= 1) gm = fmaxf(gm, __shfl_xor(gm, o));
      for (int o = grp; o < kWave; o <<= 1) gm = fminf(gm, __shfl_xor(gm, o));
      s.thr = gm;
      // a ring of kUnroll loads in flight: each chunk's slot (the first group's too) is refilled with the
      // load kUnroll chunks ahead as soon as its registers are unpacked, before its arithmetic
      for (; c + 2 * kUnroll <= cfull; c += kUnroll) {
        lp += kUnroll * (CH / VEC);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          float x[VEC];
          unpack(q[u], x);
          q[u] = stream_load(lp + u * (CH / VEC));
          chunk_full<VEC>(s, x, (c + u) * CH, K);
        }
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        float x[VEC];
        unpack(q[u], x);
        chunk_full<VEC>(s, x, (c + u) * CH, K);
      }
      c += kUnroll;
    }
    for (; c < cfull; ++c) {
      float x[VEC];
      unpack(stream_load(p4 + (c * CH + lane * VEC) / VEC), x);
      chunk_full<VEC>(s, x, c * CH, K);
    }
  }
  for (; c < c1; ++c) {   // unaligned rows, or the ragged last chunk of the row
    float x[VEC];
    const int e = c * CH + lane * VEC;
    unsigned ok;
    if (kAligned && e + VEC <= V) {         // a whole vector of this lane lies in the row
      unpack(stream_load(reinterpret_cast<const uint4*>(rowp + e)), x);
      ok = (1u << VEC) - 1u;
    } else {
      ok = load_guarded<T, VEC>(rowp, e, V, x);
    }
    chunk<VEC>(s, x, ok, c * CH, K);
  }

  // wave sum of the per-lane accumulators (fixed order: a DPP scan, the total in the last lane)
  const double acc = xp::rl_d(xp::wave_incl_scan(s.acc), kWave - 1);
  if (S > 1) {
    if (S * K <= kWave) {
      if (lane < K) {
        s_key[wave * K + lane] = order_key(s.lv, s.lid);
        s_kv[wave * K + lane] = s.lv;
        s_kr[wave * K + lane] = s.lr;
      }
    } else if (lane < 16) {
      s_lv[wave][lane] = s.lv; s_lid[wave][lane] = s.lid; s_lr[wave][lane] = s.lr;
    }
  }
  if (lane == 0) { s_acc[wave] = acc; s_r[wave] = s.r; }
  __syncthreads();
  if (wave != 0) return;

  if (S == 1) {
    // one wave per row: its list is the row's
  } else if (S * K <= kWave) {
    // every wave's K best, one per lane: a lane's rank among them is its slot in the merged list.  Real
    // entries have distinct keys (ids are distinct); the padding of a segment with fewer than K elements
    // shares one key below every real one.  Only slots below K are needed, and those hold real entries
    const int n = S * K;
    const bool has = lane < n;
    const uint64_t key = has ? s_key[lane] : 0ull;
    const uint32_t klo = (uint32_t)key, khi = (uint32_t)(key >> 32);
    int rank = 0;
#pragma unroll
    for (int j = 0; j < S * 16 && j < kWave; ++j) {
      if (j < n) {
        const uint64_t kj = ((uint64_t)(uint32_t)readlane_i((int)khi, j) << 32) | (uint32_t)readlane_i((int)klo, j);
        rank += kj > key ? 1 : 0;
      }
    }
    // the row holds at least K elements, so slots 0 .. K - 1 each receive exactly one lane; the first
    // store only keeps every slot a valid index
    if (lane < K) s_sel[lane] = lane;
    if (has && rank < K) s_sel[rank] = lane;
    if (lane < K) {
      const int src = s_sel[lane];
      s.lid = key_id(s_key[src]);
      s.lv = s_kv[src];
      s.lr = s_kr[src];
    }
  } else {
    for (int w = 1; w < S; ++w) {
      for (int k = 0; k < K; ++k) {
        const float v = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(s_lv[w][k])));
        const int id = __builtin_amdgcn_readfirstlane(s_lid[w][k]);
        const float rr = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(s_lr[w][k])));
        if (!before(v, id, s.thr, s.thr_id)) break;   // the rest of this sorted list cannot enter
        list_insert(s, v, id, rr, K);
      }
    }
  }
  float R = s_r[0];
#pragma unroll
  for (int w = 1; w < S; ++w) R = fmaxf(R, s_r[w]);
  double sum = 0.0;
#pragma unroll
  for (int w = 0; w < S; ++w) sum += ldexp(s_acc[w], (int)fmaxf(s_r[w] - R, -2000.f));
  double corr = 0.0;
  if (lane < K) {
    const double approx = ldexp((double)term(s.lv, s.lr), (int)fmaxf(s.lr - R, -2000.f));
    const double exact = exp2((double)s.lv * kLog2eD - (double)R);
    corr = exact - approx;
  }
  corr = xp::rl_d(xp::wave_incl_scan(corr), kWave - 1);
  const double lse = (double)R * kLn2D + log(sum + corr);
  if (lane < K) {
    const int64_t o = row * K + lane;
    out_ids[o] = s.lid;
    out_logit[o] = s.lv;
    if (out_lq) out_lq[o] = (float)((double)s.lv - lse);
  }
  if (lane == 0) out_lse[row] = lse;
}

template <typename T, bool A, int U, int S>
void launch_s(const ReduceArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL((reduce_topk_kernel<T, A, U, S>), dim3((unsigned)a.rows), dim3((unsigned)(kWave * S)), 0, stream,
                     static_cast<const T*>(a.logits), a.row_stride, a.V, a.K, a.ids, a.logit, a.lq, a.lse);
}

template <typename T, bool A, int U>
hipError_t launch_u(const ReduceArgs& a, hipStream_t stream) {
  switch (a.waves_per_row) {
    case 1: launch_s<T, A, U, 1>(a, stream); break;
    case 2: launch_s<T, A, U, 2>(a, stream); break;
    case 4: launch_s<T, A, U, 4>(a, stream); break;
    case 8: launch_s<T, A, U, 8>(a, stream); break;
    case 16: launch_s<T, A, U, 16>(a, stream); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, bool A>
hipError_t launch_t(const ReduceArgs& a, hipStream_t stream) {
  return a.unroll == 8 ? launch_u<T, A, 8>(a, stream) : launch_u<T, A, 4>(a, stream);
}

}  // namespace

// Launch shape.  The stream keeps HBM busy when about 32 MiB of loads are in
// flight across the chip (resident waves x loads per lane x 1 KiB), and a row
// split over fewer waves pays less for the start of each segment and for the
// final merge.  Large batches: one wave per row, 8 loads in flight for bf16
// (its kernel then holds 4 waves per SIMD, 4096 on the chip) and 4 for fp32
// (8 per SIMD).  Batches of at most 4096 rows: 8 loads in flight, and the
// fewest waves per row that still put 4096 waves on the chip at once.
ReduceShape reduce_default_shape(int64_t rows, int32_t V, caddtree_dtype_t dtype) {
  const int CH = kWave * (dtype == CADDTREE_BF16 ? 8 : 4);
  const int nch = (V + CH - 1) / CH;
  ReduceShape sh{1, 4};
  if (rows >= 8192) {
    sh.unroll = dtype == CADDTREE_BF16 ? 8 : 4;
  } else if (rows > 4096) {
    sh.unroll = 4;
  } else {
    sh.unroll = 8;
    while (sh.waves < 16 && rows * sh.waves * 2 <= 4096 && nch / (2 * sh.waves) >= 16) sh.waves *= 2;
  }
  return sh;
}

hipError_t launch_reduce_topk(const ReduceArgs& a, caddtree_dtype_t dtype, hipStream_t stream) {
  if (a.rows == 0) return hipSuccess;
  if (dtype == CADDTREE_BF16)
    return a.aligned ? launch_t<uint16_t, true>(a, stream) : launch_t<uint16_t, false>(a, stream);
  return a.aligned ? launch_t<float, true>(a, stream) : launch_t<float, false>(a, stream);
}

}  // namespace caddtree
