// Internal declarations shared by the libmtstep translation units (GPU path only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include <type_traits>

#include "../../include/mtstep.h"

namespace mt {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kWave = 64;
constexpr int kXcds = 8;
constexpr int kKMax = 16;  // largest supported beam
constexpr int kMaxEnsemble = 8;  // members of an ensemble
constexpr int kJointMax = 4;     // members of an ensemble whose vocabulary pass runs as one kernel

// ---------------------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------------------

// Workgroups are dispatched round-robin over the 8 XCDs (block w -> XCD w % 8).  This
// maps hardware block ids so that consecutive logical ids share an XCD (and its L2):
// logical ids [x*q, (x+1)*q) run on XCD x.  The ragged tail keeps its identity.
__device__ __forceinline__ int xcd_remap(int w, int G) {
  const int q = G / kXcds;
  if (w >= q * kXcds) return w;
  return (w % kXcds) * q + w / kXcds;
}

__device__ __forceinline__ float exp_fast(float x) {  // e^x via the hardware exp2
  return __builtin_amdgcn_exp2f(x * 1.4426950408889634f);
}
__device__ __forceinline__ float rcp_fast(float x) { return __builtin_amdgcn_rcpf(x); }
// tanh x = 1 - 2 / (e^{2x} + 1): saturates correctly at both ends (e^{2x} -> inf or 0)
__device__ __forceinline__ float tanh_fast(float x) {
  const float e = __builtin_amdgcn_exp2f(x * 2.8853900817779268f);
  return 1.0f - 2.0f * rcp_fast(e + 1.0f);
}
__device__ __forceinline__ float sigmoid_fast(float x) { return rcp_fast(1.0f + exp_fast(-x)); }

// Wave-wide sum and maximum, the result in every lane; every lane of the wave must be active.
// Within each 16-lane row, DPP moves (quad exchanges, then row rotations by 4 and 8) leave
// lanes 0, 16, 32 and 48 with their row totals (a fixed order of operations); the four are
// read into scalars and combined as (r0 + r1) + (r2 + r3).  Lane exchanges through LDS
// permutes, as a shuffle butterfly compiles to, cost a round trip of the LDS unit per step.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float lane_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
constexpr int kDppQuadSwap1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kDppQuadSwap2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kDppRowRor4 = 0x124;
constexpr int kDppRowRor8 = 0x128;
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_mov<kDppQuadSwap1>(v);
  v += dpp_mov<kDppQuadSwap2>(v);
  v += dpp_mov<kDppRowRor4>(v);
  v += dpp_mov<kDppRowRor8>(v);
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}
// Inclusive prefix sum over the 64 lanes of a wave (every lane active): within each 16-lane
// row by DPP row shifts of 1, 2, 4 and 8 (lanes shifted in from outside the row add 0), then
// across rows by the row broadcasts of lane 15 (to rows 1 and 3) and lane 31 (to rows 2 and 3).
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15 -> rows 1, 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31 -> rows 2, 3
  return v;
}
// Integer minimum / maximum over the wave (every lane active), the same DPP pattern
template <typename I, bool MAX>
__device__ __forceinline__ I wave_ext(I v) {
  auto pick = [](I x, I y) { return MAX ? (x > y ? x : y) : (x < y ? x : y); };
  auto mov = [](I x, auto ctrl) {
    return (I)__builtin_amdgcn_mov_dpp((int)x, decltype(ctrl)::value, 0xF, 0xF, false);
  };
  v = pick(v, mov(v, std::integral_constant<int, kDppQuadSwap1>()));
  v = pick(v, mov(v, std::integral_constant<int, kDppQuadSwap2>()));
  v = pick(v, mov(v, std::integral_constant<int, kDppRowRor4>()));
  v = pick(v, mov(v, std::integral_constant<int, kDppRowRor8>()));
  const I r0 = (I)__builtin_amdgcn_readlane((int)v, 0), r1 = (I)__builtin_amdgcn_readlane((int)v, 16);
  const I r2 = (I)__builtin_amdgcn_readlane((int)v, 32), r3 = (I)__builtin_amdgcn_readlane((int)v, 48);
  return pick(pick(r0, r1), pick(r2, r3));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_mov<kDppQuadSwap1>(v));
  v = fmaxf(v, dpp_mov<kDppQuadSwap2>(v));
  v = fmaxf(v, dpp_mov<kDppRowRor4>(v));
  v = fmaxf(v, dpp_mov<kDppRowRor8>(v));
  return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}

// Host-side fp32 -> bf16 bits, round to nearest with ties to even (the weight packing of every
// bf16 model uses it): a NaN stays a quiet NaN (its payload's top bits kept, the quiet bit set),
// +-inf stay infinite, values that round past the largest finite bf16 become +-inf.
inline uint16_t bf16_rne_bits(float f) {
  uint32_t u;
  __builtin_memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// bf16 <-> fp32, round to nearest even (NaN kept quiet)
__device__ __forceinline__ bf16 to_bf16(float f) { return (bf16)f; }
__device__ __forceinline__ float to_f32(bf16 h) { return (float)h; }
__device__ __forceinline__ float to_f32(float f) { return f; }

template <typename T>
struct Store;
template <>
struct Store<float> {
  __device__ __forceinline__ static void put(float *p, float v) { *p = v; }
};
template <>
struct Store<bf16> {
  __device__ __forceinline__ static void put(bf16 *p, float v) { *p = to_bf16(v); }
};

// total order used at every level of the beam selection:
// larger key first; equal keys -> smaller flat index first
__device__ __forceinline__ bool better(float ka, int ia, float kb, int ib) {
  return ka > kb || (ka == kb && ia < ib);
}

// Sorted (by `better`) list of the best KMAX (key, idx) pairs in registers, static indexing
template <int KMAX>
struct List {
  float v[KMAX];
  int i[KMAX];
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int p = 0; p < KMAX; ++p) { v[p] = -INFINITY; i[p] = 0x7fffffff; }
  }
  __device__ __forceinline__ void push(float x, int xi) {
    if (!better(x, xi, v[KMAX - 1], i[KMAX - 1])) return;
    float cv = x;
    int ci = xi;
#pragma unroll
    for (int p = 0; p < KMAX; ++p) {
      const bool sw = better(cv, ci, v[p], i[p]);
      const float tv = sw ? v[p] : cv;
      const int ti = sw ? i[p] : ci;
      v[p] = sw ? cv : v[p];
      i[p] = sw ? ci : i[p];
      cv = tv;
      ci = ti;
    }
  }
  __device__ __forceinline__ void pop() {
#pragma unroll
    for (int p = 0; p + 1 < KMAX; ++p) { v[p] = v[p + 1]; i[p] = i[p + 1]; }
    v[KMAX - 1] = -INFINITY;
    i[KMAX - 1] = 0x7fffffff;
  }
};

// Repeatedly extracts the block-wide best head of the per-thread sorted lists; the
// winner pops its head.  Writes n <= KMAX results (key bits, idx) through `emit`, called by
// threads 0..n-1 once the extraction is over (the results wait in LDS meanwhile).
template <int KMAX, typename Emit>
__device__ __forceinline__ void block_extract(List<KMAX> &L, int n, Emit emit) {
  __shared__ float wv[4];
  __shared__ int wi[4];
  __shared__ float rv[KMAX];
  __shared__ int ri[KMAX];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  for (int r = 0; r < n; ++r) {
    float bv = L.v[0];
    int bi = L.i[0];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    if (lane == 0) { wv[wave] = bv; wi[wave] = bi; }
    __syncthreads();
    bv = wv[0];
    bi = wi[0];
#pragma unroll
    for (int w = 1; w < 4; ++w)
      if (better(wv[w], wi[w], bv, bi)) { bv = wv[w]; bi = wi[w]; }
    __syncthreads();
    if (L.i[0] == bi && L.v[0] == bv) L.pop();
    if (t == 0) {
      rv[r] = bv;
      ri[r] = bi;
    }
  }
  __syncthreads();
  if (t < n) emit(t, rv[t], ri[t]);
}

// The same extraction by one wave: result r is kept by lane r, which calls emit(r, key, idx)
// once the n results are known.  Indices must be distinct.
template <int KMAX, typename Emit>
__device__ __forceinline__ void wave_extract(List<KMAX> &L, int n, Emit emit) {
  const int lane = threadIdx.x & 63;
  float mv = -INFINITY;
  int mi = 0x7fffffff;
  for (int r = 0; r < n; ++r) {
    float bv = L.v[0];
    int bi = L.i[0];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oi = __shfl_xor(bi, o, 64);
      if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    if (L.i[0] == bi && L.v[0] == bv) L.pop();
    if (lane == r) { mv = bv; mi = bi; }
  }
  if (lane < n) emit(lane, mv, mi);
}

// ---- exact selection by bisection over order-preserving key codes ----
// code(f) is a uint32 that orders like the float (-0 counts as +0); 0 marks "no entry".
__device__ __forceinline__ uint32_t key_code(float f) {
  uint32_t b = __float_as_uint(f);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float key_from_code(uint32_t u) {
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u);
}

// Wave-wide counts over R register slots per lane, of which the first rs (wave-uniform) are
// in use.  Ballots and scalar popcounts only: no cross-lane data movement.
template <int R>
__device__ __forceinline__ int wave_count_ge(const uint32_t (&u)[R], int rs, uint32_t t) {
  int c = 0;
#pragma unroll
  for (int s = 0; s < R; ++s)
    if (s < rs) c += __popcll(__ballot(u[s] >= t));
  return c;
}
template <int R>
__device__ __forceinline__ int wave_count_eq_le(const uint32_t (&u)[R], const int (&ix)[R], int rs, uint32_t t,
                                                int i) {
  int c = 0;
#pragma unroll
  for (int s = 0; s < R; ++s)
    if (s < rs) c += __popcll(__ballot(u[s] == t && ix[s] <= i));
  return c;
}

// Largest t with count(code >= t) >= K over the wave's entries (codes >= 1), given
// count(code >= 1) >= K.  Binary search between the smallest and largest code present.
template <int R>
__device__ __forceinline__ uint32_t wave_kth_code(const uint32_t (&u)[R], int rs, int K) {
  uint32_t lo = 0xffffffffu, hi = 0u;
#pragma unroll
  for (int s = 0; s < R; ++s)
    if (s < rs && u[s] != 0u) {
      lo = u[s] < lo ? u[s] : lo;
      hi = u[s] > hi ? u[s] : hi;
    }
  lo = wave_ext<uint32_t, false>(lo);
  hi = wave_ext<uint32_t, true>(hi);
  while (lo < hi) {  // invariant: count(>= lo) >= K, count(>= hi + 1) < K
    const uint32_t mid = lo + (uint32_t)(((uint64_t)hi - lo + 1u) >> 1);
    if (wave_count_ge<R>(u, rs, mid) >= K)
      lo = mid;
    else
      hi = mid - 1u;
  }
  return lo;
}

// Exact top-K of the wave's entries (code u, index ix; u == 0 = empty slot) under the order
// "larger key first, equal keys -> smaller index first".  Indices must be distinct.  The
// selected entries are compacted into scratch (>= K slots, wave-private LDS); lane j < n_sel
// (n_sel = min(K, entries)) then calls emit(rank, key, idx) for the j-th of them, with its
// rank 0..n_sel-1 in that order.  Returns n_sel (wave-uniform).
template <int R, typename Emit>
__device__ __forceinline__ int wave_topk(const uint32_t (&u)[R], const int (&ix)[R], int rs, int K,
                                         uint32_t *su, int *si, Emit emit) {
  const int lane = threadIdx.x & 63;
  const int n = wave_count_ge<R>(u, rs, 1u);
  uint32_t tau = 1u;
  int iota = 0x7fffffff;
  if (n > K) {
    // The cut: the bisection of wave_kth_code, stopped as soon as a midpoint has exactly K
    // entries at or above it (then those K are the selection; with distinct keys that takes
    // about log2 of the entry count steps instead of one per bit of the codes' spread).
    // Otherwise it runs to the K-th largest code and the ties there are resolved below.
    uint32_t lo = 0xffffffffu, hi = 0u;
#pragma unroll
    for (int s = 0; s < R; ++s)
      if (s < rs && u[s] != 0u) {
        lo = u[s] < lo ? u[s] : lo;
        hi = u[s] > hi ? u[s] : hi;
      }
    lo = wave_ext<uint32_t, false>(lo);
    hi = wave_ext<uint32_t, true>(hi);
    bool exact = false;
    while (lo < hi) {  // invariant: count(>= lo) >= K, count(>= hi + 1) < K
      const uint32_t mid = lo + (uint32_t)(((uint64_t)hi - lo + 1u) >> 1);
      const int c = wave_count_ge<R>(u, rs, mid);
      if (c == K) {
        lo = mid;
        exact = true;
        break;
      }
      if (c > K)
        lo = mid;
      else
        hi = mid - 1u;
    }
    tau = lo;
    const int gt = exact ? K : tau == 0xffffffffu ? 0 : wave_count_ge<R>(u, rs, tau + 1u);
    const int need = K - gt;
    const int eq = exact ? 0 : wave_count_eq_le<R>(u, ix, rs, tau, 0x7fffffff);
    if (eq > need) {  // ties at the cut: keep the `need` smallest indices among them
      int lo = 0x7fffffff, hi = (int)0x80000000;
#pragma unroll
      for (int s = 0; s < R; ++s)
        if (s < rs && u[s] == tau) {
          lo = ix[s] < lo ? ix[s] : lo;
          hi = ix[s] > hi ? ix[s] : hi;
        }
      lo = wave_ext<int, false>(lo);
      hi = wave_ext<int, true>(hi);
      while (lo < hi) {  // smallest i with count(code == tau, idx <= i) >= need
        const int mid = (int)(((int64_t)lo + hi) >> 1);
        if (wave_count_eq_le<R>(u, ix, rs, tau, mid) >= need)
          hi = mid;
        else
          lo = mid + 1;
      }
      iota = lo;
    }
  }
  // compact the selected entries into scratch
  int base = 0;
#pragma unroll
  for (int s = 0; s < R; ++s) {
    if (s >= rs) break;
    const bool sel = u[s] != 0u && (u[s] > tau || (u[s] == tau && ix[s] <= iota));
    const uint64_t bal = __ballot(sel);
    const int pos = base + __popcll(bal & ((1ull << lane) - 1ull));
    if (sel && pos < K) {  // more than K only if indices repeat, which callers exclude
      su[pos] = u[s];
      si[pos] = ix[s];
    }
    base += __popcll(bal);
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  const int ns = base < K ? base : K;
  // lane j < ns holds selected entry j; each counts the entries that beat it, read from the
  // other lanes' registers (one LDS read per lane, then lane reads)
  uint32_t mu = 0u;
  int mi = 0;
  if (lane < ns) {
    mu = su[lane];
    mi = si[lane];
  }
  int rank = 0;
  for (int j = 0; j < ns; ++j) {
    const uint32_t ou = (uint32_t)__builtin_amdgcn_readlane((int)mu, j);
    const int oi = __builtin_amdgcn_readlane(mi, j);
    rank += (ou > mu || (ou == mu && oi < mi)) ? 1 : 0;
  }
  if (lane < ns) emit(rank, key_from_code(mu), mi);
  return ns;
}

// The same selection by K rounds of a wave maximum (for small K): each round takes the best
// remaining entry (DPP maxima of the lanes' best codes, then of their indices among equal
// codes) and its owner clears it, so the entries come out in rank order and nothing is
// counted.  Lane j < n_sel writes entry j to scratch (su, si) and calls emit(j, key, idx).
// Returns n_sel = min(K, entries) (wave-uniform).  Indices must be distinct.
template <int R, typename Emit>
__device__ __forceinline__ int wave_topk_rounds(uint32_t (&u)[R], const int (&ix)[R], int rs, int K,
                                                uint32_t *su, int *si, Emit emit) {
  const int lane = threadIdx.x & 63;
  uint32_t my_u = 0u;
  int my_i = 0x7fffffff;
  int ns = 0;
  for (int r = 0; r < K; ++r) {
    uint32_t bu = 0u;
    int bi = 0x7fffffff;
#pragma unroll
    for (int s = 0; s < R; ++s)
      if (s < rs && (u[s] > bu || (u[s] == bu && ix[s] < bi))) {
        bu = u[s];
        bi = ix[s];
      }
    const uint32_t mu = wave_ext<uint32_t, true>(bu);
    if (mu == 0u) break;  // no entries left (wave-uniform)
    const int mi = wave_ext<int, false>(bu == mu ? bi : 0x7fffffff);
#pragma unroll
    for (int s = 0; s < R; ++s)
      if (u[s] == mu && ix[s] == mi) u[s] = 0u;
    if (lane == r) {
      my_u = mu;
      my_i = mi;
    }
    ns = r + 1;
  }
  if (lane < ns) {
    su[lane] = my_u;
    si[lane] = my_i;
    emit(lane, key_from_code(my_u), my_i);
  }
  return ns;
}

// K best of a wave's entries by whichever form is cheaper: K rounds of a wave maximum for
// K <= 6, the bisection above that (at K = 12 the rounds cost 3 us more per selection, at
// K = 5 they save 1 us; kernel traces of the beam selection).
constexpr int kRoundsMaxK = 6;
template <int R, typename Emit>
__device__ __forceinline__ int wave_select(uint32_t (&u)[R], const int (&ix)[R], int rs, int K, uint32_t *su,
                                           int *si, Emit emit) {
  if (K <= kRoundsMaxK) return wave_topk_rounds<R>(u, ix, rs, K, su, si, emit);
  return wave_topk<R>(u, ix, rs, K, su, si, emit);
}

// ---- row-level pieces shared by the log-sum-exp pass and the beam selection ----

// Log-sum-exp of one row from its per-chunk partials (m_c, s_c), s_c = sum of exp(logit - m_c)
// over chunk c: L = M + ln sum_c s_c exp(m_c - M), M = max_c m_c.  Computed by one wave with a
// fixed order of operations: lane l folds partials l, l + 64, l + 128, ... in that order, then
// the lanes are combined by wave_max and wave_sum.  Every caller obtains the same bits from the
// same partials, whether it reads them through a pointer or holds them in registers (partial
// lane + 64 j in pq[j]).  Every lane of the wave must be active.
template <int NP>
__device__ __forceinline__ float wave_row_lse_regs(const float2 (&pq)[NP], int ntiles) {
  const int lane = threadIdx.x & 63;
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < NP; ++j)
    if (lane + 64 * j < ntiles) mx = fmaxf(mx, pq[j].x);
  mx = wave_max(mx);
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NP; ++j)
    if (lane + 64 * j < ntiles) s += pq[j].y * exp_fast(pq[j].x - mx);
  s = wave_sum(s);
  return mx + __builtin_amdgcn_logf(s) * 0.6931471805599453f;
}
__device__ __forceinline__ float wave_row_lse(const float2 *pr, int ntiles) {
  const int lane = threadIdx.x & 63;
  float mx = -INFINITY;
  for (int i = lane; i < ntiles; i += 64) mx = fmaxf(mx, pr[i].x);
  mx = wave_max(mx);
  float s = 0.f;
  for (int i = lane; i < ntiles; i += 64) {
    const float2 q = pr[i];
    s += q.y * exp_fast(q.x - mx);
  }
  s = wave_sum(s);
  return mx + __builtin_amdgcn_logf(s) * 0.6931471805599453f;
}
// The same value in every thread of a workgroup (its first wave computes it)
__device__ __forceinline__ float block_row_lse(const float2 *pr, int ntiles) {
  __shared__ float sl;
  if (threadIdx.x < 64) {
    const float L = wave_row_lse(pr, ntiles);
    if (threadIdx.x == 0) sl = L;
  }
  __syncthreads();
  const float L = sl;
  __syncthreads();  // sl may be rewritten by the caller's next call
  return L;
}

// The output projection as the exact recomputation reads it: packed Wo^T in MFMA fragment
// order (32-row vocabulary block vb, k-step ks of KV = 32 / sizeof(CT) k-values: 64 lanes x 16
// bytes at ((vb * KS + ks) * 64 + lane) * 16, lane l holding row vb*32 + l%32 and k-values
// ks*KV + (l/32)*KV/2 + j), the padded bias, and the readout activations t [M][E].
struct VocabView {
  const void *t;
  const void *wp;
  const float *bias;
  int V, E, KS;
};

// Exact keys prev + (logit - L) of row m over the whole vocabulary, recomputed from the weights
// into each lane's list: the waves w0, w0 + nw, ... of the caller take every nw-th 32-entry
// vocabulary block (lane pairs (l, l+32) of a wave share one vocabulary entry).
template <typename CT, int KMAX>
__device__ __forceinline__ void row_recompute_fill(const VocabView &vv, int m, float L, float prev, int w0, int nw,
                                                   List<KMAX> &lst) {
  constexpr int epv = 16 / (int)sizeof(CT);  // k-values per lane vector
  constexpr int KV = 2 * epv;
  const int lane = threadIdx.x & 63;
  const CT *trow = (const CT *)vv.t + (size_t)m * vv.E;
  const int nvb = (vv.V + 31) / 32;
  for (int vb = w0; vb < nvb; vb += nw) {
    float acc = 0.f;
    for (int ks = 0; ks < vv.KS; ++ks) {
      const CT *wv = (const CT *)((const char *)vv.wp + (((size_t)vb * vv.KS + ks) * 64 + lane) * 16);
      const int k0 = ks * KV + (lane >> 5) * epv;
#pragma unroll
      for (int j = 0; j < epv; ++j) acc += to_f32(wv[j]) * to_f32(trow[k0 + j]);
    }
    acc += __shfl_xor(acc, 32, 64);
    const int v = vb * 32 + (lane & 31);
    if (lane < 32 && v < vv.V) lst.push(prev + ((acc + vv.bias[v]) - L), v);
  }
}
// The K best of them by a 256-thread workgroup; emit(rank, key, token) for ranks 0..K-1
template <typename CT, int KMAX, typename Emit>
__device__ __forceinline__ void row_recompute(const VocabView &vv, int m, int K, float L, float prev, Emit emit) {
  List<KMAX> lst;
  lst.init();
  row_recompute_fill<CT, KMAX>(vv, m, L, prev, threadIdx.x >> 6, 4, lst);
  block_extract<KMAX>(lst, K, emit);
}

// Exact keys prev + sum_m w[m] * logit_m(v) of row m over the whole vocabulary (a joint
// ensemble's row), recomputed from the n members' weights, split over waves as above.
template <typename CT, int KMAX>
__device__ __forceinline__ void row_recompute_ens_fill(const VocabView *vvs, const float *w, int n, int m,
                                                       float prev, int w0, int nw, List<KMAX> &lst) {
  constexpr int epv = 16 / (int)sizeof(CT);
  constexpr int KV = 2 * epv;
  const int lane = threadIdx.x & 63;
  const int V = vvs[0].V;
  const int nvb = (V + 31) / 32;
  for (int vb = w0; vb < nvb; vb += nw) {
    const int v = vb * 32 + (lane & 31);
    float c = 0.f;
    for (int mm = 0; mm < n; ++mm) {
      const VocabView &vv = vvs[mm];
      const CT *trow = (const CT *)vv.t + (size_t)m * vv.E;
      float acc = 0.f;
      for (int ks = 0; ks < vv.KS; ++ks) {
        const CT *wq = (const CT *)((const char *)vv.wp + (((size_t)vb * vv.KS + ks) * 64 + lane) * 16);
        const int k0 = ks * KV + (lane >> 5) * epv;
#pragma unroll
        for (int j = 0; j < epv; ++j) acc += to_f32(wq[j]) * to_f32(trow[k0 + j]);
      }
      acc += __shfl_xor(acc, 32, 64);
      if (v < V) c += w[mm] * (acc + vv.bias[v]);
    }
    if (lane < 32 && v < V) lst.push(prev + c, v);
  }
}
template <typename CT, int KMAX, typename Emit>
__device__ __forceinline__ void row_recompute_ens(const VocabView *vvs, const float *w, int n, int m, int K,
                                                  float prev, Emit emit) {
  List<KMAX> lst;
  lst.init();
  row_recompute_ens_fill<CT, KMAX>(vvs, w, n, m, prev, threadIdx.x >> 6, 4, lst);
  block_extract<KMAX>(lst, K, emit);
}

// ---------------------------------------------------------------------------------------
// launchers (host side).  All return hipSuccess or the launch error.
// ---------------------------------------------------------------------------------------

// EPI_SCATTER: row m is stored at output row a_idx[m] (the rows it was gathered from)
enum Epilogue { EPI_STORE = 0, EPI_TANH = 1, EPI_SCATTER = 2 };

struct GemmProblem {
  const void *A;          // activations [rows][lda] (fp32 or bf16, see a_bf16)
  const int32_t *a_idx;   // optional gather: row m reads A row a_idx[m] (clamped to a_rows)
  int a_rows;             // rows available in A (for the gather clamp)
  int lda;                // elements
  int a_bf16;             // A element type: 0 fp32, 1 bf16
  const void *Bp;         // packed weights: fp32 [N_pad][ldb] K contiguous; bf16 MFMA fragment order
  int ldb;                // = K_pad (a multiple of 128 for bf16)
  const float *bias;      // [N] or NULL
  void *out;              // [M][ldc] (fp32, or bf16 if out_bf16)
  int ldc;
  int out_bf16;
  int M, N, K;
  int32_t *err;           // device error word (bit err_bit set on a clamped gather)
  int err_bit;
  int wblk;               // fp32 weights: column block width of their packing (16 or 32)
  const int *m_dev;       // optional: row count on the device (<= M); later rows are neither
                          // read nor stored, and tiles that start past it return at once
};

// gemm dtype: 0 fp32 MFMA, 1 bf16 MFMA.  nprob = 1 or 2 (problems share one launch).
hipError_t launch_gemm(int bf16_mma, const GemmProblem *probs, int nprob, Epilogue epi,
                       hipStream_t st);
// fp32 weight packing for an [K][N] product expected at about `rows` rows: 16 (16x16x4 form) or
// 32 (32x32x2 form), whichever the tile choice expects to run faster
int gemm_f32_weight_block(long rows, long N, long K);

// ---- vocabulary projection with fused log-sum-exp partials and beam candidates ----
// hypothesis rows per workgroup (0 if E is too large for the LDS-resident activations)
int vocab_rows_per_block(int bf16_mma, int E);
// vocabulary chunks (one workgroup per chunk and row block; per-chunk outputs)
int vocab_chunks(int bf16_mma, int M, int V, int E, int num_cu);
int vocab_sample_size(int V);  // vocabulary entries of the threshold pass (padded)
int vocab_lists();             // candidate buffers per (row, chunk)
size_t vocab_pack_bytes(int bf16_mma, int V, int E);
// packs Wo^T rows into MFMA fragment order; src is Wo [E][V] or, if src_is_emb, emb [V][E]
void vocab_pack_host(int bf16_mma, int V, int E, const float *src, int src_is_emb, void *out);
// thr[m] = a value reached by K of sample[m][0 .. min(V, S)) (the K-th largest of 64 lane maxima),
// minus a rounding margin, S = vocab_sample_size(V);
// sample [M][S] holds the logits of the first S vocabulary entries (computed by launch_gemm)
// Block 0 also clears the B sentence arrival counters scnt of the following beam selection.
// A fused ensemble's last member takes it over its combined values instead: w * sample[m][v],
// plus comb[m][v] (comb [M][V], the earlier members' weighted logits) if comb is not NULL.
hipError_t launch_vocab_threshold(int M, int V, int K, const float *sample, float *thr, int *scnt, int B,
                                  hipStream_t st, const float *comb = nullptr, float w = 1.f);
// part [M][n_chunks] (reference m, sum exp(l - m)); every logit >= thr[m] goes to cbuf
// [M][cap][n_chunks * lists] (entry-major per row) with counts in ccnt [M][n_chunks][lists] (a count above cap marks
// an overflowed list); logits [M][V] or NULL.  fixed_ref: the caller has proven every logit
// lies in [-40, 40], so the reference is 0 and no running maximum is kept.
// logits_w, logits_acc: the logits are stored multiplied by logits_w, and added to the values
// already in logits when logits_acc (the members of a fused ensemble).  cap_stored (with
// logits): the candidates are the stored values rather than the logits (the last member).
// thr NULL: no candidates (the partials are still written).
hipError_t launch_vocab(int bf16_mma, const void *t, const void *wp, const float *bias_pad, int M, int V,
                        int E, int n_chunks, const float *thr, float2 *part, int2 *cbuf, int *ccnt, int cap,
                        float *logits, int fixed_ref, hipStream_t st, float logits_w = 1.f, int logits_acc = 0,
                        int cap_stored = 0);

// Fused ensemble: per row m, C[m] = sum_i w[i] * LSE_i[m] (LSE_i merged from member i's partials
// part[i] [M][ntiles[i]] exactly as the beam selection merges a row's), prev_adj[m] =
// prev[m] - C[m], and row_const[m] = C[m] if given.
struct EnsembleConst {
  int n;
  const float2 *part[kMaxEnsemble];
  int ntiles[kMaxEnsemble];
  float w[kMaxEnsemble];
  const float *prev;
  float *prev_adj;
  float *row_const;
};
hipError_t launch_ensemble_const(const EnsembleConst &a, int M, hipStream_t st);

// ---- fused ensemble: one vocabulary pass for 2..kJointMax members (same V, E and type) ----
// hypothesis rows per workgroup of the joint pass (0: not supported for this E, type and n)
int vocab_joint_rows(int bf16_mma, int E, int n);
// vocabulary chunks of the joint pass (<= vocab_chunks of the same model: its workspace holds them)
int vocab_joint_chunks(int bf16_mma, int M, int V, int E, int n, int num_cu);
struct VocabJoint {
  int n, bf16_mma, M, V, E, n_chunks, cap, fixed_ref;
  const void *t[kJointMax];      // [M][E] readout activations per member
  const void *wp[kJointMax];     // packed Wo^T per member (vocab_pack_host layout)
  const float *bias[kJointMax];  // padded output bias per member
  float w[kJointMax];
  float2 *part[kJointMax];       // [M][n_chunks] per member
  const float *thr;              // [M] threshold on the combined value
  int2 *cbuf;                    // [M][cap][n_chunks * lists]: combined values >= thr
  int *ccnt;                     // [M][n_chunks][lists]
};
hipError_t launch_vocab_joint(const VocabJoint &j, hipStream_t st);
// combined sample values sum_m w[m] * sample[m][row * ld + v] for the joint threshold
struct VocabJointSample {
  int n, ld;
  const float *sample[kJointMax];
  float w[kJointMax];
};
hipError_t launch_vocab_joint_threshold(int M, int V, int K, const VocabJointSample &smp, float *thr, int *scnt,
                                        int B, hipStream_t st);
constexpr int kVocabCap = 32;  // candidate buffer entries per (row, chunk, list)
constexpr int kVocabPad = 64;  // vocabulary rows are padded to a multiple of this

// GRU cell for M rows; a row m = aidx[m] (if given), previous state row hidx[m] (if given);
// out-of-range indices are clamped and flagged in err (bit 0: aidx, bit 1: hidx); out16 (if
// given) receives a bf16 copy [M][H] of the new state.  Layer norm: ga..bu all given, both
// paths; ga = ba = NULL with gu, bu given, the recurrent path only (a transition block, whose
// input path is its bias row, passed as a with lda = 0)
hipError_t launch_gru_cell(int M, int H, const float *a, int lda, const int32_t *aidx, int arows,
                           const float *u, int ldu, const float *hsrc, const int32_t *hidx, int hrows,
                           int32_t *err, const float *ga, const float *ba, const float *gu, const float *bu,
                           float eps, float *out, int ldo, bf16 *out16, float *tap, hipStream_t st);

// Element offsets from one cell's operands to a second cell of the same shape and options
// run by the same launch (the two directions of an encoder position): a, u, previous state,
// output, bf16 copy, keep and the layer-norm vectors (one offset for all four).
struct CellPair {
  long long da, du, dh, dout, d16, dkeep, dln;
};

// the same with row strides for the previous state (ldh; hsrc NULL: zero state) and the bf16
// copy (ld16), and keep (if given): a row m whose keep[m * keep_ld] is 0 carries its previous
// state over instead of updating.  pair (if given): a second cell at those offsets, run by
// the same launch.
hipError_t launch_gru_cell_ex(int M, int H, const float *a, int lda, const int32_t *aidx, int arows,
                              const float *u, int ldu, const float *hsrc, int ldh, const int32_t *hidx, int hrows,
                              int32_t *err, const float *ga, const float *ba, const float *gu, const float *bu,
                              float eps, float *out, int ldo, bf16 *out16, int ld16, float *tap,
                              const float *keep, int keep_ld, hipStream_t st, const CellPair *pair = nullptr);
hipError_t launch_fill_zero(float *p, long long n, hipStream_t st);

hipError_t launch_readout(int M, int E, const float *p1, int ld1, const float *p2, int ld2, const int32_t *idx2,
                          int rows2, const float *p3, int ld3, const float *bt, const float *g,
                          const float *be, float eps, void *t_out, int t_bf16, float *tap,
                          hipStream_t st);

hipError_t launch_masked_mean(int B, int S, int Cd, const void *ctx, int ctx_bf16,
                              const float *mask, float *out, hipStream_t st);
// rows of a [n] 0/1 mask that are valid (nonzero), in increasing order: idx[0..*count)
hipError_t launch_valid_rows(int n, const float *mask, int32_t *idx, int *count, hipStream_t st);

// context rows go to ctx_out [M][ldc] fp32 and/or ctx16 [M][ld16] bf16 (either may be NULL);
// srank (or NULL): the sentences by decreasing length, from launch_attention_order, which only
// decides the order in which rows are scheduled
hipError_t launch_attention(int B, int K, int S, int A, int Cd, const void *P, const void *Cx,
                            int bf16_io, const float *mask, const float *q, int ldq,
                            const float *va, float *ctx_out, int ldc, bf16 *ctx16, int ld16, float *alpha_out,
                            const int *srank, hipStream_t st);
// srank[0..B) = the sentences of mask [B][S] by decreasing number of valid positions
// (B <= attention_order_max_sentences())
hipError_t launch_attention_order(int B, int S, const float *mask, int *srank, hipStream_t st);
int attention_order_max_sentences();

// translation bookkeeping for B sentences of K ranked results each (see mt_beam_finish)
struct BeamFinish {
  int K, step, eos, final;
  float alpha;
  int32_t *tok, *bp, *row;
  float *score;
  int32_t *beam, *fin_count;
  int32_t *hist_tok, *hist_bp;  // this step's [M] record
  float *fin_score, *fin_norm;  // [B][K]
  int32_t *fin_step, *fin_parent, *fin_tok;
};
hipError_t launch_beam_finish(const BeamFinish &a, int B, hipStream_t st);
struct BeamNbest {
  int K, steps, ld_hist, ld_seq;
  const int32_t *hist_tok, *hist_bp;  // [steps][ld_hist]
  const int32_t *fin_count;           // [B]
  const float *fin_norm;              // [B][K]
  const int32_t *fin_step, *fin_parent, *fin_tok;
  int32_t *order;                     // [B][K]
  int32_t *seq;                       // [B*K][ld_seq]
};
hipError_t launch_beam_nbest(const BeamNbest &a, int B, hipStream_t st);

// ensemble combination out[i] = sum_j w[j] * in[j][i] over count elements (16-byte aligned
// buffers; out may be one of the inputs); 1 <= n <= kMaxEnsemble
hipError_t launch_ensemble(int n, const float *const *in, const float *w, long long count, float *out,
                           int num_cu, hipStream_t st);

hipError_t launch_lse(int M, int ntiles, const float2 *part, float *lse, float *logits, int V,
                      hipStream_t st);

// Beam selection, one workgroup per row m = b*K + k.  Candidates are (value, token) pairs stored
// as int2 {float bits, token} in nl lists of up to cap entries per row: cbuf [M][cap][nl]
// (entry q of every list of a row contiguous) with fill counts cnt [M][nl] (NULL: every list
// holds cap entries).
//  * part != NULL (candidates from the vocabulary pass): values are logits; the row's
//    log-sum-exp is merged from part [M][ntiles] and keys are prev_score + (logit - lse).  A
//    row whose candidates do not fit (a list count above cap, more than the row can stage,
//    or fewer than K) is recomputed exactly from vv (bf16_mma gives its compute dtype).
//  * part == NULL: values are keys (the logp path).
// The row's K best go to row_cand [M][K].  The last row of sentence b to finish (counted in
// scnt[b], which must be 0 before the first use and is left at 0) merges the sentence's K x K
// row results into score/tok/bp/row_out [B][K].
struct RowSelect {
  int B, K, V, nl, cap;
  const int *cnt;
  const int2 *cbuf;
  const float2 *part;
  int ntiles;
  const float *prev_score;
  VocabView vv;
  int bf16_mma;
  int2 *row_cand;
  int *scnt;
  float *score_out;
  int32_t *tok_out, *bp_out, *row_out;
  unsigned long long *nrecompute;  // optional: counts the rows recomputed exactly
  // A fused ensemble's combined values [M][V] (or NULL).  With it the candidates are combined
  // values c, their keys prev_score + c (no log-sum-exp: part is NULL and prev_score already
  // holds the row constant), and a row whose lists overflow is selected from its stored row.
  const float *comb;
  // A joint ensemble pass (nens > 0, comb NULL): the same keys, and a row whose lists overflow
  // is recomputed from the members' weights, sum_m ew[m] * (logit_m), with evv[m] each
  // member's view (all of type CT)
  int nens;
  VocabView evv[kJointMax];
  float ew[kJointMax];
};
hipError_t launch_row_select(const RowSelect &a, hipStream_t st);
// Chunks of one row of a materialised logp for the first selection level (both the workspace
// layout and the launch take them from here).
void topk_scan_shape(int M, int V, int *chunk, int *nchunks);
// Block (0, 0) also clears the B sentence arrival counters scnt.
hipError_t launch_topk_scan_logp(int M, int K, int V, int nchunks, const float *prev_score,
                                 const float *logp, int2 *cand_out, int *scnt, int B, hipStream_t st);

}  // namespace mt
