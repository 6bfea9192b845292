// Beam selection: the best K of the K x V extensions of each sentence.
//
// Total order at every level: larger key first, ties -> smaller index (the token within a
// row, the flat index k*V + v within a sentence).  Keys are fp32: key = prev_score +
// (logit - lse), summed in that order, which is exactly how a materialised
// log-probability (logit - lse) plus the score rounds.  Levels:
//   1. candidates per row: every logit at or above the row's threshold, collected by the
//      vocabulary kernel into per-(row, chunk, lane) lists; or, for a materialised logp, the
//      K best keys of each chunk of the row (topk_scan_logp);
//   2. per row (row_select): the K best keys among the row's candidates;
//   3. per sentence (by the last of its rows to finish row selection): the K best of the K
//      rows' K candidates.
// Levels 2 and 3 select exactly by bisection over order-preserving integer codes of the
// keys (wave_topk): every count is a ballot plus a scalar popcount, ties at the cut are
// resolved by a second bisection over the indices, and the K survivors are ranked by
// pairwise comparison.  Nothing is sorted and no step depends on a cross-lane exchange
// chain longer than one min/max reduction.
#include "mt_internal.h"

#include <algorithm>
#include <type_traits>

namespace mt {

constexpr int kTT = 256;
constexpr int kRowCap = 4096;          // candidates one row can stage in LDS
constexpr int kSlots = kRowCap / 256;  // register slots per lane when a wave takes a quarter
constexpr int kSpec = 4;               // list entries requested with the counts

// Row results cross workgroups (and XCDs, whose L2 caches are not coherent with each other)
// on their way to the sentence merge.  They are written and read with device-scope atomic
// accesses, which are coherent without the full L2 write-back a device-scope release fence
// costs; each writer waits for its stores to complete before its workgroup is counted in.
__device__ __forceinline__ void put_row(int2 *p, float key, int tok) {
  const unsigned long long v = (unsigned long long)(uint32_t)__float_as_int(key) |
                               ((unsigned long long)(uint32_t)tok << 32);
  __hip_atomic_store((unsigned long long *)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int2 get_row(const int2 *p) {
  const unsigned long long v =
      __hip_atomic_load((const unsigned long long *)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_int2((int)(uint32_t)v, (int)(uint32_t)(v >> 32));
}

// Level 3 for one sentence: the K best of the K x K row results, held as a table of (key code,
// flat index) with candidate (k, j) at k*K + j and flat index k*V + token; entries without a
// token have code 0 and distinct indices above every real one.  The order: larger key code
// first, equal codes by smaller flat index; ranks past the real entries (fewer than K) are dead
// slots: hypothesis 0 continued with score -inf.  Two forms, chosen by the table's size:
// sentence_rank (K*K <= 64), in which every entry counts the entries that beat it (16-byte LDS
// reads of a table padded to whole groups of four with entries that beat nothing), so the
// counts are a permutation and the K entries below K write themselves to their rank; and
// sentence_select_wave (larger tables), one wave's exact selection by bisection (wave_topk),
// whose cost grows with the slots per lane, not with the table's square.
constexpr int kRankMax = 64;  // tables up to this size are ranked by counting
__device__ __forceinline__ void sentence_rank(const RowSelect &a, int b, const uint32_t *su, const int *si) {
  const int t = threadIdx.x, K = a.K, V = a.V;
  const int n = K * K;
  const int n4 = (n + 3) / 4;
  if (t >= n) return;
  const uint32_t mu = su[t];
  const int mi = si[t];
  // the candidates are read four at a time, four groups per iteration (16-byte LDS reads, issued
  // together: read one by one, every iteration waited out the LDS latency)
  const uint4 *su4 = (const uint4 *)su;
  const int4 *si4 = (const int4 *)si;
  auto beats = [&](uint32_t ou, int oi) { return (ou > mu || (ou == mu && oi < mi)) ? 1 : 0; };
  int rank = 0;
#pragma unroll 4
  for (int j = 0; j < n4; ++j) {
    const uint4 u = su4[j];
    const int4 x = si4[j];
    rank += beats(u.x, x.x) + beats(u.y, x.y) + beats(u.z, x.z) + beats(u.w, x.w);
  }
  if (rank >= K) return;
  const int o = b * K + rank;
  if (mu != 0u) {
    a.score_out[o] = key_from_code(mu);
    a.tok_out[o] = mi % V;
    a.bp_out[o] = mi / V;
    if (a.row_out) a.row_out[o] = b * K + mi / V;
  } else {
    a.score_out[o] = -INFINITY;
    a.tok_out[o] = 0;
    a.bp_out[o] = 0;
    if (a.row_out) a.row_out[o] = b * K;
  }
}

// One wave (every lane active): the table's K*K <= 256 entries in four register slots, entries
// without a token empty; qu/qi: K entries of wave-private LDS scratch.
__device__ __forceinline__ void sentence_select_wave(const RowSelect &a, int b, const uint32_t *su, const int *si,
                                                     uint32_t *qu, int *qi) {
  const int lane = threadIdx.x & 63, K = a.K, V = a.V;
  const int n = K * K;
  uint32_t u[4];
  int ix[4];
#pragma unroll
  for (int s2 = 0; s2 < 4; ++s2) {
    const int j = s2 * 64 + lane;
    u[s2] = j < n ? su[j] : 0u;
    ix[s2] = j < n ? si[j] : 0x7fffffff;
  }
  auto emit_out = [&](int rank, float key, int idx) {
    const int o = b * K + rank;
    a.score_out[o] = key;
    a.tok_out[o] = idx % V;
    a.bp_out[o] = idx / V;
    if (a.row_out) a.row_out[o] = b * K + idx / V;
  };
  const int ns = wave_select<4>(u, ix, (n + 63) / 64, K, qu, qi, emit_out);
  if (lane >= ns && lane < K) {  // dead slots: hypothesis 0 continued with score -inf
    const int o = b * K + lane;
    a.score_out[o] = -INFINITY;
    a.tok_out[o] = 0;
    a.bp_out[o] = 0;
    if (a.row_out) a.row_out[o] = b * K;
  }
}
// Entry t of the table from the row candidates (key bits, token) of row k = t / K
__device__ __forceinline__ void table_entry(int t, int K, int V, float key, int tok, uint32_t *su, int *si) {
  const bool real = tok >= 0 && tok < V;
  su[t] = real ? key_code(key) : 0u;
  si[t] = real ? (t / K) * V + tok : K * V + t;
}
// The table from the row results of row_cand [M][K] (key bits, token), read by the whole
// workgroup; its first wave selects
__device__ __forceinline__ void sentence_merge(const RowSelect &a, int b, uint32_t *su, int *si, uint32_t *qu,
                                               int *qi) {
  const int t = threadIdx.x, K = a.K, V = a.V;
  const int n = K * K;  // <= 256: K <= 16
  const int n4 = (n + 3) / 4;
  if (t < n) {
    const int2 e = get_row(a.row_cand + (size_t)b * K * K + t);
    table_entry(t, K, V, __int_as_float(e.x), e.y, su, si);
  } else if (t < 4 * n4) {  // padding to whole 16-byte groups: beats nothing
    su[t] = 0u;
    si[t] = 0x7fffffff;
  }
  __syncthreads();
  if (n <= kRankMax)
    sentence_rank(a, b, su, si);
  else if (t < 64)
    sentence_select_wave(a, b, su, si, qu, qi);
}

// The K best keys prev + x[v] of one stored row x [V] (a fused ensemble's combined values),
// read by a 256-thread workgroup; emit(rank, key, token) for ranks 0..K-1.
template <int KMAX, typename Emit>
__device__ __forceinline__ void row_rescan(const float *x, int V, int K, float prev, Emit emit) {
  List<KMAX> lst;
  lst.init();
  for (int v = threadIdx.x; v < V; v += kTT) lst.push(prev + x[v], v);
  block_extract<KMAX>(lst, K, emit);
}

// Levels 2 and 3: one workgroup per row (see RowSelect).  A row's K best are staged as (key
// code, token) in LDS, four waves each select from a quarter and wave 0 merges the quarters.
// Every workgroup then counts itself in for its sentence; the last of the sentence's K rows
// merges them.
template <int KMAX, typename CT>
__global__ __launch_bounds__(kTT) void row_select_kernel(RowSelect a) {
  __shared__ __attribute__((aligned(16))) uint32_t su[kRowCap];
  __shared__ __attribute__((aligned(16))) int si[kRowCap];
  __shared__ int wtot[4];
  __shared__ uint32_t qu[4][KMAX];
  __shared__ int qi[4][KMAX];
  __shared__ int qn[4];
  __shared__ int last;
  __shared__ float res_key;  // K = 1: the row's result is the sentence's
  __shared__ int res_tok;
  __shared__ float row_lse;
  const int m = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int K = a.K, V = a.V, nl = a.nl, cap = a.cap;
  const int b = m / K;
  const bool has_lse = a.part != nullptr;
  const bool fused = has_lse || a.comb != nullptr || a.nens > 0;  // lists from the vocabulary pass
  const int *cr = a.cnt ? a.cnt + (size_t)m * nl : nullptr;

  // ---- one round trip for the usual shape (at most one partial and two lists per thread):
  // the row's log-sum-exp partial, its list fill counts and the first kSpec entries of this
  // thread's lists are all requested before any of them is needed (lists hold about one entry
  // each; entries past a list's count are loaded and ignored) ----
  const bool pre = nl <= 2 * kTT && (!has_lse || a.ntiles <= kTT);  // uniform
  float2 pq[4];  // wave 0: partials lane + 64 j
  int pc[2] = {0, 0};
  int2 pe[2][kSpec];
  if (pre) {
    if (has_lse && w == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = lane + 64 * j;
        pq[j] = i < a.ntiles ? a.part[(size_t)m * a.ntiles + i] : make_float2(0.f, 0.f);
      }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int l = t + j * kTT;
      if (l < nl) {
        pc[j] = cr ? cr[l] : cap;
        const int2 *e = a.cbuf + (size_t)m * cap * nl + l;  // entry q at e[q * nl]
#pragma unroll
        for (int q = 0; q < kSpec; ++q) pe[j][q] = q < cap ? e[(size_t)q * nl] : make_int2(0, -1);
      }
    }
  }
  // the row's log-sum-exp by wave 0 (wave_row_lse: the same bits as every other merge of these
  // partials), read by all after the next barrier
  if (w == 0) {
    const float Lw = !has_lse ? 0.f
                     : pre    ? wave_row_lse_regs<4>(pq, a.ntiles)
                              : wave_row_lse(a.part + (size_t)m * a.ntiles, a.ntiles);
    if (lane == 0) row_lse = Lw;
  }
  const float sc = fused ? a.prev_score[m] : 0.f;
  int2 *out = a.row_cand + (size_t)m * K;
  // A row result goes to the row-candidate buffer for the sentence merge; with K = 1 the row
  // is the sentence, and its result is kept in LDS for the outputs (no merge, no hand-off).
  auto emit_row = [&](int rank, float key, int tok) {
    if (K == 1) {
      res_key = key;
      res_tok = tok;
    } else {
      put_row(out + rank, key, tok);
    }
  };

  if (fused && sc == -INFINITY) {  // every key of the row is -inf: the K smallest tokens win
    if (t < K) emit_row(t, -INFINITY, t);
  } else {
    // ---- list fill counts and the block-wide offsets of this thread's entries ----
    int mine = 0;
    bool over = false;
    if (pre) {
#pragma unroll
      for (int j = 0; j < 2; ++j)
        if (t + j * kTT < nl) {
          over |= pc[j] > cap;
          mine += pc[j] < cap ? pc[j] : cap;
        }
    } else {
      for (int l = t; l < nl; l += kTT) {
        const int c = cr ? cr[l] : cap;
        over |= c > cap;
        mine += c < cap ? c : cap;
      }
    }
    const int incl = wave_incl_scan(mine);
    if (lane == 63) wtot[w] = incl;
    const bool any_over = __syncthreads_or(over);
    const float L = row_lse;
    int off = incl - mine, N = 0;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      off += v < w ? wtot[v] : 0;
      N += wtot[v];
    }
    if (any_over || N > kRowCap || (cr && N < K)) {
      // the candidates do not fit (or fall short of K): exact recomputation of the row
      if (fused) {
        if (t == 0 && a.nrecompute) atomicAdd(a.nrecompute, 1ull);
        if (a.comb)
          row_rescan<KMAX>(a.comb + (size_t)m * V, V, K, sc, emit_row);
        else if (a.nens > 0)
          row_recompute_ens<CT, KMAX>(a.evv, a.ew, a.nens, m, K, sc, emit_row);
        else
          row_recompute<CT, KMAX>(a.vv, m, K, L, sc, emit_row);
      }
    } else {
      // ---- stage the candidates as (key code, token) in LDS ----
      auto stage = [&](int pos, int2 v) {
        const int tok = v.y;
        uint32_t code = 0u;
        if (tok >= 0 && tok < V) {
          float key = __int_as_float(v.x);
          if (fused) {
            const float lp = key - L;
            key = sc + lp;
          }
          code = key_code(key);
        }
        su[pos] = code;
        si[pos] = tok;
      };
      if (pre) {
        // the first kSpec entries were loaded with the counts; of a longer list the next four
        // are requested together (one more round trip, not one per entry), the rest one by one
        int lo[2], lc[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int l = t + j * kTT;
          const int c = l < nl ? (pc[j] < cap ? pc[j] : cap) : 0;
          lo[j] = off;
          lc[j] = c;
#pragma unroll
          for (int q = 0; q < kSpec; ++q)
            if (q < c) stage(off + q, pe[j][q]);
          off += c;
        }
        int2 ex[2][4];
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int q2 = 0; q2 < 4; ++q2)
            if (kSpec + q2 < lc[j]) ex[j][q2] = a.cbuf[(size_t)m * cap * nl + t + j * kTT + (size_t)(kSpec + q2) * nl];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
#pragma unroll
          for (int q2 = 0; q2 < 4; ++q2)
            if (kSpec + q2 < lc[j]) stage(lo[j] + kSpec + q2, ex[j][q2]);
          for (int q = kSpec + 4; q < lc[j]; ++q)  // (rarer still)
            stage(lo[j] + q, a.cbuf[(size_t)m * cap * nl + t + j * kTT + (size_t)q * nl]);
        }
      } else {
        for (int l = t; l < nl; l += kTT) {
          int c = cr ? cr[l] : cap;
          c = c < cap ? c : cap;
          const int2 *e = a.cbuf + (size_t)m * cap * nl + l;
          for (int q = 0; q < c; ++q) stage(off + q, e[(size_t)q * nl]);
          off += c;
        }
      }
      __syncthreads();

      // ---- each wave selects the K best of one quarter (register slots sized to the
      // quarter: the bisection's cost grows with the slot count) ----
      {
        const int per = (N + 3) / 4;
        const int s0 = w * per, s1 = s0 + per < N ? s0 + per : N;
        const int nw = s1 > s0 ? s1 - s0 : 0;
        const int rs = (nw + 63) / 64;
        auto quarter = [&](auto slots) {
          constexpr int R = decltype(slots)::value;
          uint32_t u[R];
          int ix[R];
#pragma unroll
          for (int s = 0; s < R; ++s) {
            const int j = s0 + s * 64 + lane;
            const bool ok = s < rs && j < s1;
            u[s] = ok ? su[j] : 0u;
            ix[s] = ok ? si[j] : 0x7fffffff;
          }
          if (K == 1) {  // the best entry only: a DPP maximum of the codes, then of the indices
            uint32_t bu = 0u;
            int bi = 0x7fffffff;
#pragma unroll
            for (int s = 0; s < R; ++s)
              if (u[s] > bu || (u[s] == bu && ix[s] < bi)) {
                bu = u[s];
                bi = ix[s];
              }
            const uint32_t mu = wave_ext<uint32_t, true>(bu);
            const int mi = wave_ext<int, false>(bu == mu ? bi : 0x7fffffff);
            if (lane == 0) {
              qu[w][0] = mu;
              qi[w][0] = mi;
            }
            return mu != 0u ? 1 : 0;
          }
          return wave_select<R>(u, ix, rs, K, qu[w], qi[w], [](int, float, int) {});
        };
        int ns;
        if (rs <= 2)
          ns = quarter(std::integral_constant<int, 2>());
        else if (rs <= 4)
          ns = quarter(std::integral_constant<int, 4>());
        else
          ns = quarter(std::integral_constant<int, kSlots>());
        if (lane == 0) qn[w] = ns;
      }
      __syncthreads();

      // ---- wave 0 merges the four selections ----
      if (w == 0) {
        int base = 0, src = -1, r = 0;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          if (src < 0 && lane < base + qn[v]) {
            src = v;
            r = lane - base;
          }
          base += qn[v];
        }
        uint32_t u[1] = {src >= 0 ? qu[src][r] : 0u};
        int ix[1] = {src >= 0 ? qi[src][r] : 0x7fffffff};
        if (K == 1) {  // the best of the four quarters' best
          const uint32_t mu = wave_ext<uint32_t, true>(u[0]);
          const int mi = wave_ext<int, false>(u[0] == mu ? ix[0] : 0x7fffffff);
          if (lane == 0) {
            if (mu != 0u)
              emit_row(0, key_from_code(mu), mi);
            else
              emit_row(0, -INFINITY, 0x7fffffff);
          }
        } else {
          const int ns = wave_select<1>(u, ix, 1, K, su, si, emit_row);
          if (lane >= ns && lane < K) emit_row(lane, -INFINITY, 0x7fffffff);
        }
      }
    }
  }

  if (K == 1) {  // the sentence's result, as the merge would write it
    __syncthreads();
    if (t == 0) {
      const bool real = res_tok >= 0 && res_tok < V;
      const uint32_t mu = real ? key_code(res_key) : 0u;
      a.score_out[m] = mu != 0u ? key_from_code(mu) : -INFINITY;
      a.tok_out[m] = mu != 0u ? res_tok : 0;
      a.bp_out[m] = 0;
      if (a.row_out) a.row_out[m] = m;
    }
    return;
  }
  // ---- the last row of the sentence to finish merges the sentence ----
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): this thread's row stores have completed
  __syncthreads();
  if (t == 0) last = __hip_atomic_fetch_add(a.scnt + b, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == K - 1;
  __syncthreads();
  if (!last) return;
  sentence_merge(a, b, su, si, qu[0], qi[0]);
  if (t == 0) __hip_atomic_store(a.scnt + b, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Levels 2 and 3 for beams of K >= 2 rows whose candidate lists fit one round trip: one
// workgroup per sentence, one wave per row, so no row result leaves the workgroup (the per-row
// form hands its results to the sentence's last row through device-scope stores, an arrival
// count and loads, three round trips past the L2).  Wave k takes row b*K + k: it requests the
// row's log-sum-exp partials, list fill counts and first kSpec entries of its lists together,
// merges the log-sum-exp (wave_row_lse), stages the row's candidates in its own LDS region
// (offsets from a DPP prefix sum), selects the K best exactly (wave_topk) into the sentence's
// K x K table in LDS, and after one barrier wave 0 selects the sentence's K best of the table
// (sentence_select_wave).  A row whose lists overflow, or whose candidates
// exceed its region, is recomputed exactly by its own wave.
constexpr int kWaveCap = 1024;    // candidates one row's wave can stage
constexpr int kSentLists = 8;     // lists per lane: nl <= 512
constexpr int kSentParts = 4;     // partials per lane: ntiles <= 256

template <int KMAX, typename CT>
__global__ __launch_bounds__(64 * KMAX) void sentence_select_kernel(RowSelect a) {
  __shared__ __attribute__((aligned(16))) uint32_t su[KMAX][kWaveCap];
  __shared__ __attribute__((aligned(16))) int si[KMAX][kWaveCap];
  __shared__ uint32_t qu[KMAX][KMAX];
  __shared__ int qi[KMAX][KMAX];
  __shared__ __attribute__((aligned(16))) uint32_t tu[KMAX * KMAX + 4];
  __shared__ __attribute__((aligned(16))) int ti[KMAX * KMAX + 4];
  const int b = blockIdx.x, lane = threadIdx.x & 63;
  const int k = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int K = a.K, V = a.V, nl = a.nl, cap = a.cap;
  const int m = b * K + k;
  const bool has_lse = a.part != nullptr;
  const bool fused = has_lse || a.comb != nullptr || a.nens > 0;  // lists from the vocabulary pass
  const int *cr = a.cnt ? a.cnt + (size_t)m * nl : nullptr;
  const int2 *e0 = a.cbuf + (size_t)m * cap * nl;  // entry q of list l at e0[l + q * nl]

  // ---- one round trip: partials, list counts and the first kSpec entries of every list ----
  float2 pq[kSentParts];
#pragma unroll
  for (int j = 0; j < kSentParts; ++j) {
    const int i = lane + 64 * j;
    pq[j] = has_lse && i < a.ntiles ? a.part[(size_t)m * a.ntiles + i] : make_float2(0.f, 0.f);
  }
  int pc[kSentLists];
  int2 pe[kSentLists][kSpec];
#pragma unroll
  for (int j = 0; j < kSentLists; ++j) {
    const int l = lane + 64 * j;
    pc[j] = 0;
    if (l < nl) {
      pc[j] = cr ? cr[l] : cap;
#pragma unroll
      for (int q = 0; q < kSpec; ++q) pe[j][q] = q < cap ? e0[l + (size_t)q * nl] : make_int2(0, -1);
    }
  }
  const float sc = fused ? a.prev_score[m] : 0.f;
  const float L = has_lse ? wave_row_lse_regs<kSentParts>(pq, a.ntiles) : 0.f;

  // row results go straight into the sentence table
  uint32_t *tab_u = tu;
  int *tab_i = ti;
  auto emit_tab = [&](int rank, float key, int tok) { table_entry(k * K + rank, K, V, key, tok, tab_u, tab_i); };

  if (fused && sc == -INFINITY) {  // every key of the row is -inf: the K smallest tokens win
    if (lane < K) emit_tab(lane, -INFINITY, lane);
  } else {
    int mine = 0;
    bool over = false;
#pragma unroll
    for (int j = 0; j < kSentLists; ++j)
      if (lane + 64 * j < nl) {
        over |= pc[j] > cap;
        mine += pc[j] < cap ? pc[j] : cap;
      }
    const int incl = wave_incl_scan(mine);
    const int N = __builtin_amdgcn_readlane(incl, 63);
    const bool any_over = __ballot(over) != 0ull;
    if (any_over || N > kWaveCap || (cr && N < K)) {
      // the candidates do not fit (or fall short of K): exact recomputation of the row
      if (fused) {
        if (lane == 0 && a.nrecompute) atomicAdd(a.nrecompute, 1ull);
        List<KMAX> lst;
        lst.init();
        if (a.comb) {
          const float *x = a.comb + (size_t)m * V;
          for (int v = lane; v < V; v += 64) lst.push(sc + x[v], v);
        } else if (a.nens > 0) {
          row_recompute_ens_fill<CT, KMAX>(a.evv, a.ew, a.nens, m, sc, 0, 1, lst);
        } else {
          row_recompute_fill<CT, KMAX>(a.vv, m, L, sc, 0, 1, lst);
        }
        wave_extract<KMAX>(lst, K, emit_tab);
      } else if (lane < K) {  // (materialised lists always fit: the launch checks nl * cap)
        emit_tab(lane, -INFINITY, 0x7fffffff);
      }
    } else {
      // ---- stage the row's candidates as (key code, token) in the wave's region ----
      uint32_t *wu = su[k];
      int *wi = si[k];
      auto stage = [&](int pos, int2 v) {
        const int tok = v.y;
        uint32_t code = 0u;
        if (tok >= 0 && tok < V) {
          float key = __int_as_float(v.x);
          if (fused) key = sc + (key - L);
          code = key_code(key);
        }
        wu[pos] = code;
        wi[pos] = tok;
      };
      int off = incl - mine;
      int lo[kSentLists], lc[kSentLists];  // each list's first position and entry count
      bool longl = false;
#pragma unroll
      for (int j = 0; j < kSentLists; ++j) {
        const int l = lane + 64 * j;
        const int c = l < nl ? (pc[j] < cap ? pc[j] : cap) : 0;
        lo[j] = off;
        lc[j] = c;
#pragma unroll
        for (int q = 0; q < kSpec; ++q)
          if (q < c) stage(off + q, pe[j][q]);
        longl |= c > kSpec;
        off += c;
      }
      if (__ballot(longl) != 0ull) {
        // entries past the first kSpec: the next two of every list requested together, the
        // rest (rarer still) one by one
        int2 ex[kSentLists][2];
#pragma unroll
        for (int j = 0; j < kSentLists; ++j)
#pragma unroll
          for (int q2 = 0; q2 < 2; ++q2) {
            const int q = kSpec + q2;
            ex[j][q2] = q < lc[j] ? e0[lane + 64 * j + (size_t)q * nl] : make_int2(0, -1);
          }
#pragma unroll
        for (int j = 0; j < kSentLists; ++j) {
#pragma unroll
          for (int q2 = 0; q2 < 2; ++q2)
            if (kSpec + q2 < lc[j]) stage(lo[j] + kSpec + q2, ex[j][q2]);
          for (int q = kSpec + 2; q < lc[j]; ++q) stage(lo[j] + q, e0[lane + 64 * j + (size_t)q * nl]);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      // ---- exact K best of the row (register slots sized to its candidate count) ----
      const int rs = (N + 63) / 64;
      auto select = [&](auto slots) {
        constexpr int R = decltype(slots)::value;
        uint32_t u[R];
        int ix[R];
#pragma unroll
        for (int s2 = 0; s2 < R; ++s2) {
          const int j = s2 * 64 + lane;
          const bool ok = s2 < rs && j < N;
          u[s2] = ok ? wu[j] : 0u;
          ix[s2] = ok ? wi[j] : 0x7fffffff;
        }
        return wave_select<R>(u, ix, rs, K, qu[k], qi[k], emit_tab);
      };
      int ns;
      if (rs <= 2)
        ns = select(std::integral_constant<int, 2>());
      else if (rs <= 4)
        ns = select(std::integral_constant<int, 4>());
      else if (rs <= 8)
        ns = select(std::integral_constant<int, 8>());
      else
        ns = select(std::integral_constant<int, kWaveCap / 64>());
      if (lane >= ns && lane < K) emit_tab(lane, -INFINITY, 0x7fffffff);
    }
  }
  {  // padding of the table to whole groups of four (entries that beat nothing)
    const int t = threadIdx.x, n = K * K;
    if (t >= n && t < 4 * ((n + 3) / 4)) {
      tu[t] = 0u;
      ti[t] = 0x7fffffff;
    }
  }
  __syncthreads();
  // ---- level 3: the K best of the K x K table ----
  if (K * K <= kRankMax) {
    sentence_rank(a, b, tu, ti);
  } else if (k == 0) {
    sentence_select_wave(a, b, tu, ti, qu[0], qi[0]);
  }
}

// Level 1 for a materialised logp: the best K keys score + logp[v] of one chunk of a row (at
// most kScanKU * kTT entries, so the whole chunk is read once and stays in registers, as
// order-preserving key codes; VEC: 16-byte loads, the chunk start and the row 16-byte
// aligned).  A wave's K-th largest lane maximum bounds its K best keys from below (K of its
// keys reach it), so only keys at or above it are appended to a wave-private LDS list (ballot
// ranks); each wave then selects its K best exactly by bisection over the codes (wave_topk),
// and the first wave merges the four waves' selections the same way.  More than kCap keys at
// or above the bound (ties) are selected from the registers directly.  A chunk with fewer
// than K entries fills the rest of its K slots with no-token entries.
constexpr int kScanKU = 32;  // entries per thread of a chunk

// Rank of this lane's entry (code mu, index mi) among the n entries held by lanes 0..n-1 (n
// wave-uniform, at most 64): the number of entries that come before it in the order (larger
// code, then smaller index).  With distinct indices the ranks of the n entries are 0..n-1.
__device__ __forceinline__ int wave_rank_small(uint32_t mu, int mi, int n) {
  int rank = 0;
  for (int j = 0; j < n; ++j) {
    const uint32_t ou = __builtin_amdgcn_readlane(mu, j);
    const int oi = __builtin_amdgcn_readlane(mi, j);
    rank += (ou > mu || (ou == mu && oi < mi)) ? 1 : 0;
  }
  return rank;
}
template <int KMAX, bool VEC>
__global__ __launch_bounds__(kTT) void topk_scan_logp_kernel(int M, int K, int V, int chunk,
                                                             const float *__restrict__ prev_score,
                                                             const float *__restrict__ logp,
                                                             int2 *__restrict__ cand_out, int *scnt, int B) {
  constexpr int kCap = 256;
  __shared__ uint32_t pk[4][kCap];
  __shared__ int pi[4][kCap];
  __shared__ uint32_t wsu[4][KMAX];
  __shared__ int wsi[4][KMAX];
  __shared__ uint32_t qu[4][KMAX];
  __shared__ int qi[4][KMAX];
  __shared__ int qn[4];
  const int m = blockIdx.y, ch = blockIdx.x, nch = gridDim.x;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  if (m == 0 && ch == 0)
    for (int i = t; i < B; i += kTT) __hip_atomic_store(scnt + i, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const float sc = prev_score[m];
  const float *row = logp + (size_t)m * V;
  const int v0 = ch * chunk, v1 = min(V, v0 + chunk);
  // entry q of this thread: VEC, vector g = q / 4 of 4 consecutive entries; else one entry
  auto idx_of = [&](int q) { return VEC ? v0 + 4 * (t + (q >> 2) * kTT) + (q & 3) : v0 + t + q * kTT; };
  // keys sc + logp in registers; entries past the chunk end are -inf and never taken (an
  // entry is taken only when its key is at least the wave's bound, which is a real key)
  float key[kScanKU];
  if constexpr (VEC) {
#pragma unroll
    for (int g = 0; g < kScanKU / 4; ++g) {
      const int i0 = v0 + 4 * (t + g * kTT);
      float4 xv = make_float4(0.f, 0.f, 0.f, 0.f);
      if (i0 + 3 < v1) {
        xv = *(const float4 *)(row + i0);
      } else if (i0 < v1) {  // the chunk's ragged end
        xv.x = row[i0];
        if (i0 + 1 < v1) xv.y = row[i0 + 1];
        if (i0 + 2 < v1) xv.z = row[i0 + 2];
      }
      key[4 * g + 0] = i0 + 0 < v1 ? sc + xv.x : -INFINITY;
      key[4 * g + 1] = i0 + 1 < v1 ? sc + xv.y : -INFINITY;
      key[4 * g + 2] = i0 + 2 < v1 ? sc + xv.z : -INFINITY;
      key[4 * g + 3] = i0 + 3 < v1 ? sc + xv.w : -INFINITY;
    }
  } else {
#pragma unroll
    for (int q = 0; q < kScanKU; ++q) key[q] = idx_of(q) < v1 ? sc + row[idx_of(q)] : -INFINITY;
  }
  // lane maximum over the lane's real entries, as a code (0: none)
  float lm = -INFINITY;
  bool any = false;
#pragma unroll
  for (int q = 0; q < kScanKU; ++q) {
    lm = fmaxf(lm, key[q]);
    any |= idx_of(q) < v1;
  }
  uint32_t mx[1] = {any ? key_code(lm) : 0u};
  // the bound: the K-th largest lane maximum (with fewer than K lanes holding entries, the
  // smallest real key: every entry is then taken)
  const bool enough = wave_count_ge<1>(mx, 1, 1u) >= K;
  uint32_t tau = enough ? wave_kth_code<1>(mx, 1, K) : 1u;
  const float tauf = key_from_code(tau < 1u ? 1u : tau);
  const uint64_t lt = (1ull << lane) - 1ull;
  int npass = 0;  // wave-uniform
#pragma unroll
  for (int q = 0; q < kScanKU; ++q) {
    const bool pass = idx_of(q) < v1 && (enough ? key[q] >= tauf : true);
    const uint64_t bal = __ballot(pass);
    if (bal) {  // uniform: most entries of most waves stay under the bound
      const int slot = npass + __popcll(bal & lt);
      if (pass && slot < kCap) {
        pk[wv][slot] = key_code(key[q]);
        pi[wv][slot] = idx_of(q);
      }
      npass += __popcll(bal);
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  // this wave's K best, by rank, into qu/qi
  auto keep = [&](int rank, float key, int idx) {
    qu[wv][rank] = key_code(key);
    qi[wv][rank] = idx;
  };
  int ns;
  if (npass <= 64) {  // the usual case: one appended key per lane, ranked directly
    const bool has = lane < npass;
    const uint32_t mu = has ? pk[wv][lane] : 0u;
    const int mi = has ? pi[wv][lane] : 0x7fffffff;
    const int rank = wave_rank_small(mu, mi, npass);
    if (has && rank < K) {
      qu[wv][rank] = mu;
      qi[wv][rank] = mi;
    }
    ns = npass < K ? npass : K;
  } else if (npass <= kCap) {
    constexpr int R = kCap / 64;
    uint32_t cu[R];
    int ci[R];
    const int rs = (npass + 63) / 64;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int j = r * 64 + lane;
      const bool ok = j < npass;
      cu[r] = ok ? pk[wv][j] : 0u;
      ci[r] = ok ? pi[wv][j] : 0x7fffffff;
    }
    ns = wave_topk<R>(cu, ci, rs, K, wsu[wv], wsi[wv], keep);
  } else {  // more than kCap keys at or above the bound (ties): select from the registers
    uint32_t u[kScanKU];
    int ix[kScanKU];
#pragma unroll
    for (int q = 0; q < kScanKU; ++q) {
      ix[q] = idx_of(q);
      u[q] = ix[q] < v1 ? key_code(key[q]) : 0u;
    }
    ns = wave_topk<kScanKU>(u, ix, kScanKU, K, wsu[wv], wsi[wv], keep);
  }
  if (lane == 0) qn[wv] = ns;
  __syncthreads();
  if (wv != 0) return;
  // the first wave merges the four selections (at most 4 K <= 64 entries, one per lane)
  int base = 0, src = -1, r = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    if (src < 0 && lane < base + qn[w]) {
      src = w;
      r = lane - base;
    }
    base += qn[w];
  }
  const uint32_t mu = src >= 0 ? qu[src][r] : 0u;
  const int mi = src >= 0 ? qi[src][r] : 0x7fffffff;
  int2 *o = cand_out + (size_t)m * K * nch + ch;  // entry r at o[r * nch] (entry-major per row)
  const int rank = wave_rank_small(mu, mi, base);  // base = the four selections' entries (<= 4 K)
  if (src >= 0 && rank < K) o[(size_t)rank * nch] = make_int2(__float_as_int(key_from_code(mu)), mi);
  const int nsel = base < K ? base : K;
  if (lane >= nsel && lane < K) o[(size_t)lane * nch] = make_int2(0, -1);  // no entry
}

// chunks of a materialised row: at most kScanKU * kTT entries each (register-resident), a
// multiple of 1024 (16-byte aligned starts), and for few rows enough chunks for about 3072
// workgroups in all
void topk_scan_shape(int M, int V, int *chunk, int *nchunks) {
  const long nmin = ((long)V + kScanKU * kTT - 1) / (kScanKU * kTT);
  const long want = (3072 + (long)M - 1) / (M > 0 ? M : 1);
  const long most = ((long)V + 1023) / 1024;
  const long n = std::max(nmin, std::min(want, most));
  long c = ((long)V + n - 1) / n;
  c = (c + 1023) / 1024 * 1024;
  *chunk = (int)c;
  *nchunks = (int)(((long)V + c - 1) / c);
}

static int kbucket(int K) { return K <= 1 ? 1 : K <= 2 ? 2 : K <= 4 ? 4 : K <= 8 ? 8 : 16; }

#define MT_KSWITCH(K, CALL) \
  switch (kbucket(K)) {     \
    case 1: CALL(1); break; \
    case 2: CALL(2); break; \
    case 4: CALL(4); break; \
    case 8: CALL(8); break; \
    default: CALL(16); break; \
  }

hipError_t launch_row_select(const RowSelect &a, hipStream_t st) {
  const int M = a.B * a.K;
  if (M == 0) return hipSuccess;
  const bool fused = a.part != nullptr || a.comb != nullptr || a.nens > 0;
  // One workgroup per sentence when a row's work is light: a materialised row's candidates
  // (nl * cap of them) fit a wave's region, or a fused row has at most one list per lane.  The
  // workgroups then occupy only B compute units, and with the vocabulary pass's lists of a
  // large vocabulary (a few hundred per row, about one candidate each) the per-row form, over
  // every unit, is faster despite its hand-off (17 against 23 us at B = 64, K = 12, V = 50k).
  // Materialised lists go by sentence at any K (K = 1: one wave per row, 6.0 against 7.8 us
  // at B = 1024); fused lists of a large vocabulary keep the per-row form at K = 1 too (one
  // wave per row, 11.9 against 9.8 us).
  const bool light = fused ? a.K >= 2 && a.nl <= 64 : (long)a.nl * a.cap <= kWaveCap;
  const bool by_sentence = a.K >= 1 && a.K <= 16 && a.nl <= 64 * kSentLists &&
                           (a.part == nullptr || a.ntiles <= 64 * kSentParts) && light;
  if (by_sentence) {
#define MT_SS(N)                                                                                        \
  if (a.bf16_mma)                                                                                       \
    hipLaunchKernelGGL((sentence_select_kernel<N, bf16>), dim3(a.B), dim3(64 * a.K), 0, st, a);         \
  else                                                                                                  \
    hipLaunchKernelGGL((sentence_select_kernel<N, float>), dim3(a.B), dim3(64 * a.K), 0, st, a);
    MT_KSWITCH(a.K, MT_SS)
#undef MT_SS
    return hipGetLastError();
  }
#define MT_RS(N)                                                                          \
  if (a.bf16_mma)                                                                         \
    hipLaunchKernelGGL((row_select_kernel<N, bf16>), dim3(M), dim3(kTT), 0, st, a);       \
  else                                                                                    \
    hipLaunchKernelGGL((row_select_kernel<N, float>), dim3(M), dim3(kTT), 0, st, a);
  MT_KSWITCH(a.K, MT_RS)
#undef MT_RS
  return hipGetLastError();
}

hipError_t launch_topk_scan_logp(int M, int K, int V, int nchunks, const float *prev_score,
                                 const float *logp, int2 *cand_out, int *scnt, int B, hipStream_t st) {
  if (M == 0) return hipSuccess;
  int chunk = 0, nch = 0;
  topk_scan_shape(M, V, &chunk, &nch);
  if (nch != nchunks) return hipErrorInvalidValue;  // the workspace holds nchunks lists per row
  const bool vec = V % 4 == 0 && ((uintptr_t)logp & 15) == 0;
#define MT_TS(N)                                                                                               \
  if (vec)                                                                                                     \
    hipLaunchKernelGGL((topk_scan_logp_kernel<N, true>), dim3(nch, M), dim3(kTT), 0, st, M, K, V, chunk,        \
                       prev_score, logp, cand_out, scnt, B);                                                   \
  else                                                                                                         \
    hipLaunchKernelGGL((topk_scan_logp_kernel<N, false>), dim3(nch, M), dim3(kTT), 0, st, M, K, V, chunk,       \
                       prev_score, logp, cand_out, scnt, B);
  MT_KSWITCH(K, MT_TS)
#undef MT_TS
  return hipGetLastError();
}

}  // namespace mt
