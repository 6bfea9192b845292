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
//   3. per sentence (topk_sentence): the K best of the K rows' K candidates.
// Levels 2 and 3 select exactly by bisection over order-preserving integer codes of the
// keys (wave_topk): every count is a ballot plus a scalar popcount, ties at the cut are
// resolved by a second bisection over the indices, and the K survivors are ranked by
// pairwise comparison.  Nothing is sorted and no step depends on a cross-lane exchange
// chain longer than one min/max reduction.
#include "mt_internal.h"

namespace mt {

constexpr int kTT = 256;
constexpr int kRowCap = 4096;          // candidates one row can stage in LDS
constexpr int kSlots = kRowCap / 256;  // register slots per lane when a wave takes a quarter

// Level 2.  Row m's candidates sit in nl lists of up to cap entries: cbuf [M][nl][cap] of
// (value bits, token), with fill counts cnt [M][nl] (NULL: every list holds cap entries).
// lse != NULL: values are logits, turned into keys prev_score + (logit - lse); else values
// are keys.  Tokens outside [0, V) are padding.  A row whose candidates do not fit (a list
// count above cap, or more than kRowCap in total), or, with fill counts, a row with fewer
// than K candidates (its threshold was above its K-th best), is flagged in ovf[m] (if given)
// and left for the exact recomputation; other rows get ovf[m] = 0 and their K best in row_out.
template <int KMAX>
__global__ __launch_bounds__(kTT) void row_select_kernel(int M, int K, int V, int nl, int cap,
                                                         const int *__restrict__ cnt,
                                                         const int2 *__restrict__ cbuf,
                                                         const float *__restrict__ lse,
                                                         const float *__restrict__ prev_score,
                                                         int2 *__restrict__ row_out, int *__restrict__ ovf) {
  __shared__ uint32_t su[kRowCap];
  __shared__ int si[kRowCap];
  __shared__ int wtot[4];
  __shared__ uint32_t qu[4][KMAX];
  __shared__ int qi[4][KMAX];
  __shared__ int qn[4];
  const int m = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
  const float L = lse ? lse[m] : 0.f;
  const float sc = lse ? prev_score[m] : 0.f;
  int2 *out = row_out + (size_t)m * K;
  if (lse && sc == -INFINITY) {  // every key of the row is -inf: the K smallest tokens win
    if (t < K) out[t] = make_int2(__float_as_int(-INFINITY), t);
    if (t == 0 && ovf) ovf[m] = 0;
    return;
  }
  const int *cr = cnt ? cnt + (size_t)m * nl : nullptr;

  // ---- list fill counts and the block-wide offsets of this thread's entries ----
  int mine = 0;
  bool over = false;
  for (int l = t; l < nl; l += kTT) {
    const int c = cr ? cr[l] : cap;
    over |= c > cap;
    mine += c < cap ? c : cap;
  }
  int incl = mine;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wtot[w] = incl;
  const bool any_over = __syncthreads_or(over);
  int off = incl - mine, N = 0;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    off += v < w ? wtot[v] : 0;
    N += wtot[v];
  }
  if (any_over || N > kRowCap || (cr && N < K)) {
    if (t == 0 && ovf) ovf[m] = 1;
    return;
  }
  if (t == 0 && ovf) ovf[m] = 0;

  // ---- stage the candidates as (key code, token) in LDS ----
  for (int l = t; l < nl; l += kTT) {
    int c = cr ? cr[l] : cap;
    c = c < cap ? c : cap;
    const int2 *e = cbuf + ((size_t)m * nl + l) * cap;
    for (int q0 = 0; q0 < c; q0 += 8) {
      int2 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = q0 + u < c ? e[q0 + u] : make_int2(0, -1);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (q0 + u >= c) continue;
        const int tok = v[u].y;
        uint32_t code = 0u;
        if (tok >= 0 && tok < V) {
          float key = __int_as_float(v[u].x);
          if (lse) {
            const float lp = key - L;
            key = sc + lp;
          }
          code = key_code(key);
        }
        su[off + q0 + u] = code;
        si[off + q0 + u] = tok;
      }
    }
    off += c;
  }
  __syncthreads();

  // ---- each wave selects the K best of one quarter ----
  {
    const int per = (N + 3) / 4;
    const int s0 = w * per, s1 = s0 + per < N ? s0 + per : N;
    const int nw = s1 > s0 ? s1 - s0 : 0;
    const int rs = (nw + 63) / 64;
    uint32_t u[kSlots];
    int ix[kSlots];
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
      const int j = s0 + s * 64 + lane;
      const bool ok = s < rs && j < s1;
      u[s] = ok ? su[j] : 0u;
      ix[s] = ok ? si[j] : 0x7fffffff;
    }
    const int ns = wave_topk<kSlots>(u, ix, rs, K, qu[w], qi[w], [](int, float, int) {});
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
    const int ns = wave_topk<1>(u, ix, 1, K, su, si, [&](int rank, float key, int tok) {
      out[rank] = make_int2(__float_as_int(key), tok);
    });
    if (lane >= ns && lane < K) out[lane] = make_int2(__float_as_int(-INFINITY), 0x7fffffff);
  }
}

// Level 1 for a materialised logp: the best K keys score + logp[v] of one chunk of a row.
template <int KMAX>
__global__ __launch_bounds__(kTT) void topk_scan_logp_kernel(int M, int K, int V, int chunk,
                                                             const float *__restrict__ prev_score,
                                                             const float *__restrict__ logp,
                                                             int2 *__restrict__ cand_out) {
  const int m = blockIdx.y, ch = blockIdx.x, nch = gridDim.x;
  const float sc = prev_score[m];
  const float *row = logp + (size_t)m * V;
  const int v0 = ch * chunk, v1 = min(V, v0 + chunk);
  List<KMAX> lst;
  lst.init();
  for (int v = v0 + threadIdx.x; v < v1; v += kTT) lst.push(sc + row[v], v);
  int2 *o = cand_out + ((size_t)m * nch + ch) * K;
  block_extract<KMAX>(lst, K, [&](int r, float v, int i) { o[r] = make_int2(__float_as_int(v), i); });
}

// Level 3: one wave per sentence over the K x K row candidates (row_cand [M][K] of
// (key bits, token)); candidate (k, j) has flat index k*V + token.
template <int KMAX>
__global__ __launch_bounds__(256) void topk_sentence_kernel(int B, int K, int V,
                                                            const int2 *__restrict__ row_cand,
                                                            float *__restrict__ score_out,
                                                            int32_t *__restrict__ tok_out,
                                                            int32_t *__restrict__ bp_out,
                                                            int32_t *__restrict__ row_out) {
  constexpr int R = (KMAX * KMAX + 63) / 64;
  __shared__ uint32_t su[4][KMAX];
  __shared__ int si[4][KMAX];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int b = blockIdx.x * 4 + w;
  if (b >= B) return;  // uniform per wave
  const int n = K * K;
  uint32_t u[R];
  int ix[R];
#pragma unroll
  for (int s = 0; s < R; ++s) {
    const int j = s * 64 + lane;
    u[s] = 0u;
    ix[s] = 0x7fffffff;
    if (j < n) {
      const int k = j / K;
      const int2 e = row_cand[(size_t)(b * K + k) * K + (j - k * K)];
      if (e.y >= 0 && e.y < V) {
        u[s] = key_code(__int_as_float(e.x));
        ix[s] = k * V + e.y;
      }
    }
  }
  const int ns = wave_topk<R>(u, ix, (n + 63) / 64, K, su[w], si[w], [&](int rank, float key, int i) {
    const int o = b * K + rank;
    score_out[o] = key;
    tok_out[o] = i % V;
    bp_out[o] = i / V;
    if (row_out) row_out[o] = b * K + i / V;
  });
  if (lane >= ns && lane < K) {  // fewer than K candidates: dead slots continue hypothesis 0
    const int o = b * K + lane;
    score_out[o] = -INFINITY;
    tok_out[o] = 0;
    bp_out[o] = 0;
    if (row_out) row_out[o] = b * K;
  }
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

hipError_t launch_row_select(int M, int K, int V, int nl, int cap, const int *cnt, const int2 *cbuf,
                             const float *lse, const float *prev_score, int2 *row_out, int *ovf,
                             hipStream_t st) {
  if (M == 0) return hipSuccess;
#define MT_RS(N) \
  hipLaunchKernelGGL((row_select_kernel<N>), dim3(M), dim3(kTT), 0, st, M, K, V, nl, cap, cnt, cbuf, lse, prev_score, row_out, ovf)
  MT_KSWITCH(K, MT_RS)
#undef MT_RS
  return hipGetLastError();
}

hipError_t launch_topk_scan_logp(int M, int K, int V, int nchunks, const float *prev_score,
                                 const float *logp, int2 *cand_out, hipStream_t st) {
  if (M == 0) return hipSuccess;
  const int chunk = (V + nchunks - 1) / nchunks;
#define MT_TS(N) hipLaunchKernelGGL((topk_scan_logp_kernel<N>), dim3(nchunks, M), dim3(kTT), 0, st, M, K, V, chunk, prev_score, logp, cand_out)
  MT_KSWITCH(K, MT_TS)
#undef MT_TS
  return hipGetLastError();
}

hipError_t launch_topk_sentence(int B, int K, int V, const int2 *row_cand, float *score_out,
                                int32_t *tok_out, int32_t *bp_out, int32_t *row_out,
                                hipStream_t st) {
  if (B == 0) return hipSuccess;
#define MT_TSN(N) hipLaunchKernelGGL((topk_sentence_kernel<N>), dim3((B + 3) / 4), dim3(256), 0, st, B, K, V, row_cand, score_out, tok_out, bp_out, row_out)
  MT_KSWITCH(K, MT_TSN)
#undef MT_TSN
  return hipGetLastError();
}

}  // namespace mt
