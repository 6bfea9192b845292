// Beam selection: the best K of the K x V extensions of each sentence.
//
// Total order at every level: larger key first, ties -> smaller flat index k*V + v.
// Keys are fp32: key = prev_score + (logit - lse), summed in that order, which is
// exactly how a materialised log-probability (logit - lse) plus the score would be
// rounded.  Levels:
//   1. per (row, vocabulary tile): the vocabulary GEMM epilogue keeps the tile's best
//      kc logits (or topk_scan_logp keeps the best keys of a chunk of a given logp row);
//   2. per row: topk_rows turns the row's tile candidates into keys and keeps the K best;
//   3. per sentence: topk_sentence merges the K rows' K candidates into the new beam.
// Within a row the key is a non-decreasing function of the logit, so a row's K best
// keys are among its tiles' K best logits, except where rounding makes unequal logits
// produce equal keys (ties at the cut).
#include "mt_internal.h"

namespace mt {

constexpr int kTT = 256;

// Level 2.  cand: [M][ncand] (key or logit bits, token); lse != NULL means the values are
// logits to turn into keys with prev_score; tokens >= V are padding and skipped.
template <int KMAX>
__global__ __launch_bounds__(kTT) void topk_rows_kernel(int M, int K, int V, int ncand,
                                                        const int2 *__restrict__ cand,
                                                        const float *__restrict__ lse,
                                                        const float *__restrict__ prev_score,
                                                        int2 *__restrict__ row_out) {
  const int m = blockIdx.x;
  const int2 *c = cand + (size_t)m * ncand;
  const float L = lse ? lse[m] : 0.f;
  const float sc = lse ? prev_score[m] : 0.f;
  List<KMAX> lst;
  lst.init();
  for (int j = threadIdx.x; j < ncand; j += kTT) {
    const int2 e = c[j];
    if (e.y >= V || e.y < 0) continue;
    float key = __int_as_float(e.x);
    if (lse) {
      const float lp = key - L;
      key = sc + lp;
    }
    lst.push(key, e.y);
  }
  block_extract<KMAX>(lst, K, [&](int r, float v, int i) { row_out[(size_t)m * K + r] = make_int2(__float_as_int(v), i); });
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

// Level 3: one wave per sentence; candidate (k, j) -> flat index k*V + token.
template <int KMAX>
__global__ __launch_bounds__(256) void topk_sentence_kernel(int B, int K, int V,
                                                            const int2 *__restrict__ row_cand,
                                                            float *__restrict__ score_out,
                                                            int32_t *__restrict__ tok_out,
                                                            int32_t *__restrict__ bp_out,
                                                            int32_t *__restrict__ row_out) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;  // uniform per wave
  const int n = K * K;
  List<KMAX> lst;
  lst.init();
  for (int j = lane; j < n; j += 64) {
    const int k = j / K;
    const int2 e = row_cand[(size_t)(b * K + k) * K + (j % K)];
    if (e.y < 0 || e.y >= V) continue;
    lst.push(__int_as_float(e.x), k * V + e.y);
  }
  wave_extract<KMAX>(lst, K, [&](int r, float v, int i) {
    if (lane != 0) return;
    const int o = b * K + r;
    // a flat index beyond the K x V range only appears if fewer than K candidates exist
    const int k = i < K * V ? i / V : 0;
    const int tok = i < K * V ? i % V : 0;
    score_out[o] = v;
    tok_out[o] = tok;
    bp_out[o] = k;
    if (row_out) row_out[o] = b * K + k;
  });
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

hipError_t launch_topk_rows(int M, int K, int V, int ncand, const int2 *cand, const float *lse,
                            const float *prev_score, int2 *row_out, hipStream_t st) {
  if (M == 0) return hipSuccess;
#define MT_TR(N) hipLaunchKernelGGL((topk_rows_kernel<N>), dim3(M), dim3(kTT), 0, st, M, K, V, ncand, cand, lse, prev_score, row_out)
  MT_KSWITCH(K, MT_TR)
#undef MT_TR
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
