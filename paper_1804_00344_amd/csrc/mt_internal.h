// Internal declarations shared by the libmtstep translation units (GPU path only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "../../include/mtstep.h"

namespace mt {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kWave = 64;
constexpr int kXcds = 8;
constexpr int kKMax = 16;  // largest supported beam

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

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
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
// winner pops its head.  Writes n results (key bits, idx) through `emit`.
template <int KMAX, typename Emit>
__device__ __forceinline__ void block_extract(List<KMAX> &L, int n, Emit emit) {
  __shared__ float wv[4];
  __shared__ int wi[4];
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
    if (t == 0) emit(r, bv, bi);
  }
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
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t a = __shfl_xor(lo, o, 64), b = __shfl_xor(hi, o, 64);
    lo = a < lo ? a : lo;
    hi = b > hi ? b : hi;
  }
  lo = __builtin_amdgcn_readfirstlane(lo);
  hi = __builtin_amdgcn_readfirstlane(hi);
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
    tau = wave_kth_code<R>(u, rs, K);
    const int gt = tau == 0xffffffffu ? 0 : wave_count_ge<R>(u, rs, tau + 1u);
    const int need = K - gt;
    const int eq = wave_count_eq_le<R>(u, ix, rs, tau, 0x7fffffff);
    if (eq > need) {  // ties at the cut: keep the `need` smallest indices among them
      int lo = 0x7fffffff, hi = (int)0x80000000;
#pragma unroll
      for (int s = 0; s < R; ++s)
        if (s < rs && u[s] == tau) {
          lo = ix[s] < lo ? ix[s] : lo;
          hi = ix[s] > hi ? ix[s] : hi;
        }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const int a = __shfl_xor(lo, o, 64), b = __shfl_xor(hi, o, 64);
        lo = a < lo ? a : lo;
        hi = b > hi ? b : hi;
      }
      lo = __builtin_amdgcn_readfirstlane(lo);
      hi = __builtin_amdgcn_readfirstlane(hi);
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
  if (lane < ns) {
    const uint32_t mu = su[lane];
    const int mi = si[lane];
    int rank = 0;
    for (int j = 0; j < ns; ++j) {
      const uint32_t ou = su[j];
      const int oi = si[j];
      rank += (ou > mu || (ou == mu && oi < mi)) ? 1 : 0;
    }
    emit(rank, key_from_code(mu), mi);
  }
  return ns;
}

// ---------------------------------------------------------------------------------------
// launchers (host side).  All return hipSuccess or the launch error.
// ---------------------------------------------------------------------------------------

enum Epilogue { EPI_STORE = 0, EPI_TANH = 1 };

struct GemmProblem {
  const void *A;          // activations [rows][lda] (fp32 or bf16, see a_bf16)
  const int32_t *a_idx;   // optional gather: row m reads A row a_idx[m] (clamped to a_rows)
  int a_rows;             // rows available in A (for the gather clamp)
  int lda;                // elements
  int a_bf16;             // A element type: 0 fp32, 1 bf16
  const void *Bp;         // packed weights [N_pad][ldb], K contiguous, compute dtype
  int ldb;                // = K_pad
  const float *bias;      // [N] or NULL
  void *out;              // [M][ldc] (fp32, or bf16 if out_bf16)
  int ldc;
  int out_bf16;
  int M, N, K;
  int32_t *err;           // device error word (bit err_bit set on a clamped gather)
  int err_bit;
};

// gemm dtype: 0 fp32 MFMA, 1 bf16 MFMA.  nprob = 1 or 2 (problems share one launch).
hipError_t launch_gemm(int bf16_mma, const GemmProblem *probs, int nprob, Epilogue epi,
                       hipStream_t st);

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
hipError_t launch_vocab_threshold(int M, int V, int K, const float *sample, float *thr, hipStream_t st);
// part [M][n_chunks] (reference m, sum exp(l - m)); every logit >= thr[m] goes to cbuf
// [M][n_chunks][lists][cap] with counts in ccnt [M][n_chunks][lists] (a count above cap marks
// an overflowed list); logits [M][V] or NULL.  fixed_ref: the caller has proven every logit
// lies in [-40, 40], so the reference is 0 and no running maximum is kept.
hipError_t launch_vocab(int bf16_mma, const void *t, const void *wp, const float *bias_pad, int M, int V,
                        int E, int n_chunks, const float *thr, float2 *part, int2 *cbuf, int *ccnt, int cap,
                        float *logits, int fixed_ref, hipStream_t st);
// exact recomputation of the rows with ovf[m] != 0: row_out[m] = the K best keys
// prev_score + (logit - lse) over the whole vocabulary
hipError_t launch_vocab_fallback(int bf16_mma, const void *t, const void *wp, const float *bias_pad, int M,
                                 int V, int E, int K, const float *lse, const float *prev_score, int2 *row_out,
                                 const int *ovf, hipStream_t st);
constexpr int kVocabCap = 32;  // candidate buffer entries per (row, chunk, list)
constexpr int kVocabPad = 64;  // vocabulary rows are padded to a multiple of this

// GRU cell for M rows; a row m = aidx[m] (if given), previous state row hidx[m] (if given);
// out-of-range indices are clamped and flagged in err (bit 0: aidx, bit 1: hidx)
hipError_t launch_gru_cell(int M, int H, const float *a, int lda, const int32_t *aidx, int arows,
                           const float *u, int ldu, const float *hsrc, const int32_t *hidx, int hrows,
                           int32_t *err, const float *ga, const float *ba, const float *gu, const float *bu,
                           float eps, float *out, int ldo, float *tap, hipStream_t st);

hipError_t launch_readout(int M, int E, const float *p1, int ld1, const float *p2, int ld2, const int32_t *idx2,
                          int rows2, const float *p3, int ld3, const float *bt, const float *g,
                          const float *be, float eps, void *t_out, int t_bf16, float *tap,
                          hipStream_t st);

hipError_t launch_masked_mean(int B, int S, int Cd, const void *ctx, int ctx_bf16,
                              const float *mask, float *out, hipStream_t st);

hipError_t launch_attention(int B, int K, int S, int A, int Cd, const void *P, const void *Cx,
                            int bf16_io, const float *mask, const float *q, int ldq,
                            const float *va, float *ctx_out, int ldc, float *alpha_out,
                            hipStream_t st);

hipError_t launch_lse(int M, int ntiles, const float2 *part, float *lse, float *logits, int V,
                      hipStream_t st);

// candidates are (value, token) pairs stored as int2 {float bits, token}.  Row selection: the K
// best keys of each row from nl lists of up to cap candidates (cnt NULL = lists full; lse NULL
// = values are keys, else logits keyed as prev_score + (logit - lse)); rows whose candidates do
// not fit get ovf[m] = 1 and no output (see launch_vocab_fallback), the others ovf[m] = 0.
hipError_t launch_row_select(int M, int K, int V, int nl, int cap, const int *cnt, const int2 *cbuf,
                             const float *lse, const float *prev_score, int2 *row_out, int *ovf,
                             hipStream_t st);
hipError_t launch_topk_scan_logp(int M, int K, int V, int nchunks, const float *prev_score,
                                 const float *logp, int2 *cand_out, hipStream_t st);
hipError_t launch_topk_sentence(int B, int K, int V, const int2 *row_cand, float *score_out,
                                int32_t *tok_out, int32_t *bp_out, int32_t *row_out,
                                hipStream_t st);

}  // namespace mt
