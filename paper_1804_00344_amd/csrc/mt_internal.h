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

// Wave-level version (no barriers): the wave's best head is found with shuffles; the owning
// lane pops it.  Every lane receives the n results in order through `emit` (lane-uniform).
template <int KMAX, typename Emit>
__device__ __forceinline__ void wave_extract(List<KMAX> &L, int n, Emit emit) {
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
    emit(r, bv, bi);
  }
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
// thr[m] = K-th best of sample[m][0 .. min(V, S)) minus a rounding margin, S = vocab_sample_size(V);
// sample [M][S] holds the logits of the first S vocabulary entries (computed by launch_gemm)
hipError_t launch_vocab_threshold(int M, int V, int K, const float *sample, float *thr, hipStream_t st);
// part [M][n_chunks] (max, sum exp(l - max)); every logit >= thr[m] goes to cbuf
// [M][n_chunks][lists][cap] with counts in ccnt [M][n_chunks][lists]; logits [M][V] or NULL
hipError_t launch_vocab(int bf16_mma, const void *t, const void *wp, const float *bias_pad, int M, int V,
                        int E, int n_chunks, const float *thr, float2 *part, int2 *cbuf, int *ccnt, int cap,
                        float *logits, hipStream_t st);
// row_out [M][K] (key bits, token): the K best keys prev_score + (logit - lse) of each row
hipError_t launch_vocab_rows(int bf16_mma, const void *t, const void *wp, const float *bias_pad, int M, int V,
                             int E, int K, int n_chunks, const int2 *cbuf, const int *ccnt, int cap,
                             const float *lse, const float *prev_score, int2 *row_out, int *ovf,
                             hipStream_t st);
constexpr int kVocabCap = 32;  // candidate buffer entries per (row, chunk, list)
constexpr int kVocabPad = 64;  // vocabulary rows are padded to a multiple of this

hipError_t launch_gru_cell(int M, int H, const float *a, int lda, const float *u, int ldu,
                           const float *hsrc, const int32_t *hidx, int hrows, int32_t *err,
                           const float *ga, const float *ba, const float *gu, const float *bu,
                           float eps, float *out, int ldo, float *tap, hipStream_t st);

hipError_t launch_readout(int M, int E, const float *p1, int ld1, const float *p2, int ld2,
                          const float *p3, int ld3, const float *bt, const float *g,
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

// candidates are (key, idx) pairs stored as int2 {float bits, idx}
hipError_t launch_topk_rows(int M, int K, int V, int ncand_per_row, const int2 *cand,
                            const float *lse, const float *prev_score, int2 *row_out,
                            hipStream_t st);
hipError_t launch_topk_scan_logp(int M, int K, int V, int nchunks, const float *prev_score,
                                 const float *logp, int2 *cand_out, hipStream_t st);
hipError_t launch_topk_sentence(int B, int K, int V, const int2 *row_cand, float *score_out,
                                int32_t *tok_out, int32_t *bp_out, int32_t *row_out,
                                hipStream_t st);

}  // namespace mt
