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

// ---------------------------------------------------------------------------------------
// launchers (host side).  All return hipSuccess or the launch error.
// ---------------------------------------------------------------------------------------

enum Epilogue { EPI_STORE = 0, EPI_TANH = 1, EPI_VOCAB = 2 };

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

struct VocabOut {          // fused epilogue outputs of the vocabulary GEMM
  float2 *part;            // [M][ntiles] (tile max, sum exp(l - max))
  int2 *cand;              // [M][ntiles][kc] (key bits, token) best kc of the tile
  int kc;                  // candidates kept per (row, tile)
  int ntiles;
  float *logits;           // [M][N] or NULL
};

// gemm dtype: 0 fp32 MFMA, 1 bf16 MFMA.  nprob = 1 or 2 (problems share one launch).
hipError_t launch_gemm(int bf16_mma, const GemmProblem *probs, int nprob, Epilogue epi,
                       const VocabOut *vo, hipStream_t st);
int vocab_tile_n();  // BN of the vocabulary GEMM (columns per candidate tile)

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
