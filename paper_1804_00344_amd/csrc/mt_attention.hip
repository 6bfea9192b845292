// Additive attention with a masked softmax over the source positions of one sentence,
// one 256-thread workgroup per hypothesis row (m = b*K + k):
//   e_i   = sum_a va[a] * tanh(P[b,i,a] + q[m,a])      (valid i only)
//   alpha = exp(e_i - max_valid e) / sum_valid exp(...)  (exactly 0 at masked i)
//   c[m]  = sum_valid alpha_i * Cx[b,i,:]
// The valid positions are first compacted into an LDS list (ballot prefix sums), so neither
// loop branches on the mask or reads a masked row.  Scores: each wave takes two valid
// positions per iteration; its 64 lanes stream the A features of P[b,i] in coalesced 16-byte
// granules against q and va held in registers, and reduce with cross-lane shuffles.  Softmax:
// one wave over the compacted scores.  Context: each thread owns 16-byte column granules of
// C and walks the valid positions four at a time, so four rows of loads are in flight.
// Workgroup ids are remapped so that the K rows of one sentence run on one XCD and share its
// L2 copy of P[b] and Cx[b].
#include "mt_internal.h"

namespace mt {

constexpr int kAT = 256;
constexpr int kMaxS = 1024;

template <typename T>
struct Gran;  // one 16-byte granule of a row, widened to fp32
template <>
struct Gran<float> {
  static constexpr int N = 4;
  __device__ __forceinline__ static void load(const float *p, float (&x)[4]) {
    const float4 v = *(const float4 *)p;
    x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
  }
};
template <>
struct Gran<bf16> {
  static constexpr int N = 8;
  __device__ __forceinline__ static void load(const bf16 *p, float (&x)[8]) {
    const bf16x8 v = *(const bf16x8 *)p;
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (float)v[j];
  }
};

// MAXJ: granules per lane of a score row (A <= 64 * MAXJ * Gran<T>::N)
template <typename T, int MAXJ>
__global__ __launch_bounds__(kAT) void attention_kernel(int B, int K, int S, int A, int Cd,
                                                        const T *__restrict__ P,
                                                        const T *__restrict__ Cx,
                                                        const float *__restrict__ mask,
                                                        const float *__restrict__ q, int ldq,
                                                        const float *__restrict__ va,
                                                        float *__restrict__ ctx_out, int ldc,
                                                        float *__restrict__ alpha_out) {
  constexpr int G = Gran<T>::N;
  __shared__ float es[kMaxS];
  __shared__ int vidx[kMaxS];
  __shared__ float stat[2];
  __shared__ int nvalid;
  const int m = xcd_remap(blockIdx.x, gridDim.x);
  const int b = m / K;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int ng = A / G;  // granules per P row

  // ---- compact the valid positions ----
  if (wave == 0) {
    const float *msk = mask + (size_t)b * S;
    int n = 0;
    for (int base = 0; base < S; base += 64) {
      const int i = base + lane;
      const bool ok = i < S && msk[i] != 0.f;
      const unsigned long long bal = __ballot(ok);
      const int pos = __popcll(bal & ((1ull << lane) - 1ull));
      if (ok) vidx[n + pos] = i;
      n += __popcll(bal);
    }
    if (lane == 0) nvalid = n;
  }

  float qr[MAXJ][G], vr[MAXJ][G];
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    const int g = j * 64 + lane;
#pragma unroll
    for (int e = 0; e < G; ++e) {
      qr[j][e] = g < ng ? q[(size_t)m * ldq + g * G + e] : 0.f;
      vr[j][e] = g < ng ? va[g * G + e] : 0.f;
    }
  }
  __syncthreads();
  const int n = nvalid;

  // ---- scores, two positions per wave iteration ----
  for (int j = wave; j < n; j += 8) {
    const bool two = j + 4 < n;
    const int i0 = vidx[j], i1 = two ? vidx[j + 4] : i0;
    const T *P0 = P + ((size_t)b * S + i0) * A;
    const T *P1 = P + ((size_t)b * S + i1) * A;
    float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
    for (int jj = 0; jj < MAXJ; ++jj) {
      const int g = jj * 64 + lane;
      if (g < ng) {
        float x0[G], x1[G];
        Gran<T>::load(P0 + g * G, x0);
        Gran<T>::load(P1 + g * G, x1);
#pragma unroll
        for (int e = 0; e < G; ++e) {
          acc0 += vr[jj][e] * tanh_fast(x0[e] + qr[jj][e]);
          acc1 += vr[jj][e] * tanh_fast(x1[e] + qr[jj][e]);
        }
      }
    }
    acc0 = wave_sum(acc0);
    acc1 = wave_sum(acc1);
    if (lane == 0) {
      es[j] = acc0;
      if (two) es[j + 4] = acc1;
    }
  }
  __syncthreads();

  // ---- masked softmax over the compacted scores (wave 0) ----
  if (wave == 0) {
    float mx = -INFINITY;
    for (int j = lane; j < n; j += 64) mx = fmaxf(mx, es[j]);
    mx = wave_max(mx);
    float s = 0.f;
    for (int j = lane; j < n; j += 64) s += exp_fast(es[j] - mx);
    s = wave_sum(s);
    if (lane == 0) {
      stat[0] = mx;
      stat[1] = s > 0.f ? 1.0f / s : 0.f;
    }
  }
  __syncthreads();
  {
    const float mx = stat[0], inv = stat[1];
    for (int j = t; j < n; j += kAT) es[j] = exp_fast(es[j] - mx) * inv;
    if (alpha_out)
      for (int i = t; i < S; i += kAT) alpha_out[(size_t)m * S + i] = 0.f;
  }
  __syncthreads();
  if (alpha_out)
    for (int j = t; j < n; j += kAT) alpha_out[(size_t)m * S + vidx[j]] = es[j];

  // ---- context: granules g of the C columns, four positions per iteration ----
  const int ncg = Cd / G;
  const T *Cb = Cx + (size_t)b * S * Cd;
  for (int g = t; g < ncg; g += kAT) {
    float c[G];
#pragma unroll
    for (int e = 0; e < G; ++e) c[e] = 0.f;
    int j = 0;
    for (; j + 4 <= n; j += 4) {
      float x[4][G];
#pragma unroll
      for (int u = 0; u < 4; ++u) Gran<T>::load(Cb + (size_t)vidx[j + u] * Cd + g * G, x[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float al = es[j + u];
#pragma unroll
        for (int e = 0; e < G; ++e) c[e] += al * x[u][e];
      }
    }
    for (; j < n; ++j) {
      float x[G];
      Gran<T>::load(Cb + (size_t)vidx[j] * Cd + g * G, x);
      const float al = es[j];
#pragma unroll
      for (int e = 0; e < G; ++e) c[e] += al * x[e];
    }
    float *o = ctx_out + (size_t)m * ldc + g * G;
#pragma unroll
    for (int e = 0; e < G; e += 4) *(float4 *)(o + e) = make_float4(c[e], c[e + 1], c[e + 2], c[e + 3]);
  }
}

template <typename T>
static void attn_go(int B, int K, int S, int A, int Cd, const T *P, const T *Cx, const float *mask,
                    const float *q, int ldq, const float *va, float *ctx_out, int ldc,
                    float *alpha_out, hipStream_t st) {
  const int M = B * K;
  const int j = (A / Gran<T>::N + 63) / 64;
#define MT_AT(N)                                                                                    \
  hipLaunchKernelGGL((attention_kernel<T, N>), dim3(M), dim3(kAT), 0, st, B, K, S, A, Cd, P, Cx,    \
                     mask, q, ldq, va, ctx_out, ldc, alpha_out)
  if (j <= 1) MT_AT(1);
  else if (j <= 2) MT_AT(2);
  else if (j <= 4) MT_AT(4);
  else if (j <= 8) MT_AT(8);
  else MT_AT(16);
#undef MT_AT
}

hipError_t launch_attention(int B, int K, int S, int A, int Cd, const void *P, const void *Cx,
                            int bf16_io, const float *mask, const float *q, int ldq,
                            const float *va, float *ctx_out, int ldc, float *alpha_out,
                            hipStream_t st) {
  if (B * K == 0) return hipSuccess;
  if (bf16_io)
    attn_go<bf16>(B, K, S, A, Cd, (const bf16 *)P, (const bf16 *)Cx, mask, q, ldq, va, ctx_out, ldc, alpha_out, st);
  else
    attn_go<float>(B, K, S, A, Cd, (const float *)P, (const float *)Cx, mask, q, ldq, va, ctx_out, ldc, alpha_out, st);
  return hipGetLastError();
}

}  // namespace mt
