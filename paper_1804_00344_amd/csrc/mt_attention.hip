// Additive attention with a masked softmax over the source positions of one sentence,
// one 256-thread workgroup per hypothesis row (m = b*K + k):
//   e_i   = sum_a va[a] * tanh(P[b,i,a] + q[m,a])      (valid i only)
//   alpha = exp(e_i - max_valid e) / sum_valid exp(...)  (exactly 0 at masked i)
//   c[m]  = sum_valid alpha_i * Cx[b,i,:]
// Scores: each wave takes positions i = wave, wave+4, ...; its 64 lanes stream the A
// features of P[b,i] in coalesced 4-element granules against q and va held in
// registers, and reduce with cross-lane shuffles.  Softmax: one wave over the S scores
// kept in LDS.  Context: each thread owns 4-column granules of C and walks the valid
// positions, reading rows of Cx[b] coalesced.  Masked positions of P and Cx are never
// read.  Workgroup ids are remapped so that the K rows of one sentence run on one XCD
// and share its L2 copy of P[b] and Cx[b].
#include "mt_internal.h"

namespace mt {

constexpr int kAT = 256;
constexpr int kMaxS = 1024;

template <typename T>
struct Vec4;
template <>
struct Vec4<float> {
  __device__ __forceinline__ static float4 load(const float *p) { return *(const float4 *)p; }
};
template <>
struct Vec4<bf16> {
  __device__ __forceinline__ static float4 load(const bf16 *p) {
    typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
    const bf16x4 v = *(const bf16x4 *)p;
    return make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
  }
};

// MAXJ: granules of 4 features per lane (A <= 256 * MAXJ)
template <typename T, int MAXJ>
__global__ __launch_bounds__(kAT) void attention_kernel(int B, int K, int S, int A, int Cd,
                                                        const T *__restrict__ P,
                                                        const T *__restrict__ Cx,
                                                        const float *__restrict__ mask,
                                                        const float *__restrict__ q, int ldq,
                                                        const float *__restrict__ va,
                                                        float *__restrict__ ctx_out, int ldc,
                                                        float *__restrict__ alpha_out) {
  __shared__ float es[kMaxS];
  __shared__ float stat[2];
  const int m = xcd_remap(blockIdx.x, gridDim.x);
  const int b = m / K;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int ng = A >> 2;  // granules of 4 features
  const float *msk = mask + (size_t)b * S;

  float4 qr[MAXJ], vr[MAXJ];
#pragma unroll
  for (int j = 0; j < MAXJ; ++j) {
    const int g = j * 64 + lane;
    if (g < ng) {
      qr[j] = *(const float4 *)(q + (size_t)m * ldq + 4 * g);
      vr[j] = *(const float4 *)(va + 4 * g);
    } else {
      qr[j] = make_float4(0.f, 0.f, 0.f, 0.f);
      vr[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }

  // ---- scores ----
  for (int i = wave; i < S; i += 4) {
    if (msk[i] == 0.f) continue;  // uniform over the wave
    const T *Pr = P + ((size_t)b * S + i) * A;
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < MAXJ; ++j) {
      const int g = j * 64 + lane;
      if (g < ng) {
        const float4 p = Vec4<T>::load(Pr + 4 * g);
        acc += vr[j].x * tanh_fast(p.x + qr[j].x);
        acc += vr[j].y * tanh_fast(p.y + qr[j].y);
        acc += vr[j].z * tanh_fast(p.z + qr[j].z);
        acc += vr[j].w * tanh_fast(p.w + qr[j].w);
      }
    }
    acc = wave_sum(acc);
    if (lane == 0) es[i] = acc;
  }
  __syncthreads();

  // ---- masked softmax (wave 0) ----
  if (wave == 0) {
    float mx = -INFINITY;
    for (int i = lane; i < S; i += 64)
      if (msk[i] != 0.f) mx = fmaxf(mx, es[i]);
    mx = wave_max(mx);
    float s = 0.f;
    for (int i = lane; i < S; i += 64)
      if (msk[i] != 0.f) s += exp_fast(es[i] - mx);
    s = wave_sum(s);
    if (lane == 0) {
      stat[0] = mx;
      stat[1] = s > 0.f ? 1.0f / s : 0.f;
    }
  }
  __syncthreads();
  const float mx = stat[0], inv = stat[1];
  for (int i = t; i < S; i += kAT) {
    const float a = msk[i] != 0.f ? exp_fast(es[i] - mx) * inv : 0.f;
    es[i] = a;  // each i is owned by one thread: read then overwrite
    if (alpha_out) alpha_out[(size_t)m * S + i] = a;
  }
  __syncthreads();

  // ---- context ----
  const int ncg = Cd >> 2;
  for (int g0 = t; g0 < ncg; g0 += kAT * 2) {
    const int g1 = g0 + kAT;
    float4 c0 = make_float4(0.f, 0.f, 0.f, 0.f), c1 = c0;
    for (int i = 0; i < S; ++i) {
      if (msk[i] == 0.f) continue;
      const float a = es[i];
      const T *Cr = Cx + ((size_t)b * S + i) * Cd;
      const float4 x0 = Vec4<T>::load(Cr + 4 * g0);
      c0.x += a * x0.x; c0.y += a * x0.y; c0.z += a * x0.z; c0.w += a * x0.w;
      if (g1 < ncg) {
        const float4 x1 = Vec4<T>::load(Cr + 4 * g1);
        c1.x += a * x1.x; c1.y += a * x1.y; c1.z += a * x1.z; c1.w += a * x1.w;
      }
    }
    *(float4 *)(ctx_out + (size_t)m * ldc + 4 * g0) = c0;
    if (g1 < ncg) *(float4 *)(ctx_out + (size_t)m * ldc + 4 * g1) = c1;
  }
}

template <typename T>
static void attn_go(int B, int K, int S, int A, int Cd, const T *P, const T *Cx, const float *mask,
                    const float *q, int ldq, const float *va, float *ctx_out, int ldc,
                    float *alpha_out, hipStream_t st) {
  const int M = B * K;
  const int j = (A / 4 + 63) / 64;
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
