// Row-wise kernels of the decoder step: the GRU cell update (with per-block layer
// normalisation), the readout (sum of three projections, layer norm, tanh), the masked
// mean of the encoder context (start state), and the log-sum-exp merge of the
// vocabulary partials (optionally turning stored logits into log-probabilities).
//
// One 256-thread workgroup per row; each thread keeps its NPT elements per block in
// registers.  Layer-norm statistics are two-pass (mean, then mean squared deviation)
// over register-resident values: wave shuffles, then 4 partials through LDS.
#include "mt_internal.h"

namespace mt {

constexpr int kT = 256;

// sum of NV values over the 256-thread block; every thread receives the totals
template <int NV>
__device__ __forceinline__ void block_sum(float (&v)[NV], float (*red)[NV]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = wave_sum(v[i]);
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) red[wave][i] = v[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = red[0][i] + red[1][i] + red[2][i] + red[3][i];
  __syncthreads();
}

// GRU cell (reset applied to the recurrent product, z gates the previous state):
//   r = sig(a_r + u_r), z = sig(a_z + u_z), hh = tanh(a_h + r u_h), out = (1-z) hh + z h
// a and u hold the three H-blocks (r, z, h) of the input and recurrent products; with
// layer norm each of the six blocks is normalised on its own before the gates.
template <int NPT, bool LN>
__global__ __launch_bounds__(kT) void gru_cell_kernel(int M, int H, const float *__restrict__ a, int lda,
                                                      const float *__restrict__ u, int ldu,
                                                      const float *__restrict__ hsrc,
                                                      const int32_t *__restrict__ hidx, int hrows,
                                                      int32_t *err, const float *__restrict__ ga,
                                                      const float *__restrict__ ba,
                                                      const float *__restrict__ gu,
                                                      const float *__restrict__ bu, float eps,
                                                      float *__restrict__ out, int ldo,
                                                      float *__restrict__ tap) {
  __shared__ float red[4][6];
  const int m = blockIdx.x;
  const int t = threadIdx.x;
  int hr = m;
  if (hidx) {
    hr = hidx[m];
    if (hr < 0 || hr >= hrows) {
      if (t == 0 && err) atomicOr(err, 2);
      hr = hr < 0 ? 0 : hrows - 1;
    }
  }
  const float *ar = a + (size_t)m * lda;
  const float *ur = u + (size_t)m * ldu;
  const float *hp = hsrc + (size_t)hr * H;
  float x[6][NPT], h[NPT];
#pragma unroll
  for (int p = 0; p < NPT; ++p) {
    const int j = t + kT * p;
    const bool ok = j < H;
#pragma unroll
    for (int g = 0; g < 3; ++g) {
      x[g][p] = ok ? ar[g * H + j] : 0.f;
      x[3 + g][p] = ok ? ur[g * H + j] : 0.f;
    }
    h[p] = ok ? hp[j] : 0.f;
  }
  if (LN) {
    float s[6];
#pragma unroll
    for (int g = 0; g < 6; ++g) {
      s[g] = 0.f;
#pragma unroll
      for (int p = 0; p < NPT; ++p) s[g] += x[g][p];
    }
    block_sum<6>(s, red);
    float mean[6], d[6];
#pragma unroll
    for (int g = 0; g < 6; ++g) {
      mean[g] = s[g] / (float)H;
      d[g] = 0.f;
#pragma unroll
      for (int p = 0; p < NPT; ++p) {
        const int j = t + kT * p;
        const float e = j < H ? x[g][p] - mean[g] : 0.f;
        d[g] += e * e;
      }
    }
    block_sum<6>(d, red);
#pragma unroll
    for (int g = 0; g < 6; ++g) {
      const float inv = 1.0f / sqrtf(d[g] / (float)H + eps);
      const float *gg = g < 3 ? ga + g * H : gu + (g - 3) * H;
      const float *bb = g < 3 ? ba + g * H : bu + (g - 3) * H;
#pragma unroll
      for (int p = 0; p < NPT; ++p) {
        const int j = t + kT * p;
        if (j < H) x[g][p] = gg[j] * (x[g][p] - mean[g]) * inv + bb[j];
      }
    }
  }
  float *o = out + (size_t)m * ldo;
#pragma unroll
  for (int p = 0; p < NPT; ++p) {
    const int j = t + kT * p;
    if (j >= H) continue;
    const float r = sigmoid_fast(x[0][p] + x[3][p]);
    const float z = sigmoid_fast(x[1][p] + x[4][p]);
    const float hh = tanh_fast(x[2][p] + r * x[5][p]);
    const float v = (1.0f - z) * hh + z * h[p];
    o[j] = v;
    if (tap) tap[(size_t)m * H + j] = v;
  }
}

// t = tanh(LN?(p1 + p2 + p3 + bt)), written in the vocabulary GEMM's operand type
template <int NPT, bool LN, typename TO>
__global__ __launch_bounds__(kT) void readout_kernel(int M, int E, const float *__restrict__ p1, int ld1,
                                                     const float *__restrict__ p2, int ld2,
                                                     const float *__restrict__ p3, int ld3,
                                                     const float *__restrict__ bt,
                                                     const float *__restrict__ g,
                                                     const float *__restrict__ be, float eps,
                                                     TO *__restrict__ tout, float *__restrict__ tap) {
  __shared__ float red[4][1];
  const int m = blockIdx.x, t = threadIdx.x;
  float x[NPT];
  float s[1] = {0.f};
#pragma unroll
  for (int p = 0; p < NPT; ++p) {
    const int j = t + kT * p;
    x[p] = j < E ? p1[(size_t)m * ld1 + j] + p2[(size_t)m * ld2 + j] + p3[(size_t)m * ld3 + j] + bt[j] : 0.f;
    s[0] += x[p];
  }
  if (LN) {
    block_sum<1>(s, red);
    const float mean = s[0] / (float)E;
    float d[1] = {0.f};
#pragma unroll
    for (int p = 0; p < NPT; ++p) {
      const int j = t + kT * p;
      const float e = j < E ? x[p] - mean : 0.f;
      d[0] += e * e;
    }
    block_sum<1>(d, red);
    const float inv = 1.0f / sqrtf(d[0] / (float)E + eps);
#pragma unroll
    for (int p = 0; p < NPT; ++p) {
      const int j = t + kT * p;
      if (j < E) x[p] = g[j] * (x[p] - mean) * inv + be[j];
    }
  }
#pragma unroll
  for (int p = 0; p < NPT; ++p) {
    const int j = t + kT * p;
    if (j >= E) continue;
    const float v = tanh_fast(x[p]);
    Store<TO>::put(tout + (size_t)m * E + j, v);
    if (tap) tap[(size_t)m * E + j] = v;
  }
}

// cbar[b, c] = mean over valid positions i of ctx[b, i, c] (0 if none are valid)
template <typename T>
__global__ __launch_bounds__(kT) void masked_mean_kernel(int B, int S, int Cd, const T *__restrict__ ctx,
                                                         const float *__restrict__ mask,
                                                         float *__restrict__ out) {
  const int b = blockIdx.y;
  const int c = blockIdx.x * kT + threadIdx.x;
  if (c >= Cd) return;
  float acc = 0.f;
  int n = 0;
  for (int i = 0; i < S; ++i) {
    if (mask[(size_t)b * S + i] == 0.f) continue;
    acc += to_f32(ctx[((size_t)b * S + i) * Cd + c]);
    ++n;
  }
  out[(size_t)b * Cd + c] = n ? acc / (float)n : 0.f;
}

// LSE over the (max, sum exp) partials of one row: L = M + log(sum_t s_t exp(m_t - M)).
// With `logits`, the row's stored logits become logits - L in place.
__global__ __launch_bounds__(kT) void lse_kernel(int M, int ntiles, const float2 *__restrict__ part,
                                                 float *__restrict__ lse, float *__restrict__ logits,
                                                 int V) {
  __shared__ float red[4][1];
  const int m = blockIdx.x, t = threadIdx.x;
  const float2 *pr = part + (size_t)m * ntiles;
  float mx = -INFINITY;
  for (int i = t; i < ntiles; i += kT) mx = fmaxf(mx, pr[i].x);
  mx = wave_max(mx);
  __shared__ float wmx[4];
  if ((t & 63) == 0) wmx[t >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(wmx[0], wmx[1]), fmaxf(wmx[2], wmx[3]));
  float s[1] = {0.f};
  for (int i = t; i < ntiles; i += kT) {
    const float2 q = pr[i];
    s[0] += q.y * exp_fast(q.x - mx);
  }
  block_sum<1>(s, red);
  const float L = mx + __builtin_amdgcn_logf(s[0]) * 0.6931471805599453f;
  if (t == 0) lse[m] = L;
  if (logits) {
    float *row = logits + (size_t)m * V;
    for (int v = t; v < V; v += kT) row[v] = row[v] - L;
  }
}

// ---------------------------------------------------------------------------------------

static int npt_for(int n) {
  const int q = (n + kT - 1) / kT;
  return q <= 1 ? 1 : q <= 2 ? 2 : q <= 4 ? 4 : q <= 8 ? 8 : 16;
}

hipError_t launch_gru_cell(int M, int H, const float *a, int lda, const float *u, int ldu,
                           const float *hsrc, const int32_t *hidx, int hrows, int32_t *err,
                           const float *ga, const float *ba, const float *gu, const float *bu,
                           float eps, float *out, int ldo, float *tap, hipStream_t st) {
  if (M == 0) return hipSuccess;
  const bool ln = ga != nullptr;
#define MT_GRU(N)                                                                                       \
  if (ln)                                                                                               \
    hipLaunchKernelGGL((gru_cell_kernel<N, true>), dim3(M), dim3(kT), 0, st, M, H, a, lda, u, ldu,      \
                       hsrc, hidx, hrows, err, ga, ba, gu, bu, eps, out, ldo, tap);                     \
  else                                                                                                  \
    hipLaunchKernelGGL((gru_cell_kernel<N, false>), dim3(M), dim3(kT), 0, st, M, H, a, lda, u, ldu,     \
                       hsrc, hidx, hrows, err, ga, ba, gu, bu, eps, out, ldo, tap);
  switch (npt_for(H)) {
    case 1: MT_GRU(1) break;
    case 2: MT_GRU(2) break;
    case 4: MT_GRU(4) break;
    case 8: MT_GRU(8) break;
    default: MT_GRU(16) break;
  }
#undef MT_GRU
  return hipGetLastError();
}

template <typename TO>
static void readout_go(int npt, bool ln, int M, int E, const float *p1, int ld1, const float *p2,
                       int ld2, const float *p3, int ld3, const float *bt, const float *g,
                       const float *be, float eps, TO *t, float *tap, hipStream_t st) {
#define MT_RO(N)                                                                                      \
  if (ln)                                                                                             \
    hipLaunchKernelGGL((readout_kernel<N, true, TO>), dim3(M), dim3(kT), 0, st, M, E, p1, ld1, p2,    \
                       ld2, p3, ld3, bt, g, be, eps, t, tap);                                         \
  else                                                                                                \
    hipLaunchKernelGGL((readout_kernel<N, false, TO>), dim3(M), dim3(kT), 0, st, M, E, p1, ld1, p2,   \
                       ld2, p3, ld3, bt, g, be, eps, t, tap);
  switch (npt) {
    case 1: MT_RO(1) break;
    case 2: MT_RO(2) break;
    case 4: MT_RO(4) break;
    case 8: MT_RO(8) break;
    default: MT_RO(16) break;
  }
#undef MT_RO
}

hipError_t launch_readout(int M, int E, const float *p1, int ld1, const float *p2, int ld2,
                          const float *p3, int ld3, const float *bt, const float *g,
                          const float *be, float eps, void *t_out, int t_bf16, float *tap,
                          hipStream_t st) {
  if (M == 0) return hipSuccess;
  const bool ln = g != nullptr;
  if (t_bf16)
    readout_go<bf16>(npt_for(E), ln, M, E, p1, ld1, p2, ld2, p3, ld3, bt, g, be, eps, (bf16 *)t_out, tap, st);
  else
    readout_go<float>(npt_for(E), ln, M, E, p1, ld1, p2, ld2, p3, ld3, bt, g, be, eps, (float *)t_out, tap, st);
  return hipGetLastError();
}

hipError_t launch_masked_mean(int B, int S, int Cd, const void *ctx, int ctx_bf16,
                              const float *mask, float *out, hipStream_t st) {
  if (B == 0) return hipSuccess;
  dim3 grid((Cd + kT - 1) / kT, B);
  if (ctx_bf16)
    hipLaunchKernelGGL(masked_mean_kernel<bf16>, grid, dim3(kT), 0, st, B, S, Cd, (const bf16 *)ctx, mask, out);
  else
    hipLaunchKernelGGL(masked_mean_kernel<float>, grid, dim3(kT), 0, st, B, S, Cd, (const float *)ctx, mask, out);
  return hipGetLastError();
}

hipError_t launch_lse(int M, int ntiles, const float2 *part, float *lse, float *logits, int V,
                      hipStream_t st) {
  if (M == 0) return hipSuccess;
  hipLaunchKernelGGL(lse_kernel, dim3(M), dim3(kT), 0, st, M, ntiles, part, lse, logits, V);
  return hipGetLastError();
}

}  // namespace mt
