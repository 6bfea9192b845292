// Row-wise kernels of the decoder step: the GRU cell update (with per-block layer
// normalisation), the readout (sum of three projections, layer norm, tanh), the masked
// mean of the encoder context (start state), and the log-sum-exp merge of the
// vocabulary partials (optionally turning stored logits into log-probabilities).
//
// GRU cell and readout: one 256-thread workgroup per row; thread t holds 16-byte granules
// 4t + 1024p of each H-block in registers, and every operand (products, previous state,
// layer-norm gains and shifts) is loaded up front so the row costs one memory round trip
// (the row indices of gathered operands are read together before it).  Layer-norm
// statistics need one workgroup barrier: each wave takes the mean of its own values and the
// sum of their squared deviations from it (two DPP reductions over registers, no
// cancellation), and the four waves' (count, mean, squared deviations) are combined through
// LDS with the pairwise update of Chan, Golub and LeVeque:
//   mean = sum_w n_w m_w / n,   M2 = sum_w (M2_w + n_w (m_w - mean)^2).
#include "mt_internal.h"

namespace mt {

constexpr int kT = 256;

// Layer-norm statistics of NB blocks of n values each, thread t holding elements 4t + 1024p
// (p < G) of every block as x(g, p, e): on return mean[g] and inv[g] = 1/sqrt(var + eps)
// (population variance), in every thread.  One barrier; `red` is used once.
template <int NB, int G, typename X>
__device__ __forceinline__ void ln_stats(X x, int n, float eps, float (*red)[2][NB], float (&mean)[NB],
                                         float (&inv)[NB]) {
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  auto wave_count = [&](int w) {  // values held by wave w
    int c = 0;
#pragma unroll
    for (int p = 0; p < G; ++p) {
      const int r = n - 4 * kT * p - 256 * w;
      c += r <= 0 ? 0 : r < 256 ? r : 256;
    }
    return c;
  };
  const int nw = wave_count(wv);
  const float rn = nw ? 1.0f / (float)nw : 0.f;
  float wm[NB], wq[NB];
#pragma unroll
  for (int g = 0; g < NB; ++g) {
    float s1 = 0.f;
#pragma unroll
    for (int p = 0; p < G; ++p) {
      const bool ok = 4 * t + 4 * kT * p < n;
#pragma unroll
      for (int e = 0; e < 4; ++e) s1 += ok ? x(g, p, e) : 0.f;
    }
    wm[g] = wave_sum(s1) * rn;
  }
#pragma unroll
  for (int g = 0; g < NB; ++g) {
    float s2 = 0.f;
#pragma unroll
    for (int p = 0; p < G; ++p) {
      const bool ok = 4 * t + 4 * kT * p < n;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float d = x(g, p, e) - wm[g];
        s2 += ok ? d * d : 0.f;
      }
    }
    wq[g] = wave_sum(s2);
  }
  if (lane == 0) {
#pragma unroll
    for (int g = 0; g < NB; ++g) {
      red[wv][0][g] = wm[g];
      red[wv][1][g] = wq[g];
    }
  }
  __syncthreads();
  float cn[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) cn[w] = (float)wave_count(w);
  const float invn = 1.0f / (float)n;
#pragma unroll
  for (int g = 0; g < NB; ++g) {
    float mu = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) mu += cn[w] * red[w][0][g];
    mu *= invn;
    float m2 = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float d = red[w][0][g] - mu;
      m2 += red[w][1][g] + cn[w] * d * d;
    }
    mean[g] = mu;
    inv[g] = 1.0f / sqrtf(m2 * invn + eps);
  }
}

// Row index idx[m] clamped to [0, rows); an out-of-range index sets error bit `bit`
__device__ __forceinline__ int clamp_idx(int r, int rows, int32_t *err, int bit) {
  if (r < 0 || r >= rows) {
    if (threadIdx.x == 0 && err) atomicOr(err, 1 << bit);
    r = r < 0 ? 0 : rows - 1;
  }
  return r;
}

__device__ __forceinline__ float4 ld4(const float *p) { return *(const float4 *)p; }
__device__ __forceinline__ void st4(float *p, float a, float b, float c, float d) {
  *(float4 *)p = make_float4(a, b, c, d);
}

__device__ __forceinline__ int clamp_row(const int32_t *idx, int m, int rows, int32_t *err, int bit) {
  int r = idx[m];
  if (r < 0 || r >= rows) {
    if (threadIdx.x == 0 && err) atomicOr(err, 1 << bit);
    r = r < 0 ? 0 : rows - 1;
  }
  return r;
}

// GRU cell (reset applied to the recurrent product, z gates the previous state):
//   r = sig(a_r + u_r), z = sig(a_z + u_z), hh = tanh(a_h + r u_h), out = (1-z) hh + z h
// a and u hold the three H-blocks (r, z, h) of the input and recurrent products; with
// layer norm each of the six blocks is normalised on its own before the gates.  Row m
// reads a from row aidx[m] (if given; error bit 0 on a clamp) and the previous state from
// row hidx[m] (if given; error bit 1).  G = 16-byte granules per thread per block.
// LNM: 0 no layer norm; 1 on all six blocks; 2 on the recurrent blocks only (a transition
// block of a deep-transition cell: a is its bias row, read with lda = 0).
template <int G, int LNM>
__global__ __launch_bounds__(kT) void gru_cell_kernel(int M, int H, const float *__restrict__ a, int lda,
                                                      const int32_t *__restrict__ aidx, int arows,
                                                      const float *__restrict__ u, int ldu,
                                                      const float *__restrict__ hsrc,
                                                      const int32_t *__restrict__ hidx, int hrows,
                                                      int32_t *err, const float *__restrict__ ga,
                                                      const float *__restrict__ ba,
                                                      const float *__restrict__ gu,
                                                      const float *__restrict__ bu, float eps,
                                                      float *__restrict__ out, int ldo,
                                                      bf16 *__restrict__ out16,
                                                      float *__restrict__ tap, int ldh, int ld16,
                                                      const float *__restrict__ keep, int keep_ld,
                                                      CellPair pr) {
  constexpr bool LN = LNM != 0;
  constexpr int G0 = LNM == 2 ? 3 : 0;  // first normalised block
  constexpr int NB = 6 - G0;            // normalised blocks
  __shared__ float red[4][2][NB];
  const int m = blockIdx.x;
  const int t = threadIdx.x;
  if (blockIdx.y) {  // the launch's second cell
    a += pr.da;
    u += pr.du;
    if (hsrc) hsrc += pr.dh;
    out += pr.dout;
    if (out16) out16 += pr.d16;
    if (keep) keep += pr.dkeep;
    if (ga) ga += pr.dln, ba += pr.dln;
    if (gu) gu += pr.dln, bu += pr.dln;
  }
  float x[6][G][4], h[G][4];
  float lg[6][G][4], lb[6][G][4];
  // the operands that do not depend on a row index are requested first, so that the index
  // loads' round trip runs under them
  const float *urow = u + (size_t)m * ldu;
#pragma unroll
  for (int p = 0; p < G; ++p) {
    const int j = 4 * t + 4 * kT * p;
    const int jc = j < H ? j : 0;  // lanes past H read element 0 and take no part
#pragma unroll
    for (int g = 0; g < 3; ++g) {
      const float4 vu = ld4(urow + g * H + jc);
      x[3 + g][p][0] = vu.x; x[3 + g][p][1] = vu.y; x[3 + g][p][2] = vu.z; x[3 + g][p][3] = vu.w;
      if (LNM == 1) {
        const float4 g0 = ld4(ga + g * H + jc), b0 = ld4(ba + g * H + jc);
        lg[g][p][0] = g0.x; lg[g][p][1] = g0.y; lg[g][p][2] = g0.z; lg[g][p][3] = g0.w;
        lb[g][p][0] = b0.x; lb[g][p][1] = b0.y; lb[g][p][2] = b0.z; lb[g][p][3] = b0.w;
      }
      if (LN) {
        const float4 g1 = ld4(gu + g * H + jc), b1 = ld4(bu + g * H + jc);
        lg[3 + g][p][0] = g1.x; lg[3 + g][p][1] = g1.y; lg[3 + g][p][2] = g1.z; lg[3 + g][p][3] = g1.w;
        lb[3 + g][p][0] = b1.x; lb[3 + g][p][1] = b1.y; lb[3 + g][p][2] = b1.z; lb[3 + g][p][3] = b1.w;
      }
    }
  }
  // both row indices and the keep flag are requested before any of them is used
  int ar = m, hr = m;
  if (aidx) ar = aidx[m];
  if (hidx) hr = hidx[m];
  // keep (if given): a row whose keep value is 0 carries its previous state over
  const bool upd = keep == nullptr || keep[(size_t)m * keep_ld] != 0.f;
  if (aidx) ar = clamp_idx(ar, arows, err, 0);
  if (hidx) hr = clamp_idx(hr, hrows, err, 1);
  const float *arow = a + (size_t)ar * lda;
  const float *hp = hsrc ? hsrc + (size_t)hr * ldh : nullptr;  // no previous state: zero
#pragma unroll
  for (int p = 0; p < G; ++p) {
    const int j = 4 * t + 4 * kT * p;
    const int jc = j < H ? j : 0;
#pragma unroll
    for (int g = 0; g < 3; ++g) {
      const float4 va = ld4(arow + g * H + jc);
      x[g][p][0] = va.x; x[g][p][1] = va.y; x[g][p][2] = va.z; x[g][p][3] = va.w;
    }
    const float4 vh = hp ? ld4(hp + jc) : make_float4(0.f, 0.f, 0.f, 0.f);
    h[p][0] = vh.x; h[p][1] = vh.y; h[p][2] = vh.z; h[p][3] = vh.w;
  }
  if (LN) {
    float mean[NB], inv[NB];
    ln_stats<NB, G>([&](int g, int p, int e) { return x[G0 + g][p][e]; }, H, eps, red, mean, inv);
#pragma unroll
    for (int g = 0; g < NB; ++g)
#pragma unroll
      for (int p = 0; p < G; ++p)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          x[G0 + g][p][e] = lg[G0 + g][p][e] * (x[G0 + g][p][e] - mean[g]) * inv[g] + lb[G0 + g][p][e];
  }
  float *o = out + (size_t)m * ldo;
#pragma unroll
  for (int p = 0; p < G; ++p) {
    const int j = 4 * t + 4 * kT * p;
    if (j >= H) continue;
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float r = sigmoid_fast(x[0][p][e] + x[3][p][e]);
      const float z = sigmoid_fast(x[1][p][e] + x[4][p][e]);
      const float hh = tanh_fast(x[2][p][e] + r * x[5][p][e]);
      v[e] = upd ? (1.0f - z) * hh + z * h[p][e] : h[p][e];
    }
    st4(o + j, v[0], v[1], v[2], v[3]);
    if (out16) {  // bf16 copy for a following bf16 product (same rounding as its operand staging)
      bf16 h4[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) h4[e] = to_bf16(v[e]);
      __builtin_memcpy(out16 + (size_t)m * ld16 + j, h4, sizeof(h4));
    }
    if (tap) st4(tap + (size_t)m * H + j, v[0], v[1], v[2], v[3]);
  }
}

// t = tanh(LN?(p1 + p2 + p3 + bt)), written in the vocabulary GEMM's operand type; row m
// reads p2 from row idx2[m] (if given, clamped)
template <int G, bool LN, typename TO>
__global__ __launch_bounds__(kT) void readout_kernel(int M, int E, const float *__restrict__ p1, int ld1,
                                                     const float *__restrict__ p2, int ld2,
                                                     const int32_t *__restrict__ idx2, int rows2,
                                                     const float *__restrict__ p3, int ld3,
                                                     const float *__restrict__ bt,
                                                     const float *__restrict__ g,
                                                     const float *__restrict__ be, float eps,
                                                     TO *__restrict__ tout, float *__restrict__ tap) {
  __shared__ float red[4][2][1];
  const int m = blockIdx.x, t = threadIdx.x;
  const int r2 = idx2 ? clamp_row(idx2, m, rows2, nullptr, 0) : m;
  const float *q1 = p1 + (size_t)m * ld1, *q2 = p2 + (size_t)r2 * ld2, *q3 = p3 + (size_t)m * ld3;
  float x[G][4], lg[G][4], lb[G][4];
#pragma unroll
  for (int p = 0; p < G; ++p) {
    const int j = 4 * t + 4 * kT * p;
    const int jc = j < E ? j : 0;
    const float4 a = ld4(q1 + jc), b = ld4(q2 + jc), c = ld4(q3 + jc), d = ld4(bt + jc);
    x[p][0] = a.x + b.x + c.x + d.x;
    x[p][1] = a.y + b.y + c.y + d.y;
    x[p][2] = a.z + b.z + c.z + d.z;
    x[p][3] = a.w + b.w + c.w + d.w;
    if (LN) {
      const float4 g0 = ld4(g + jc), b0 = ld4(be + jc);
      lg[p][0] = g0.x; lg[p][1] = g0.y; lg[p][2] = g0.z; lg[p][3] = g0.w;
      lb[p][0] = b0.x; lb[p][1] = b0.y; lb[p][2] = b0.z; lb[p][3] = b0.w;
    }
  }
  if (LN) {
    float mean[1], inv[1];
    ln_stats<1, G>([&](int, int p, int e) { return x[p][e]; }, E, eps, red, mean, inv);
#pragma unroll
    for (int p = 0; p < G; ++p)
#pragma unroll
      for (int e = 0; e < 4; ++e) x[p][e] = lg[p][e] * (x[p][e] - mean[0]) * inv[0] + lb[p][e];
  }
#pragma unroll
  for (int p = 0; p < G; ++p) {
    const int j = 4 * t + 4 * kT * p;
    if (j >= E) continue;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float v = tanh_fast(x[p][e]);
      Store<TO>::put(tout + (size_t)m * E + j + e, v);
      if (tap) tap[(size_t)m * E + j + e] = v;
    }
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
  // no branch on the mask: every row is loaded (in bounds) and masked rows are selected away,
  // so the loads of successive positions overlap
  float acc = 0.f;
  int n = 0;
#pragma unroll 8
  for (int i = 0; i < S; ++i) {
    const bool ok = mask[(size_t)b * S + i] != 0.f;
    const float x = to_f32(ctx[((size_t)b * S + i) * Cd + c]);
    acc += ok ? x : 0.f;
    n += ok ? 1 : 0;
  }
  out[(size_t)b * Cd + c] = n ? acc / (float)n : 0.f;
}

// Valid rows of a 0/1 mask in increasing order, by one workgroup: per 1024-entry chunk, wave
// ballots give each valid entry its rank within its wave and the wave totals (through LDS)
// its wave's offset.
__global__ __launch_bounds__(1024) void valid_rows_kernel(int n, const float *__restrict__ mask,
                                                         int32_t *__restrict__ idx, int *__restrict__ count) {
  __shared__ int wsum[16];
  __shared__ int base;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  if (t == 0) base = 0;
  __syncthreads();
  for (int c0 = 0; c0 < n; c0 += 1024) {
    const int i = c0 + t;
    const bool ok = i < n && mask[i] != 0.f;
    const unsigned long long bal = __ballot(ok);
    if (lane == 0) wsum[wave] = __popcll(bal);
    __syncthreads();
    int off = base;
    for (int w = 0; w < wave; ++w) off += wsum[w];
    if (ok) idx[off + __popcll(bal & ((1ull << lane) - 1ull))] = i;
    __syncthreads();
    if (t == 0) {
      int s = 0;
      for (int w = 0; w < 16; ++w) s += wsum[w];
      base += s;
    }
    __syncthreads();
  }
  if (t == 0) *count = base;
}

// LSE over the (max, sum exp) partials of one row: L = M + log(sum_t s_t exp(m_t - M)).
// With `logits`, the row's stored logits become logits - L in place.
__global__ __launch_bounds__(kT) void lse_kernel(int M, int ntiles, const float2 *__restrict__ part,
                                                 float *__restrict__ lse, float *__restrict__ logits,
                                                 int V) {
  const int m = blockIdx.x, t = threadIdx.x;
  const float L = block_row_lse(part + (size_t)m * ntiles, ntiles);
  if (t == 0) lse[m] = L;
  if (logits) {
    // 16-byte accesses over the aligned middle of the row, single elements at its ends
    float *row = logits + (size_t)m * V;
    const int mis = (int)(((uintptr_t)row & 15) / 4);  // floats past a 16-byte boundary
    const int head = ((4 - mis) & 3) < V ? ((4 - mis) & 3) : V;
    const int n4 = (V - head) / 4;
    if (t < head) row[t] = row[t] - L;
    float4 *r4 = (float4 *)(row + head);
    for (int i = t; i < n4; i += kT) {
      float4 x = r4[i];
      x.x -= L; x.y -= L; x.z -= L; x.w -= L;
      r4[i] = x;
    }
    for (int v = head + 4 * n4 + t; v < V; v += kT) row[v] = row[v] - L;
  }
}

// ---------------------------------------------------------------------------------------

static int gran_for(int n) {  // 16-byte granules per thread for an n-wide row
  const int q = (n / 4 + kT - 1) / kT;
  return q <= 1 ? 1 : q <= 2 ? 2 : 4;
}

hipError_t launch_gru_cell(int M, int H, const float *a, int lda, const int32_t *aidx, int arows,
                           const float *u, int ldu, const float *hsrc, const int32_t *hidx, int hrows,
                           int32_t *err, const float *ga, const float *ba, const float *gu, const float *bu,
                           float eps, float *out, int ldo, bf16 *out16, float *tap, hipStream_t st) {
  return launch_gru_cell_ex(M, H, a, lda, aidx, arows, u, ldu, hsrc, H, hidx, hrows, err, ga, ba, gu, bu, eps, out,
                            ldo, out16, H, tap, nullptr, 0, st);
}

hipError_t launch_gru_cell_ex(int M, int H, const float *a, int lda, const int32_t *aidx, int arows,
                              const float *u, int ldu, const float *hsrc, int ldh, const int32_t *hidx, int hrows,
                              int32_t *err, const float *ga, const float *ba, const float *gu, const float *bu,
                              float eps, float *out, int ldo, bf16 *out16, int ld16, float *tap,
                              const float *keep, int keep_ld, hipStream_t st, const CellPair *pair) {
  if (M == 0) return hipSuccess;
  if (pair && (tap || aidx || hidx)) return hipErrorInvalidValue;  // not offset by the pair
  const CellPair pr = pair ? *pair : CellPair{};
  const dim3 grid(M, pair ? 2 : 1);
  // layer norm on both paths (ga given), on the recurrent path only (gu alone), or none
  const int lnm = ga ? 1 : gu ? 2 : 0;
#define MT_GRU_L(N, L)                                                                                  \
  hipLaunchKernelGGL((gru_cell_kernel<N, L>), grid, dim3(kT), 0, st, M, H, a, lda, aidx, arows, u,     \
                     ldu, hsrc, hidx, hrows, err, ga, ba, gu, bu, eps, out, ldo, out16, tap, ldh, ld16,    \
                     keep, keep_ld, pr)
#define MT_GRU(N)              \
  if (lnm == 1)                \
    MT_GRU_L(N, 1);            \
  else if (lnm == 2)           \
    MT_GRU_L(N, 2);            \
  else                         \
    MT_GRU_L(N, 0);
  switch (gran_for(H)) {
    case 1: MT_GRU(1) break;
    case 2: MT_GRU(2) break;
    default: MT_GRU(4) break;
  }
#undef MT_GRU
#undef MT_GRU_L
  return hipGetLastError();
}

template <typename TO>
static void readout_go(int gr, bool ln, int M, int E, const float *p1, int ld1, const float *p2, int ld2,
                       const int32_t *idx2, int rows2, const float *p3, int ld3, const float *bt,
                       const float *g, const float *be, float eps, TO *t, float *tap, hipStream_t st) {
#define MT_RO(N)                                                                                      \
  if (ln)                                                                                             \
    hipLaunchKernelGGL((readout_kernel<N, true, TO>), dim3(M), dim3(kT), 0, st, M, E, p1, ld1, p2,    \
                       ld2, idx2, rows2, p3, ld3, bt, g, be, eps, t, tap);                            \
  else                                                                                                \
    hipLaunchKernelGGL((readout_kernel<N, false, TO>), dim3(M), dim3(kT), 0, st, M, E, p1, ld1, p2,   \
                       ld2, idx2, rows2, p3, ld3, bt, g, be, eps, t, tap);
  switch (gr) {
    case 1: MT_RO(1) break;
    case 2: MT_RO(2) break;
    default: MT_RO(4) break;
  }
#undef MT_RO
}

hipError_t launch_readout(int M, int E, const float *p1, int ld1, const float *p2, int ld2, const int32_t *idx2,
                          int rows2, const float *p3, int ld3, const float *bt, const float *g,
                          const float *be, float eps, void *t_out, int t_bf16, float *tap,
                          hipStream_t st) {
  if (M == 0) return hipSuccess;
  const bool ln = g != nullptr;
  if (t_bf16)
    readout_go<bf16>(gran_for(E), ln, M, E, p1, ld1, p2, ld2, idx2, rows2, p3, ld3, bt, g, be, eps, (bf16 *)t_out,
                     tap, st);
  else
    readout_go<float>(gran_for(E), ln, M, E, p1, ld1, p2, ld2, idx2, rows2, p3, ld3, bt, g, be, eps, (float *)t_out,
                      tap, st);
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

__global__ __launch_bounds__(256) void fill_zero_kernel(float *__restrict__ p, long long n) {
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long long)gridDim.x * 256) p[i] = 0.f;
}

hipError_t launch_fill_zero(float *p, long long n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  long long blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

hipError_t launch_valid_rows(int n, const float *mask, int32_t *idx, int *count, hipStream_t st) {
  hipLaunchKernelGGL(valid_rows_kernel, dim3(1), dim3(1024), 0, st, n, mask, idx, count);
  return hipGetLastError();
}

hipError_t launch_lse(int M, int ntiles, const float2 *part, float *lse, float *logits, int V,
                      hipStream_t st) {
  if (M == 0) return hipSuccess;
  hipLaunchKernelGGL(lse_kernel, dim3(M), dim3(kT), 0, st, M, ntiles, part, lse, logits, V);
  return hipGetLastError();
}

}  // namespace mt
