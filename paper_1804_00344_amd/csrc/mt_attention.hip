// Additive attention with a masked softmax over the source positions of one sentence,
// one 256-thread workgroup per hypothesis row (m = b*K + k):
//   e_i   = sum_a va[a] * tanh(P[b,i,a] + q[m,a])      (valid i only)
//   alpha = exp(e_i - max_valid e) / sum_valid exp(...)  (exactly 0 at masked i)
//   c[m]  = sum_valid alpha_i * Cx[b,i,:]
//
// The valid positions are first compacted into an LDS list (ballot prefix sums), so no loop
// branches on the mask or reads a masked row.
//
// Scores.  tanh x = 1 - 2 / (2^(x * 2/ln2) + 1), so
//   e_i = sum_a va[a] - sum_a 2 va[a] / (2^(P[i,a] c + q[m,a] c) + 1),   c = 2/ln2.
// The row's q is held pre-scaled by c and va pre-scaled by -2, which leaves one FMA, one
// exp2, one add, one reciprocal and one FMA per element; sum_a va[a] is a per-row constant.
// Each wave walks every fourth valid position: its 64 lanes cover the A features of P[b,i]
// in 16-byte granules, and the rows pass through a two-deep ring of raw granules, so the
// loads of the next row are in flight while the current one is scored (lanes beyond A read a
// clamped in-range address and carry zero weight, so the loop has no per-granule branch).
// Cross-lane shuffles reduce the sums.
//
// Context.  Each thread owns 16-byte column granules of Cx and walks the valid positions in
// groups (eight positions for up to two granules per thread), with the next group's row
// loads in flight while the current group is accumulated; the first two groups are loaded
// before the softmax.
//
// Scheduling: a small kernel orders the sentences by length, and the longest rows start
// first on every XCD, with the K rows of one sentence on one XCD sharing its L2 copy of P[b]
// and Cx[b] (row_of_block).
#include "mt_internal.h"

namespace mt {

constexpr int kAT = 256;
constexpr int kMaxS = 1024;
constexpr float kTwoOverLn2 = 2.8853900817779268f;  // 2 / ln 2

template <typename T>
struct Gran;  // one 16-byte granule of a row, widened to fp32
template <>
struct Gran<float> {
  static constexpr int N = 4;
  template <typename V>
  __device__ __forceinline__ static void unpack(const V &v, float (&x)[4]) {
    __builtin_memcpy(x, &v, 16);
  }
  __device__ __forceinline__ static void load(const float *p, float (&x)[4]) {
    const float4 v = *(const float4 *)p;
    x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
  }
};
template <>
struct Gran<bf16> {
  static constexpr int N = 8;
  template <typename V>
  __device__ __forceinline__ static void unpack(const V &v, float (&x)[8]) {
    bf16x8 h;
    __builtin_memcpy(&h, &v, 16);
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (float)h[j];
  }
  __device__ __forceinline__ static void load(const bf16 *p, float (&x)[8]) {
    const bf16x8 v = *(const bf16x8 *)p;
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = (float)v[j];
  }
};

// Row of workgroup w.  With a sentence order (srank[s] = the sentence of rank s, longest
// first), sentence rank s runs on XCD s % 8 (workgroups are dispatched round-robin over the 8
// XCDs: w -> XCD w % 8), and within an XCD the sentences follow their rank, each one's K rows
// in a row: the longest rows start first on every XCD, and the K rows of a sentence share its
// XCD's L2 copy of the keys and the context.  The sentences past the last multiple of 8 (the
// shortest) take the last workgroups in order.  Without an order: consecutive rows on one XCD.
__device__ __forceinline__ int row_of_block(int w, int B, int K, const int *srank) {
  if (!srank) return xcd_remap(w, B * K);
  const int nfull = B & ~(kXcds - 1);
  int s, k;
  if (w < nfull * K) {
    const int j = w / kXcds;
    s = (j / K) * kXcds + w % kXcds;
    k = j % K;
  } else {
    const int r = w - nfull * K;
    s = nfull + r / K;
    k = r % K;
  }
  return srank[s] * K + k;
}

// Sentences by decreasing number of valid positions (the order of equal lengths is
// unspecified: it only schedules work), one 1024-thread workgroup: a histogram of the
// lengths, its exclusive prefix sums from the longest length down, then each sentence takes
// the next slot of its length.
constexpr int kOrderMaxB = 8192;
__global__ __launch_bounds__(1024) void attention_order_kernel(int B, int S, const float *__restrict__ mask,
                                                               int *__restrict__ srank) {
  __shared__ int hist[kMaxS + 1];
  __shared__ int lens[kOrderMaxB];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  for (int l = t; l <= S; l += 1024) hist[l] = 0;
  __syncthreads();
  for (int b = w; b < B; b += 16) {  // one wave per sentence: coalesced mask rows, ballot counts
    const float *mr = mask + (size_t)b * S;
    int n = 0;
    for (int i0 = 0; i0 < S; i0 += 64) n += __popcll(__ballot(i0 + lane < S && mr[i0 + lane] != 0.f));
    if (lane == 0) {
      lens[b] = n;
      atomicAdd(&hist[n], 1);
    }
  }
  __syncthreads();
  if (w == 0) {  // start[L] = sentences longer than L, for L = S .. 0 (reversed index r = S - L)
    const int nb = S + 1, per = (nb + 63) / 64;
    int sum = 0;
    for (int i = 0; i < per; ++i) {
      const int r = lane * per + i;
      if (r < nb) sum += hist[S - r];
    }
    int incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o, 64);
      if (lane >= o) incl += y;
    }
    int run = incl - sum;
    for (int i = 0; i < per; ++i) {
      const int r = lane * per + i;
      if (r < nb) {
        const int h = hist[S - r];
        hist[S - r] = run;
        run += h;
      }
    }
  }
  __syncthreads();
  for (int b = t; b < B; b += 1024) srank[atomicAdd(&hist[lens[b]], 1)] = b;
}

// NG: granules per lane of a score row (A <= 64 * NG * Gran<T>::N);
// NC: granules per thread of a context row (2H <= 256 * NC * Gran<T>::N);
// RD: key rows in flight per wave in the score loop (two cover the latency: deeper rings, 4 to
// 8 rows at one beam row per sentence, measured no faster)
template <typename T, int NG, int NC, int RD>
__global__ __launch_bounds__(kAT) void attention_kernel(int B, int K, int S, int A, int Cd,
                                                        const T *__restrict__ P,
                                                        const T *__restrict__ Cx,
                                                        const float *__restrict__ mask,
                                                        const float *__restrict__ q, int ldq,
                                                        const float *__restrict__ va,
                                                        float *__restrict__ ctx_out, int ldc,
                                                        bf16 *__restrict__ ctx16, int ld16,
                                                        float *__restrict__ alpha_out,
                                                        const int *__restrict__ srank) {
  constexpr int G = Gran<T>::N;
  constexpr int U = NC <= 2 ? 8 : NC == 4 ? 4 : 2;  // context positions in flight per thread
  __shared__ float es[kMaxS];
  __shared__ int vidx[kMaxS];
  __shared__ float stat[2];
  __shared__ int nvalid;
  const int m = row_of_block(blockIdx.x, B, K, srank);
  const int b = m / K;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int ng = A / G;  // granules per P row

  // ---- this lane's slice of q (scaled by 2/ln2) and va (scaled by -2): requested before the
  // mask is read and used after it, so the two round trips overlap ----
  float qr[NG][G], vr[NG][G];
  int goff[NG];  // element offset of the lane's granule j in a P row (clamped)
  float4 qraw[NG][G / 4], vraw[NG][G / 4];
#pragma unroll
  for (int j = 0; j < NG; ++j) {
    const int g = j * 64 + lane;
    goff[j] = (g < ng ? g : ng - 1) * G;
#pragma unroll
    for (int e = 0; e < G; e += 4) {
      qraw[j][e / 4] = *(const float4 *)(q + (size_t)m * ldq + goff[j] + e);
      vraw[j][e / 4] = *(const float4 *)(va + goff[j] + e);
    }
  }
  // ---- the wave's first key rows, requested before the valid positions are known on the
  // guess that they form a prefix (as padding does): rows wave + 4 d, clamped to the padded
  // length; a row that is not the compacted position it stands for is loaded again below ----
  typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));
  v4u32 ring[RD][NG];
#pragma unroll
  for (int d = 0; d < RD; ++d) {
    const int i = wave + 4 * d < S ? wave + 4 * d : S - 1;
    const char *row = (const char *)(P + ((size_t)b * S + i) * A);
#pragma unroll
    for (int jj = 0; jj < NG; ++jj) ring[d][jj] = *(const v4u32 *)(row + (size_t)goff[jj] * sizeof(T));
  }

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

  float vsum = 0.f;
#pragma unroll
  for (int j = 0; j < NG; ++j) {
    const bool ok = j * 64 + lane < ng;
    float qv[G], vv[G];
#pragma unroll
    for (int e = 0; e < G; e += 4) {
      __builtin_memcpy(qv + e, &qraw[j][e / 4], 16);
      __builtin_memcpy(vv + e, &vraw[j][e / 4], 16);
    }
#pragma unroll
    for (int e = 0; e < G; ++e) {
      qr[j][e] = ok ? qv[e] * kTwoOverLn2 : 0.f;
      vr[j][e] = ok ? -2.0f * vv[e] : 0.f;
      vsum += ok ? vv[e] : 0.f;
    }
  }
  vsum = wave_sum(vsum);
  __syncthreads();
  const int n = nvalid;

  // ---- scores: wave w takes positions w, w + 4, w + 8, ... through a two-deep ring of
  // raw P rows, so the next row's loads are in flight while the current one is scored ----
  auto load_raw = [&](int jp, v4u32(&r)[NG]) {
    const int i = vidx[jp < n ? jp : 0];  // past the end: an in-range row, never scored
    const char *row = (const char *)(P + ((size_t)b * S + i) * A);
#pragma unroll
    for (int jj = 0; jj < NG; ++jj) r[jj] = *(const v4u32 *)(row + (size_t)goff[jj] * sizeof(T));
  };
  auto score_raw = [&](const v4u32(&r)[NG]) {
    float acc = 0.f;
#pragma unroll
    for (int jj = 0; jj < NG; ++jj) {
      float x[G];
      Gran<T>::unpack(r[jj], x);
#pragma unroll
      for (int e = 0; e < G; ++e) {
        const float d = __builtin_amdgcn_exp2f(__builtin_fmaf(x[e], kTwoOverLn2, qr[jj][e])) + 1.0f;
        acc = __builtin_fmaf(vr[jj][e], rcp_fast(d), acc);
      }
    }
    return wave_sum(acc);
  };
  if (wave < n) {  // wave-uniform
#pragma unroll
    for (int d = 0; d < RD; ++d)
      if (wave + 4 * d < n && vidx[wave + 4 * d] != wave + 4 * d) load_raw(wave + 4 * d, ring[d]);
    int j = wave;
    bool go = true;
    while (go) {
#pragma unroll
      for (int d = 0; d < RD; ++d) {
        if (go) {
          const float sc = score_raw(ring[d]);
          if (lane == 0) es[j] = vsum + sc;
          load_raw(j + 4 * RD, ring[d]);
          j += 4;
          go = j < n;
        }
      }
    }
  }
  __syncthreads();

  // ---- the first context rows are loaded now: they do not depend on the weights, so their
  // latency runs under the softmax ----
  const int ncg = Cd / G;
  const T *Cb = Cx + (size_t)b * S * Cd;
  float c[NC][G];
  int coff[NC];
#pragma unroll
  for (int p = 0; p < NC; ++p) {
    const int g = t + kAT * p;
    coff[p] = (g < ncg ? g : ncg - 1) * G;
#pragma unroll
    for (int e = 0; e < G; ++e) c[p][e] = 0.f;
  }
  // raw 16-byte granules of U context rows (a group); two groups in flight
  typedef uint32_t v4c __attribute__((ext_vector_type(4)));
  auto load_group = [&](int j0, v4c(&r)[U][NC]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u;
      const char *row = (const char *)(Cb + (size_t)vidx[j < n ? j : 0] * Cd);  // past the end: weight 0
#pragma unroll
      for (int p = 0; p < NC; ++p) r[u][p] = *(const v4c *)(row + (size_t)coff[p] * sizeof(T));
    }
  };
  v4c ga[U][NC], gb[U][NC];
  if (n > 0) {
    load_group(0, ga);
    load_group(U, gb);
  }

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

  // ---- context: the groups of U positions pass through the two-deep ring ----
  auto accumulate = [&](int j0, const v4c(&r)[U][NC]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u;
      const float al = j < n ? es[j] : 0.f;
#pragma unroll
      for (int p = 0; p < NC; ++p) {
        float x[G];
        Gran<T>::unpack(r[u][p], x);
#pragma unroll
        for (int e = 0; e < G; ++e) c[p][e] = __builtin_fmaf(al, x[e], c[p][e]);
      }
    }
  };
  for (int j0 = 0; j0 < n;) {
    accumulate(j0, ga);
    load_group(j0 + 2 * U, ga);
    j0 += U;
    if (j0 >= n) break;
    accumulate(j0, gb);
    load_group(j0 + 2 * U, gb);
    j0 += U;
  }
#pragma unroll
  for (int p = 0; p < NC; ++p) {
    const int g = t + kAT * p;
    if (g >= ncg) continue;
    if (ctx_out) {
      float *o = ctx_out + (size_t)m * ldc + g * G;
#pragma unroll
      for (int e = 0; e < G; e += 4) *(float4 *)(o + e) = make_float4(c[p][e], c[p][e + 1], c[p][e + 2], c[p][e + 3]);
    }
    if (ctx16) {  // bf16 context rows [M][Cd] for a following bf16 product
      bf16 h[G];
#pragma unroll
      for (int e = 0; e < G; ++e) h[e] = to_bf16(c[p][e]);
      __builtin_memcpy(ctx16 + (size_t)m * ld16 + g * G, h, sizeof(h));
    }
  }
}

#ifndef MT_ATTN_RING_K1
#define MT_ATTN_RING_K1 2
#endif
constexpr int kAttnRingK1 = MT_ATTN_RING_K1;

static int bucket(int n) { return n <= 1 ? 1 : n <= 2 ? 2 : n <= 4 ? 4 : n <= 8 ? 8 : 16; }

template <typename T, int NG>
static void attn_go_c(int nc, int B, int K, int S, int A, int Cd, const T *P, const T *Cx, const float *mask,
                      const float *q, int ldq, const float *va, float *ctx_out, int ldc, bf16 *ctx16,
                      int ld16, float *alpha_out, const int *srank, hipStream_t st) {
  const int M = B * K;
#define MT_AT1(NC, RD)                                                                                   \
  hipLaunchKernelGGL((attention_kernel<T, NG, NC, RD>), dim3(M), dim3(kAT), 0, st, B, K, S, A, Cd, P, Cx, \
                     mask, q, ldq, va, ctx_out, ldc, ctx16, ld16, alpha_out, srank)
#define MT_AT(NC)                       \
  do {                                  \
    if (K == 1)                         \
      MT_AT1(NC, kAttnRingK1);          \
    else                                \
      MT_AT1(NC, 2);                    \
  } while (0)
  if (nc <= 1) MT_AT(1);
  else if (nc <= 2) MT_AT(2);
  else if (nc <= 4) MT_AT(4);
  else MT_AT(8);
#undef MT_AT
#undef MT_AT1
}

template <typename T>
static void attn_go(int B, int K, int S, int A, int Cd, const T *P, const T *Cx, const float *mask,
                    const float *q, int ldq, const float *va, float *ctx_out, int ldc, bf16 *ctx16,
                    int ld16, float *alpha_out, const int *srank, hipStream_t st) {
  constexpr int G = Gran<T>::N;
  const int ng = bucket((A / G + 63) / 64);
  const int nc = bucket((Cd / G + kAT - 1) / kAT);
#define MT_AG(NG) attn_go_c<T, NG>(nc, B, K, S, A, Cd, P, Cx, mask, q, ldq, va, ctx_out, ldc, ctx16, ld16, alpha_out, srank, st)
  switch (ng) {
    case 1: MT_AG(1); break;
    case 2: MT_AG(2); break;
    case 4: MT_AG(4); break;
    case 8: MT_AG(8); break;
    default: MT_AG(16); break;
  }
#undef MT_AG
}

hipError_t launch_attention_order(int B, int S, const float *mask, int *srank, hipStream_t st) {
  if (B < 1 || B > kOrderMaxB || S < 1 || S > kMaxS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(attention_order_kernel, dim3(1), dim3(1024), 0, st, B, S, mask, srank);
  return hipGetLastError();
}

int attention_order_max_sentences() { return kOrderMaxB; }

hipError_t launch_attention(int B, int K, int S, int A, int Cd, const void *P, const void *Cx,
                            int bf16_io, const float *mask, const float *q, int ldq,
                            const float *va, float *ctx_out, int ldc, bf16 *ctx16, int ld16, float *alpha_out,
                            const int *srank, hipStream_t st) {
  if (B * K == 0) return hipSuccess;
  if (bf16_io)
    attn_go<bf16>(B, K, S, A, Cd, (const bf16 *)P, (const bf16 *)Cx, mask, q, ldq, va, ctx_out, ldc, ctx16,
                  ld16, alpha_out, srank, st);
  else
    attn_go<float>(B, K, S, A, Cd, (const float *)P, (const float *)Cx, mask, q, ldq, va, ctx_out, ldc, ctx16,
                   ld16, alpha_out, srank, st);
  return hipGetLastError();
}

}  // namespace mt
