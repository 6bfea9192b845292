// Ensemble combination (Section 2.3: ensembling of models inside batched beam search): the
// members' log-probabilities over the same hypothesis rows are summed with their weights
// before one beam selection,
//   out[i] = sum_j w_j * logp_j[i],  i < M * V, members in order j = 0, 1, ...
// A pure stream: each element is read once from every member and written once, so the kernel
// is bound by HBM bandwidth ((n + 1) * 4 bytes per element).  (The fused ensemble path instead
// adds each member's weighted logits in its vocabulary kernel and subtracts the per-row
// constant sum_i w_i LSE_i at selection: ensemble_const_kernel below.)  Every thread takes 16-byte
// granules in a grid-stride loop and issues the loads of all members before the sums.
#include "mt_internal.h"

namespace mt {

struct EnsembleArgs {
  const float *in[kMaxEnsemble];
  float w[kMaxEnsemble];
  int n;
  long long count;  // elements
  float *out;
};

constexpr int kEnT = 256;

template <int N>
__global__ __launch_bounds__(kEnT) void ensemble_kernel(EnsembleArgs a) {
  const long long n4 = a.count / 4;
  const long long stride = (long long)gridDim.x * kEnT;
  for (long long i = (long long)blockIdx.x * kEnT + threadIdx.x; i < n4; i += stride) {
    float4 x[N];
#pragma unroll
    for (int j = 0; j < N; ++j) x[j] = ((const float4 *)a.in[j])[i];
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < N; ++j) {
      s.x = __builtin_fmaf(a.w[j], x[j].x, s.x);
      s.y = __builtin_fmaf(a.w[j], x[j].y, s.y);
      s.z = __builtin_fmaf(a.w[j], x[j].z, s.z);
      s.w = __builtin_fmaf(a.w[j], x[j].w, s.w);
    }
    ((float4 *)a.out)[i] = s;
  }
  // the last count % 4 elements
  if (blockIdx.x == 0 && threadIdx.x < (int)(a.count - n4 * 4)) {
    const long long i = n4 * 4 + threadIdx.x;
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < N; ++j) s = __builtin_fmaf(a.w[j], a.in[j][i], s);
    a.out[i] = s;
  }
}

hipError_t launch_ensemble(int n, const float *const *in, const float *w, long long count, float *out,
                           int num_cu, hipStream_t st) {
  if (n < 1 || n > kMaxEnsemble) return hipErrorInvalidValue;
  if (count == 0) return hipSuccess;
  EnsembleArgs a{};
  for (int j = 0; j < n; ++j) {
    a.in[j] = in[j];
    a.w[j] = w[j];
  }
  a.n = n;
  a.count = count;
  a.out = out;
  // enough resident waves to keep the HBM queues full, no more blocks than work
  long long blocks = (long long)num_cu * 8;
  const long long need = (count / 4 + kEnT - 1) / kEnT;
  if (blocks > need) blocks = need > 0 ? need : 1;
#define MT_EN(N) hipLaunchKernelGGL((ensemble_kernel<N>), dim3((unsigned)blocks), dim3(kEnT), 0, st, a)
  switch (n) {
    case 1: MT_EN(1); break;
    case 2: MT_EN(2); break;
    case 3: MT_EN(3); break;
    case 4: MT_EN(4); break;
    case 5: MT_EN(5); break;
    case 6: MT_EN(6); break;
    case 7: MT_EN(7); break;
    default: MT_EN(8); break;
  }
#undef MT_EN
  return hipGetLastError();
}

// Row constant of a fused ensemble (see EnsembleConst): one wave per row (four rows per
// workgroup); each member's log-sum-exp is merged by the same routine, in the same order, as the
// beam selection merges a row's partials (wave_row_lse).
__global__ __launch_bounds__(256) void ensemble_const_kernel(EnsembleConst a, int M) {
  const int m = blockIdx.x * 4 + (int)(threadIdx.x >> 6);
  if (m >= M) return;  // wave-uniform
  float c = 0.f;
  for (int i = 0; i < a.n; ++i) {
    const float L = wave_row_lse(a.part[i] + (size_t)m * a.ntiles[i], a.ntiles[i]);
    c = __builtin_fmaf(a.w[i], L, c);
  }
  if ((threadIdx.x & 63) == 0) {
    a.prev_adj[m] = a.prev[m] - c;
    if (a.row_const) a.row_const[m] = c;
  }
}

hipError_t launch_ensemble_const(const EnsembleConst &a, int M, hipStream_t st) {
  if (M == 0) return hipSuccess;
  hipLaunchKernelGGL(ensemble_const_kernel, dim3((M + 3) / 4), dim3(256), 0, st, a, M);
  return hipGetLastError();
}

}  // namespace mt
