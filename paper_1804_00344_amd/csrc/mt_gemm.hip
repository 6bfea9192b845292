// Matrix products of the decoder step on CDNA4 matrix cores.
//
// out[m, n] = sum_k A[m, k] * W[k, n] (+ bias[n]), with W pre-packed by mt_load_weights
// as Wt[n][k] (K contiguous, zero padded to N_pad x K_pad) in the compute dtype.
//  * fp32 operands: v_mfma_f32_16x16x4_f32.  A 16-byte LDS vector holds 4 consecutive k
//    of one row; lane group g = lane/16 owns k = 4g..4g+3 of each 16-k chunk and feeds
//    them to 4 successive MFMAs (A and B use the same k assignment, so the sum is the
//    plain dot product).
//  * bf16 operands: v_mfma_f32_16x16x32_bf16, one 16-byte vector (8 k) per lane per MFMA.
// Both paths read LDS identically: per 64-byte k-chunk, lane l reads 16 bytes at row
// (l % 16), byte offset 16 * (l / 16).
//
// Tiles: BM x BN per 256-thread workgroup, 2 x 2 waves, each wave (BM/2) x (BN/2) as
// 16 x 16 MFMA blocks.  K advances 128 bytes per tile through a double-buffered LDS
// ring; the next tile's global loads are issued before the current tile's MFMAs.
// The A operand may be gathered by a row index (token -> embedding row, backpointer ->
// state row) and converted fp32 -> bf16 while staged.
//
// Epilogues: plain store (fp32 or bf16) and tanh store, with an optional bias.
#include "mt_internal.h"

namespace mt {

constexpr int kRowBytes = 128;              // K bytes per LDS tile row
constexpr int kLdsStride = kRowBytes + 16;  // padded row stride: conflict-free 16B reads
constexpr int kThreads = 256;

template <typename CT, int BM, int BN>
struct Cfg {
  static constexpr int EPV = 16 / (int)sizeof(CT);  // elements per 16-byte vector
  static constexpr int BK = kRowBytes / (int)sizeof(CT);
  static constexpr int WM = BM / 2, WN = BN / 2;
  static constexpr int FM = WM / 16, FN = WN / 16;
  static constexpr int A_PER_T = BM * 8 / kThreads;  // 16B vectors per thread per tile
  static constexpr int B_PER_T = BN * 8 / kThreads;
  static constexpr int STAGE = (BM + BN) * kLdsStride;
  static constexpr int LDS = 2 * STAGE;
};

struct Problems {
  GemmProblem p[2];
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename T>
__device__ __forceinline__ T bitcast16(const u32x4 &v) {
  T r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

__device__ __forceinline__ u32x4 pack_bf16x8(const float4 &a, const float4 &b) {
  bf16x8 h;
  h[0] = to_bf16(a.x); h[1] = to_bf16(a.y); h[2] = to_bf16(a.z); h[3] = to_bf16(a.w);
  h[4] = to_bf16(b.x); h[5] = to_bf16(b.y); h[6] = to_bf16(b.z); h[7] = to_bf16(b.w);
  u32x4 r;
  __builtin_memcpy(&r, &h, 16);
  return r;
}

template <typename CT, int EPI, int BM, int BN>
__global__ __launch_bounds__(kThreads) void gemm_kernel(Problems probs) {
  using C = Cfg<CT, BM, BN>;
  __shared__ __attribute__((aligned(16))) char lds[C::LDS];

  const GemmProblem &P = probs.p[blockIdx.z];
  const int tilesM = (P.M + BM - 1) / BM;
  const int tilesN = (P.N + BN - 1) / BN;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  if (tile >= tilesM * tilesN) return;
  const int tm = tile % tilesM, tn = tile / tilesM;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;

  // ---- per-thread global source rows (fixed across k tiles) ----
  const char *a_src[C::A_PER_T];
  bool a_ok[C::A_PER_T];
  int a_kv[C::A_PER_T];
  const int a_bf16 = P.a_bf16;
  const int a_es = (sizeof(CT) == 2 && !a_bf16) ? 4 : (int)sizeof(CT);  // source element bytes
#pragma unroll
  for (int p = 0; p < C::A_PER_T; ++p) {
    const int v = tid + kThreads * p;
    const int r = v >> 3;
    a_kv[p] = v & 7;
    const int m = m0 + r;
    a_ok[p] = m < P.M;
    int src = m;
    if (P.a_idx && a_ok[p]) {
      src = P.a_idx[m];
      if (src < 0 || src >= P.a_rows) {
        if (P.err) atomicOr(P.err, 1 << P.err_bit);
        src = src < 0 ? 0 : P.a_rows - 1;
      }
    }
    a_src[p] = (const char *)P.A + (size_t)(a_ok[p] ? src : 0) * P.lda * a_es;
  }
  const char *b_src[C::B_PER_T];
#pragma unroll
  for (int p = 0; p < C::B_PER_T; ++p) {
    const int v = tid + kThreads * p;
    b_src[p] = (const char *)P.Bp + ((size_t)(n0 + (v >> 3)) * P.ldb + (v & 7) * C::EPV) * sizeof(CT);
  }

  u32x4 ra[C::A_PER_T], rb[C::B_PER_T];
  auto load_tile = [&](int kt) {
    const int kbase = kt * C::BK;
#pragma unroll
    for (int p = 0; p < C::A_PER_T; ++p) {
      const int k = kbase + a_kv[p] * C::EPV;
      if (!a_ok[p] || k >= P.K) {
        ra[p] = u32x4{0u, 0u, 0u, 0u};
      } else if (sizeof(CT) == 2 && !a_bf16) {
        const float4 *s = (const float4 *)(a_src[p] + (size_t)k * 4);
        ra[p] = pack_bf16x8(s[0], s[1]);
      } else {
        ra[p] = *(const u32x4 *)(a_src[p] + (size_t)k * sizeof(CT));
      }
    }
#pragma unroll
    for (int p = 0; p < C::B_PER_T; ++p) rb[p] = *(const u32x4 *)(b_src[p] + (size_t)kbase * sizeof(CT));
  };
  auto store_tile = [&](int buf) {
    char *As = lds + buf * C::STAGE;
    char *Bs = As + BM * kLdsStride;
#pragma unroll
    for (int p = 0; p < C::A_PER_T; ++p) {
      const int v = tid + kThreads * p;
      *(u32x4 *)(As + (v >> 3) * kLdsStride + (v & 7) * 16) = ra[p];
    }
#pragma unroll
    for (int p = 0; p < C::B_PER_T; ++p) {
      const int v = tid + kThreads * p;
      *(u32x4 *)(Bs + (v >> 3) * kLdsStride + (v & 7) * 16) = rb[p];
    }
  };

  f32x4 acc[C::FM][C::FN];
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (P.K + C::BK - 1) / C::BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) load_tile(kt + 1);
    const char *As = lds + (kt & 1) * C::STAGE;
    const char *Bs = As + BM * kLdsStride;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      u32x4 af[C::FM], bfv[C::FN];
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
        af[i] = *(const u32x4 *)(As + (wm * C::WM + i * 16 + (lane & 15)) * kLdsStride + c * 64 + (lane >> 4) * 16);
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
        bfv[j] = *(const u32x4 *)(Bs + (wn * C::WN + j * 16 + (lane & 15)) * kLdsStride + c * 64 + (lane >> 4) * 16);
      if constexpr (sizeof(CT) == 2) {
#pragma unroll
        for (int i = 0; i < C::FM; ++i)
#pragma unroll
          for (int j = 0; j < C::FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bitcast16<bf16x8>(af[i]),
                                                                 bitcast16<bf16x8>(bfv[j]), acc[i][j], 0, 0, 0);
      } else {
        // element s of each vector feeds MFMA s (copied out through memcpy: a bit cast of
        // a vector element reference is miscompiled into element 0 by this toolchain)
        float fa[C::FM][4], fb[C::FN][4];
#pragma unroll
        for (int i = 0; i < C::FM; ++i) __builtin_memcpy(fa[i], &af[i], 16);
#pragma unroll
        for (int j = 0; j < C::FN; ++j) __builtin_memcpy(fb[j], &bfv[j], 16);
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int i = 0; i < C::FM; ++i)
#pragma unroll
            for (int j = 0; j < C::FN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i][s], fb[j][s], acc[i][j], 0, 0, 0);
      }
    }
    if (kt + 1 < nk) store_tile((kt + 1) & 1);
    __syncthreads();
  }

  {
    // lane holds D[row = 4*(lane/16) + r][col = lane % 16] of each 16x16 block
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int j = 0; j < C::FN; ++j) {
        const int col = n0 + wn * C::WN + j * 16 + (lane & 15);
        if (col >= P.N) continue;
        const float bias = P.bias ? P.bias[col] : 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m0 + wm * C::WM + i * 16 + (lane >> 4) * 4 + r;
          if (row >= P.M) continue;
          float v = acc[i][j][r] + bias;
          if (EPI == EPI_TANH) v = tanh_fast(v);
          if (P.out_bf16)
            ((bf16 *)P.out)[(size_t)row * P.ldc + col] = to_bf16(v);
          else
            ((float *)P.out)[(size_t)row * P.ldc + col] = v;
        }
      }
  }
}



template <typename CT, int EPI, int BM, int BN>
static hipError_t go(const Problems &ps, int nprob, hipStream_t st) {
  int maxt = 0;
  for (int i = 0; i < nprob; ++i) {
    const int t = ((ps.p[i].M + BM - 1) / BM) * ((ps.p[i].N + BN - 1) / BN);
    maxt = t > maxt ? t : maxt;
  }
  if (maxt == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<CT, EPI, BM, BN>), dim3(maxt, 1, nprob), dim3(kThreads), 0, st, ps);
  return hipGetLastError();
}

template <typename CT>
static hipError_t dispatch(const Problems &ps, int nprob, Epilogue epi, hipStream_t st) {
  // big tiles when they already fill the chip, else 64 x 64
  long t128 = 0;
  for (int i = 0; i < nprob; ++i)
    t128 += (long)((ps.p[i].M + 127) / 128) * ((ps.p[i].N + 127) / 128);
  const bool big = t128 >= 512;
  if (epi == EPI_TANH)
    return big ? go<CT, EPI_TANH, 128, 128>(ps, nprob, st) : go<CT, EPI_TANH, 64, 64>(ps, nprob, st);
  return big ? go<CT, EPI_STORE, 128, 128>(ps, nprob, st) : go<CT, EPI_STORE, 64, 64>(ps, nprob, st);
}

hipError_t launch_gemm(int bf16_mma, const GemmProblem *probs, int nprob, Epilogue epi, hipStream_t st) {
  Problems ps{};
  for (int i = 0; i < nprob; ++i) ps.p[i] = probs[i];
  return bf16_mma ? dispatch<bf16>(ps, nprob, epi, st) : dispatch<float>(ps, nprob, epi, st);
}

}  // namespace mt
