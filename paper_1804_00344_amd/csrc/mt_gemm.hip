// Matrix products of the decoder step on CDNA4 matrix cores.
//
// out[m, n] = sum_k A[m, k] * W[k, n] (+ bias[n]), with W pre-packed by mt_load_weights
// as Wt[n][k] (K contiguous, zero padded to N_pad x K_pad) in the compute dtype.
//  * fp32 operands: v_mfma_f32_16x16x4_f32.  A 16-byte LDS vector holds 4 consecutive k
//    of one row; lane group g = lane/16 owns k = 4g..4g+3 of each 16-k chunk and feeds
//    them to 4 successive MFMAs (A and B use the same k assignment, so the sum is the
//    plain dot product).
//  * bf16 operands, wave tiles of 32 x 32 or more: v_mfma_f32_32x32x16_bf16, whose rate
//    is twice that of the 16 x 16 x 32 form on this chip.  Per 32-byte k-step lane l reads
//    16 bytes (8 k) at row (l % 32), byte offset 16 * (l / 32).
//  * fp32 operands, wave tiles of 32 x 64 or more: v_mfma_f32_32x32x2f32 with the same reads,
//    each 16-byte vector feeding 4 successive MFMAs (lane half g supplies k = 4g + e to
//    MFMA e).
//  * bf16 operands, 16 x 16 wave tiles: v_mfma_f32_16x16x32_bf16, one 16-byte vector (8 k)
//    per lane per MFMA.
// The 16 x 16 forms read LDS identically: per 64-byte k-chunk, lane l reads 16 bytes at row
// (l % 16), byte offset 16 * (l / 16).
//
// Tiles: BM x BN (32 x 32 up to 128 x 128) per 256-thread workgroup, 2 x 2 waves, each wave
// (BM/2) x (BN/2) as 16 x 16 or 32 x 32 MFMA blocks.  K advances 128 bytes (of the compute dtype) per
// tile through a double-buffered LDS ring fed from two register stages: the global loads of
// tile k+2 are issued while tile k is multiplied, and tile k+1 is written to LDS behind it,
// so every load has two tiles of MFMA work to arrive.  Loads are unconditional straight-line
// code and nothing is masked: a row past M reads row 0 and its output row is never stored,
// and a vector past K reads the row's last in-range vector, which meets the zero padding of
// the packed weights (finite x 0 adds nothing).  The fp32 -> bf16 rounding of an fp32 A
// operand happens when a stage is written to LDS; scheduling fences keep the load, multiply
// and store phases in that order, so no wait on the loads is forced early.
// The A operand may be gathered by a row index (token -> embedding row, backpointer ->
// state row).  Every problem of one launch has the same A element type AT.
//
// Epilogues: plain store (fp32 or bf16) and tanh store, with an optional bias.
#include "mt_internal.h"

namespace mt {

constexpr int kRowBytes = 128;              // K bytes per LDS tile row
constexpr int kLdsStride = kRowBytes + 16;  // padded row stride: conflict-free 16B reads
constexpr int kThreads = 256;

template <typename CT, typename AT, int BM, int BN>
struct Cfg {
  static constexpr int EPV = 16 / (int)sizeof(CT);  // compute elements per 16-byte vector
  static constexpr int AV = (int)sizeof(AT) / (int)sizeof(CT);  // 16-byte source loads per vector
  static constexpr int BK = kRowBytes / (int)sizeof(CT);
  static constexpr int WM = BM / 2, WN = BN / 2;
  static constexpr int FM = WM / 16, FN = WN / 16;
  // wave tiles of whole 32 x 32 blocks: the 32 x 32 MFMA (bf16 32x32x16; fp32 32x32x2 when
  // the wave has at least two blocks, so that successive MFMAs alternate accumulators)
  static constexpr bool M32 = WM % 32 == 0 && (sizeof(CT) == 2 ? WN % 32 == 0 : WN % 64 == 0);
  static constexpr int FM32 = WM / 32, FN32 = WN / 32;
  static constexpr int A_PER_T = BM * 8 / kThreads;  // 16B vectors per thread per tile
  static constexpr int B_PER_T = BN * 8 / kThreads;
  static constexpr int STAGE = (BM + BN) * kLdsStride;
  static constexpr int LDS = 2 * STAGE;
};

struct Problems {
  GemmProblem p[2];
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

template <typename T>
__device__ __forceinline__ T bitcast16(const u32x4 &v) {
  T r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

__device__ __forceinline__ u32x4 pack_bf16x8(const u32x4 &lo, const u32x4 &hi) {
  float a[4], b[4];
  __builtin_memcpy(a, &lo, 16);
  __builtin_memcpy(b, &hi, 16);
  bf16x8 h;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    h[j] = to_bf16(a[j]);
    h[4 + j] = to_bf16(b[j]);
  }
  u32x4 r;
  __builtin_memcpy(&r, &h, 16);
  return r;
}

// one tile's global data in flight: raw A source vectors and B vectors
template <int A_PER_T, int AV, int B_PER_T>
struct Stage {
  u32x4 a[A_PER_T][AV];
  u32x4 b[B_PER_T];
};

template <typename CT, typename AT, int EPI, int BM, int BN>
__global__ __launch_bounds__(kThreads) void gemm_kernel(Problems probs) {
  using C = Cfg<CT, AT, BM, BN>;
  using St = Stage<C::A_PER_T, C::AV, C::B_PER_T>;
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
  bool a_row_ok[C::A_PER_T];
  int a_kv[C::A_PER_T];
#pragma unroll
  for (int p = 0; p < C::A_PER_T; ++p) {
    const int v = tid + kThreads * p;
    const int r = v >> 3;
    a_kv[p] = v & 7;
    const int m = m0 + r;
    a_row_ok[p] = m < P.M;
    int src = m;
    if (P.a_idx && a_row_ok[p]) {
      src = P.a_idx[m];
      if (src < 0 || src >= P.a_rows) {
        if (P.err) atomicOr(P.err, 1 << P.err_bit);
        src = src < 0 ? 0 : P.a_rows - 1;
      }
    }
    a_src[p] = (const char *)P.A + (size_t)(a_row_ok[p] ? src : 0) * P.lda * sizeof(AT);
  }
  const char *b_src[C::B_PER_T];
#pragma unroll
  for (int p = 0; p < C::B_PER_T; ++p) {
    const int v = tid + kThreads * p;
    b_src[p] = (const char *)P.Bp + ((size_t)(n0 + (v >> 3)) * P.ldb + (v & 7) * C::EPV) * sizeof(CT);
  }

  auto load_tile = [&](int kt, St &S) {
    const int kbase = kt * C::BK;
#pragma unroll
    for (int p = 0; p < C::A_PER_T; ++p) {
      const int k = kbase + a_kv[p] * C::EPV;
      const int kc = k < P.K ? k : P.K - C::EPV;
      const char *src = a_src[p] + (size_t)kc * sizeof(AT);
#pragma unroll
      for (int v = 0; v < C::AV; ++v) S.a[p][v] = *(const u32x4 *)(src + 16 * v);
    }
#pragma unroll
    for (int p = 0; p < C::B_PER_T; ++p) S.b[p] = *(const u32x4 *)(b_src[p] + (size_t)kbase * sizeof(CT));
  };
  auto store_tile = [&](int buf, const St &S) {
    char *As = lds + buf * C::STAGE;
    char *Bs = As + BM * kLdsStride;
#pragma unroll
    for (int p = 0; p < C::A_PER_T; ++p) {
      const int v = tid + kThreads * p;
      u32x4 val;
      if constexpr (C::AV == 2)
        val = pack_bf16x8(S.a[p][0], S.a[p][1]);
      else
        val = S.a[p][0];
      *(u32x4 *)(As + (v >> 3) * kLdsStride + (v & 7) * 16) = val;
    }
#pragma unroll
    for (int p = 0; p < C::B_PER_T; ++p) {
      const int v = tid + kThreads * p;
      *(u32x4 *)(Bs + (v >> 3) * kLdsStride + (v & 7) * 16) = S.b[p];
    }
  };

  f32x4 acc[C::M32 ? 1 : C::FM][C::M32 ? 1 : C::FN];
  f32x16 acc32[C::M32 ? C::FM32 : 1][C::M32 ? C::FN32 : 1];
  if constexpr (C::M32) {
#pragma unroll
    for (int i = 0; i < C::FM32; ++i)
#pragma unroll
      for (int j = 0; j < C::FN32; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc32[i][j][r] = 0.f;
  } else {
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int j = 0; j < C::FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  auto compute = [&](int buf) {
    const char *As = lds + buf * C::STAGE;
    const char *Bs = As + BM * kLdsStride;
    if constexpr (C::M32) {
#pragma unroll
      for (int s = 0; s < kRowBytes / 32; ++s) {
        u32x4 af[C::FM32], bfv[C::FN32];
#pragma unroll
        for (int i = 0; i < C::FM32; ++i)
          af[i] = *(const u32x4 *)(As + (wm * C::WM + i * 32 + (lane & 31)) * kLdsStride + s * 32 + (lane >> 5) * 16);
#pragma unroll
        for (int j = 0; j < C::FN32; ++j)
          bfv[j] = *(const u32x4 *)(Bs + (wn * C::WN + j * 32 + (lane & 31)) * kLdsStride + s * 32 + (lane >> 5) * 16);
        if constexpr (sizeof(CT) == 2) {
#pragma unroll
          for (int i = 0; i < C::FM32; ++i)
#pragma unroll
            for (int j = 0; j < C::FN32; ++j)
              acc32[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bitcast16<bf16x8>(af[i]),
                                                                    bitcast16<bf16x8>(bfv[j]), acc32[i][j], 0, 0, 0);
        } else {
          // fp32: the 32-byte step is 8 k; element e of a lane's vector feeds MFMA e, lane half
          // g supplying k = 4g + e (the same assignment on both operands)
          float fa[C::FM32][4], fb[C::FN32][4];
#pragma unroll
          for (int i = 0; i < C::FM32; ++i) __builtin_memcpy(fa[i], &af[i], 16);
#pragma unroll
          for (int j = 0; j < C::FN32; ++j) __builtin_memcpy(fb[j], &bfv[j], 16);
#pragma unroll
          for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int i = 0; i < C::FM32; ++i)
#pragma unroll
              for (int j = 0; j < C::FN32; ++j)
                acc32[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[i][e], fb[j][e], acc32[i][j], 0, 0, 0);
        }
      }
      return;
    }
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
  };

  // Iteration kt multiplies LDS stage kt & 1 (tile kt), loads tile kt + 2 into register
  // stage kt & 1 and writes register stage (kt + 1) & 1 (tile kt + 1, loaded one iteration
  // earlier) into the other LDS stage.  Tile indices clamp to the last tile, so the body is
  // branch-free (the last two iterations re-load the last tile, an L2 hit, and the final
  // LDS write is never read): conditional loads would make the compiler drain every
  // outstanding load at the loop header.
  St s0, s1;
  const int nk = (P.K + C::BK - 1) / C::BK;
  const int last = nk - 1;
  auto step = [&](int kt, St &cur, St &nxt, int buf) {
    load_tile(kt + 2 < last ? kt + 2 : last, cur);
    __builtin_amdgcn_sched_barrier(0);
    compute(buf);
    __builtin_amdgcn_sched_barrier(0);
    store_tile(buf ^ 1, nxt);
    __syncthreads();
  };
  load_tile(0, s0);
  load_tile(1 < last ? 1 : last, s1);
  store_tile(0, s0);
  __syncthreads();
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    step(kt, s0, s1, 0);
    step(kt + 1, s1, s0, 1);
  }
  if (kt < nk) step(kt, s0, s1, 0);

  if constexpr (C::M32) {
    // lane holds D[row = 8*(r/4) + 4*(lane/32) + r%4][col = lane % 32] of each 32x32 block
#pragma unroll
    for (int i = 0; i < C::FM32; ++i)
#pragma unroll
      for (int j = 0; j < C::FN32; ++j) {
        const int col = n0 + wn * C::WN + j * 32 + (lane & 31);
        if (col >= P.N) continue;
        const float bias = P.bias ? P.bias[col] : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm * C::WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (row >= P.M) continue;
          float v = acc32[i][j][r] + bias;
          if (EPI == EPI_TANH) v = tanh_fast(v);
          if (P.out_bf16)
            ((bf16 *)P.out)[(size_t)row * P.ldc + col] = to_bf16(v);
          else
            ((float *)P.out)[(size_t)row * P.ldc + col] = v;
        }
      }
  } else {
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

template <typename CT, typename AT, int EPI, int BM, int BN>
static hipError_t go(const Problems &ps, int nprob, hipStream_t st) {
  int maxt = 0;
  for (int i = 0; i < nprob; ++i) {
    const int t = ((ps.p[i].M + BM - 1) / BM) * ((ps.p[i].N + BN - 1) / BN);
    maxt = t > maxt ? t : maxt;
  }
  if (maxt == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<CT, AT, EPI, BM, BN>), dim3(maxt, 1, nprob), dim3(kThreads), 0, st, ps);
  return hipGetLastError();
}

template <typename CT, typename AT, int EPI>
static hipError_t go_tiles(const Problems &ps, int nprob, hipStream_t st) {
  // 128 x 128 tiles when they already fill the chip, 32 x 32 when 64 x 64 tiles would leave
  // CUs idle, else 64 x 64; bf16 takes 64 x 128 (32 x 64 per wave, 32 x 32 x 16 MFMAs) when
  // that fills the chip.  (fp32 stays on 64 x 64: at these shapes the time follows the
  // number of tiles per CU, and 64 x 128 tiles divide worse over 256 CUs.)
  long t128 = 0, t64 = 0, t64x128 = 0;
  for (int i = 0; i < nprob; ++i) {
    t128 += (long)((ps.p[i].M + 127) / 128) * ((ps.p[i].N + 127) / 128);
    t64 += (long)((ps.p[i].M + 63) / 64) * ((ps.p[i].N + 63) / 64);
    t64x128 += (long)((ps.p[i].M + 63) / 64) * ((ps.p[i].N + 127) / 128);
  }
  if (t128 >= 512) return go<CT, AT, EPI, 128, 128>(ps, nprob, st);
  if (sizeof(CT) == 2 && t64x128 >= 256) return go<CT, AT, EPI, 64, 128>(ps, nprob, st);
  if (t64 < 256) return go<CT, AT, EPI, 32, 32>(ps, nprob, st);
  return go<CT, AT, EPI, 64, 64>(ps, nprob, st);
}

template <typename CT, typename AT>
static hipError_t go_epi(const Problems &ps, int nprob, Epilogue epi, hipStream_t st) {
  return epi == EPI_TANH ? go_tiles<CT, AT, EPI_TANH>(ps, nprob, st) : go_tiles<CT, AT, EPI_STORE>(ps, nprob, st);
}

hipError_t launch_gemm(int bf16_mma, const GemmProblem *probs, int nprob, Epilogue epi, hipStream_t st) {
  Problems ps{};
  for (int i = 0; i < nprob; ++i) {
    ps.p[i] = probs[i];
    if (probs[i].a_bf16 != probs[0].a_bf16 || (probs[i].a_bf16 && !bf16_mma)) return hipErrorInvalidValue;
  }
  if (!bf16_mma) return go_epi<float, float>(ps, nprob, epi, st);
  return probs[0].a_bf16 ? go_epi<bf16, bf16>(ps, nprob, epi, st) : go_epi<bf16, float>(ps, nprob, epi, st);
}

}  // namespace mt
