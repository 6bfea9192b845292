// Matrix products of the decoder step on CDNA4 matrix cores:
// out[m, n] = sum_k A[m, k] * W[k, n] (+ bias[n]), tanh optional, fp32 or bf16 output.
// The A operand may be gathered by a row index (token -> embedding row, backpointer -> state
// row); every problem of one launch has the same A element type.
//
// fp32 operands (gemm_kernel): W pre-packed by mt_load_weights as Wt[n][k] (K contiguous, zero
// padded to N_pad x K_pad).  Both operands pass through LDS.
//  * v_mfma_f32_16x16x4_f32: a 16-byte LDS vector holds 4 consecutive k of one row; lane group
//    g = lane/16 owns k = 4g..4g+3 of each 16-k chunk and feeds them to 4 successive MFMAs (A
//    and B use the same k assignment, so the sum is the plain dot product).  Per 64-byte
//    k-chunk lane l reads 16 bytes at row (l % 16), byte offset 16 * (l / 16).
//  * v_mfma_f32_32x32x2f32 for wave tiles of 32 x 64 or more: per 32-byte k-step lane l reads
//    16 bytes at row (l % 32), byte offset 16 * (l / 32), each vector feeding 4 successive
//    MFMAs (lane half g supplies k = 4g + e to MFMA e).
// Tiles: BM x BN (32 x 32 up to 128 x 128) per 256-thread workgroup, 2 x 2 waves.  K advances
// 128 bytes per tile through a double-buffered LDS ring fed from two register stages: the
// global loads of tile k+2 are issued while tile k is multiplied, and tile k+1 is written to
// LDS behind it, so every load has two tiles of MFMA work to arrive.  Loads are unconditional
// straight-line code and nothing is masked: a row past M reads row 0 and its output row is
// never stored, and a vector past K reads the row's last in-range vector, which meets the
// zero padding of the packed weights (finite x 0 adds nothing).
//
// bf16 operands (gemm_wd_kernel, below): weights in MFMA fragment order streamed straight
// into registers, activations through a small LDS ring.
#include "mt_internal.h"

namespace mt {

template <typename T>
__device__ __forceinline__ T pin_s(T x) {  // keep a uniform value in a scalar register
  asm volatile("" : "+s"(x));
  return x;
}

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
  // the 32x32x2 MFMA when the wave has at least two 32 x 32 blocks (successive MFMAs then
  // alternate accumulators)
  static constexpr bool M32 = WM % 32 == 0 && WN % 64 == 0;
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
        {
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
      {
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

  // ---- epilogue ----
  // Problem fields read once into scalar registers (as references into the argument block they
  // would be re-read, each with a full wait, at every store), and the bias values loaded before
  // any store and waited for once: a load between the stores would make every store wait for
  // all earlier stores (the memory counter counts both).
  const int eM = pin_s(P.M), eN = pin_s(P.N), ldc = pin_s(P.ldc), obf = pin_s(P.out_bf16);
  const float *const biasp = pin_s(P.bias);
  char *const outp = (char *)pin_s(P.out);
  constexpr int NJ = C::M32 ? C::FN32 : C::FN;  // column blocks of this wave
  constexpr int JW = C::M32 ? 32 : 16;          // their width
  float bias[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int col = n0 + wn * C::WN + j * JW + (lane & (JW - 1));
    bias[j] = biasp ? ((const __attribute__((address_space(1))) float *)biasp)[col < eN ? col : eN - 1] : 0.f;
  }
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  auto put = [&](auto bf, int row, int col, float v) {
    if (EPI == EPI_TANH) v = tanh_fast(v);
    if constexpr (decltype(bf)::value)
      ((__attribute__((address_space(1))) bf16 *)outp)[(size_t)row * ldc + col] = to_bf16(v);
    else
      ((__attribute__((address_space(1))) float *)outp)[(size_t)row * ldc + col] = v;
  };
  auto epilogue = [&](auto bf) {
    if constexpr (C::M32) {
      // lane holds D[row = 8*(r/4) + 4*(lane/32) + r%4][col = lane % 32] of each 32x32 block
#pragma unroll
      for (int j = 0; j < C::FN32; ++j) {
        const int col = n0 + wn * C::WN + j * 32 + (lane & 31);
        if (col >= eN) continue;
#pragma unroll
        for (int i = 0; i < C::FM32; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = m0 + wm * C::WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (row < eM) put(bf, row, col, acc32[i][j][r] + bias[j]);
          }
      }
    } else {
      // lane holds D[row = 4*(lane/16) + r][col = lane % 16] of each 16x16 block
#pragma unroll
      for (int j = 0; j < C::FN; ++j) {
        const int col = n0 + wn * C::WN + j * 16 + (lane & 15);
        if (col >= eN) continue;
#pragma unroll
        for (int i = 0; i < C::FM; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row = m0 + wm * C::WM + i * 16 + (lane >> 4) * 4 + r;
            if (row < eM) put(bf, row, col, acc[i][j][r] + bias[j]);
          }
      }
    }
  };
  if (obf)
    epilogue(std::integral_constant<bool, true>{});
  else
    epilogue(std::integral_constant<bool, false>{});
}

// ---------------------------------------------------------------------------------------
// bf16 operands: weights streamed from global memory straight into registers.
//
// The weights are packed in the MFMA fragment order of the B operand (mt_load_weights): for
// 32-column block nb and 16-k step ks, 64 lanes x 16 bytes at ((nb * KSp + ks) * 64 + lane) * 16,
// lane l holding W[ks * 16 + (l / 32) * 8 + j][nb * 32 + l % 32], j < 8 (KSp = K_pad / 16, K_pad a
// multiple of 128, zero rows beyond K).  One coalesced 16-byte load per lane is one fragment.
//
// Block: 32 MB rows x 128 columns, two waves of 32 MB x 64 (MB x 2 blocks of 32x32x16 MFMAs;
// MB = 1 when 64-row blocks would leave most of the chip idle).  The block's activation rows
// pass through LDS in stages of 128 k (bf16, an fp32 operand rounded
// on the way), double-buffered from two register stages with one barrier per 8 k-steps; each
// wave's weight fragments come through a register ring refilled D k-steps ahead, so the only
// LDS traffic is the activations (written once, read by both waves).
constexpr int kWdCols = 128, kWdThreads = 128;
constexpr int kWdStageK = 128;                   // k per LDS stage (8 k-steps)
constexpr int kWdRowBytes = kWdStageK * 2 + 16;  // padded LDS row of one stage

template <typename AT, int EPI, int D, int MB>
__global__ __launch_bounds__(kWdThreads) void gemm_wd_kernel(Problems probs) {
  constexpr int kWdRows = 32 * MB;
  constexpr int kWdStage = kWdRows * kWdRowBytes;
  constexpr int RP = 4 * MB;  // staged rows per thread
  __shared__ __attribute__((aligned(16))) char lds[2 * kWdStage];
  constexpr int AV = (int)sizeof(AT) / 2;  // 16-byte source loads per 8-k vector
  const GemmProblem &P = probs.p[blockIdx.z];
  // problem fields read once into scalar registers (as references into the argument block
  // they would be re-read, each with a full wait, at every use in the epilogue)
  const int M = pin_s(P.M), N = pin_s(P.N), K = pin_s(P.K), lda = pin_s(P.lda), ldc = pin_s(P.ldc);
  const int KSp = pin_s(P.ldb) / 16;
  const int tilesM = (M + kWdRows - 1) / kWdRows;
  const int tilesN = (N + kWdCols - 1) / kWdCols;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  if (tile >= tilesM * tilesN) return;
  const int tm = tile % tilesM, tn = tile / tilesM;  // neighbours share a weight panel
  const int m0 = tm * kWdRows, n0 = tn * kWdCols;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- activation staging: thread t owns 8-k vector c = t % 16 of rows t / 16 + 8 p ----
  const int c = tid & 15;
  const char *a_src[RP];
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const int m = m0 + (tid >> 4) + 8 * p;
    int src = m < M ? m : 0;  // rows past M read row 0 and are never stored
    if (P.a_idx && m < M) {
      src = P.a_idx[m];
      if (src < 0 || src >= P.a_rows) {
        if (P.err) atomicOr(P.err, 1 << P.err_bit);
        src = src < 0 ? 0 : P.a_rows - 1;
      }
    }
    a_src[p] = (const char *)P.A + (size_t)src * lda * sizeof(AT);
  }
  typedef u32x4 StageRegs[RP][AV];
  auto load_stage = [&](int st, StageRegs &R) {
    const int k = st * kWdStageK + c * 8;
    const int kc = k < K ? k : K - 8;  // past K: the row's last vector (it meets zero weights)
#pragma unroll
    for (int p = 0; p < RP; ++p)
#pragma unroll
      for (int v = 0; v < AV; ++v) R[p][v] = *(const u32x4 *)(a_src[p] + (size_t)kc * sizeof(AT) + 16 * v);
  };
  auto store_stage = [&](int buf, const StageRegs &R) {
    char *base = lds + buf * kWdStage + c * 16;
#pragma unroll
    for (int p = 0; p < RP; ++p) {
      u32x4 val;
      if constexpr (AV == 2)
        val = pack_bf16x8(R[p][0], R[p][1]);
      else
        val = R[p][0];
      *(u32x4 *)(base + ((tid >> 4) + 8 * p) * kWdRowBytes) = val;
    }
  };

  // ---- weight fragments: this wave's blocks nb0, nb0 + 1; ring slot of k-step ks is ks % D ----
  const int nb0 = (n0 + wave * 64) >> 5;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)P.Bp, 0, ((N + kWdCols - 1) / kWdCols * kWdCols) * KSp * 32, 0x00020000);
  const int wvo = lane * 16;
  const int wb0 = nb0 * KSp * 1024, wstep1 = KSp * 1024;
  const int kslast = KSp - 1;
  u32x4 ring[D][2];
  auto fetch = [&](int ks, u32x4(&r)[2]) {
    const int so = wb0 + (ks < kslast ? ks : kslast) * 1024;  // clamped: in bounds, never used
    r[0] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo, so, 0);
    r[1] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo, so + wstep1, 0);
  };
#pragma unroll
  for (int d = 0; d < D; ++d) fetch(d, ring[d]);

  f32x16 acc[MB][2];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // 8 k-steps of stage st from LDS buffer buf; the ring slots of stage st are
  // (8 * (st & 1) + s) % D, static in the two-stage unrolled loop below.  The activation
  // fragments of k-step s + 1 are read before the MFMAs of k-step s (one wave per SIMD: nothing
  // else would cover the LDS latency).
  const int arow = lane & 31, akoff = (lane >> 5) * 16;
  auto compute = [&](int st, int buf, auto par) {
    const char *base = lds + buf * kWdStage + arow * kWdRowBytes + akoff;
    u32x4 af[MB], an[MB];
#pragma unroll
    for (int i = 0; i < MB; ++i) af[i] = *(const u32x4 *)(base + i * 32 * kWdRowBytes);
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      if (s + 1 < 8) {
#pragma unroll
        for (int i = 0; i < MB; ++i) an[i] = *(const u32x4 *)(base + i * 32 * kWdRowBytes + (s + 1) * 32);
      }
      u32x4(&slot)[2] = ring[(8 * decltype(par)::value + s) % D];
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bitcast16<bf16x8>(af[i]), bitcast16<bf16x8>(slot[j]),
                                                              acc[i][j], 0, 0, 0);
      fetch(st * 8 + s + D, slot);
      // keep each refill right behind the MFMAs that consumed its slot
      __builtin_amdgcn_sched_barrier(0);
      if (s + 1 < 8) {
#pragma unroll
        for (int i = 0; i < MB; ++i) af[i] = an[i];
      }
    }
  };

  // Stage st: multiply LDS buffer st & 1, load stage st + 2 into register stage st & 1 and
  // write register stage (st + 1) & 1 (loaded one stage earlier) into the other buffer.
  // Stage indices clamp to the last stage, so the body is branch-free.
  const int nst = KSp / 8;
  const int last = nst - 1;
  StageRegs s0, s1;
  load_stage(0, s0);
  load_stage(1 < last ? 1 : last, s1);
  store_stage(0, s0);
  __syncthreads();
  auto stage = [&](int st, StageRegs &cur, StageRegs &nxt, auto par) {
    load_stage(st + 2 < last ? st + 2 : last, cur);
    __builtin_amdgcn_sched_barrier(0);
    compute(st, decltype(par)::value, par);
    store_stage(decltype(par)::value ^ 1, nxt);
    __syncthreads();
  };
  int st = 0;
  for (; st + 1 < nst; st += 2) {
    stage(st, s0, s1, std::integral_constant<int, 0>{});
    stage(st + 1, s1, s0, std::integral_constant<int, 1>{});
  }
  if (st < nst) stage(st, s0, s1, std::integral_constant<int, 0>{});

  // ---- epilogue: lane holds D[row = 8*(r/4) + 4*(lane/32) + r%4][col = lane % 32] ----
  const int obf = pin_s(P.out_bf16);
  const float *const biasp = pin_s(P.bias);
  char *const outp = (char *)pin_s(P.out);
  // The bias values are loaded before any store and waited for once: a load between the stores
  // would make every store wait for all earlier stores (the memory counter counts both).
  float bias[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int col = n0 + wave * 64 + j * 32 + (lane & 31);
    bias[j] = biasp ? ((const __attribute__((address_space(1))) float *)biasp)[col < N ? col : N - 1] : 0.f;
  }
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  auto epilogue = [&](auto bf) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wave * 64 + j * 32 + (lane & 31);
      if (col >= N) continue;
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (row >= M) continue;
          float v = acc[i][j][r] + bias[j];
          if (EPI == EPI_TANH) v = tanh_fast(v);
          if constexpr (decltype(bf)::value)
            ((__attribute__((address_space(1))) bf16 *)outp)[(size_t)row * ldc + col] = to_bf16(v);
          else
            ((__attribute__((address_space(1))) float *)outp)[(size_t)row * ldc + col] = v;
        }
    }
  };
  if (obf)
    epilogue(std::integral_constant<bool, true>{});
  else
    epilogue(std::integral_constant<bool, false>{});
}

template <typename AT, int EPI, int MB>
static hipError_t go_wd_mb(const Problems &ps, int nprob, hipStream_t st) {
  int maxt = 0;
  for (int i = 0; i < nprob; ++i) {
    const int t = ((ps.p[i].M + 32 * MB - 1) / (32 * MB)) * ((ps.p[i].N + kWdCols - 1) / kWdCols);
    maxt = t > maxt ? t : maxt;
  }
  if (maxt == 0) return hipSuccess;
  // ring depth: 16 k-steps when the activation stages leave the registers for it
  constexpr int D = sizeof(AT) == 2 || MB == 1 ? 16 : 8;
  hipLaunchKernelGGL((gemm_wd_kernel<AT, EPI, D, MB>), dim3(maxt, 1, nprob), dim3(kWdThreads), 0, st, ps);
  return hipGetLastError();
}

template <typename AT, int EPI>
static hipError_t go_wd(const Problems &ps, int nprob, hipStream_t st) {
  long t64 = 0;
  for (int i = 0; i < nprob; ++i) {
    const GemmProblem &p = ps.p[i];
    if (p.ldb % kWdStageK != 0 || p.K > p.ldb || p.K % 8 != 0) return hipErrorInvalidValue;
    t64 += (long)((p.M + 63) / 64) * ((p.N + kWdCols - 1) / kWdCols);
  }
  // 64-row blocks once they cover the chip, else 32-row blocks (twice the blocks, each wave
  // half the work)
  return t64 >= 256 ? go_wd_mb<AT, EPI, 2>(ps, nprob, st) : go_wd_mb<AT, EPI, 1>(ps, nprob, st);
}

// ---------------------------------------------------------------------------------------
// fp32 operands: one wave per (16 TA) x (16 TB) output tile, both operands straight from global
// memory (at fp32 rates the MFMAs need only a few bytes per cycle, so no LDS staging).
//
// v_mfma_f32_16x16x4_f32 takes one fp32 per lane per operand: A lane l holds row l % 16 and k
// (l / 16), B lane l holds column l % 16 and k (l / 16).  A 16-byte vector per lane holds the k
// quadruple 4 (l / 16) + e, e < 4, of one 16-k step and feeds MFMA e, so the four MFMAs of a step
// cover its 16 k once (the same assignment on both operands).  The weights are packed at load
// time in that order: for 16-column block nb and 16-k step ks, 64 lanes x 16 bytes at
// ((nb * KSp + ks) * 64 + lane) * 16, lane l holding W[ks * 16 + (l / 16) * 4 + e][nb * 16 + l % 16]
// (KSp = K_pad / 16).  The activation vector of lane l is A[row][ks * 16 + (l / 16) * 4 ..], one
// 16-byte load.  Both come through a register ring refilled D steps ahead.
//
// Tiles are sized per launch so that the wave count fits the chip's 1024 SIMDs (go_f32): at these
// shapes the time is set by the SIMD with the most work.
template <int TA, int TB, int EPI, int D, int U>
__global__ __launch_bounds__(256) void gemm_f32_kernel(Problems probs) {
  const GemmProblem &P = probs.p[blockIdx.z];
  const int M = pin_s(P.M), N = pin_s(P.N), K = pin_s(P.K), lda = pin_s(P.lda), ldc = pin_s(P.ldc);
  const int KSp = pin_s(P.ldb) / 16;
  const int tilesM = (M + 16 * TA - 1) / (16 * TA);
  const int tilesN = (N + 16 * TB - 1) / (16 * TB);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tile = xcd_remap(blockIdx.x, gridDim.x) * 4 + wave;  // four tiles per workgroup
  if (tile >= tilesM * tilesN) return;
  const int tm = tile % tilesM, tn = tile / tilesM;  // neighbours share a weight panel
  const int m0 = tm * 16 * TA, n0 = tn * 16 * TB;
  const int lr = lane & 15, lk = (lane >> 4) * 4;

  // activation rows of this lane (gathered, clamped; rows past M read row 0, never stored), as
  // byte offsets into a buffer view of A
  const __amdgpu_buffer_rsrc_t ars =
      __builtin_amdgcn_make_buffer_rsrc((void *)P.A, 0, P.a_rows * lda * 4, 0x00020000);
  int a_off[TA];
#pragma unroll
  for (int i = 0; i < TA; ++i) {
    const int m = m0 + 16 * i + lr;
    int src = m < M ? m : 0;
    if (P.a_idx && m < M) {
      src = P.a_idx[m];
      if (src < 0 || src >= P.a_rows) {
        if (P.err) atomicOr(P.err, 1 << P.err_bit);
        src = src < 0 ? 0 : P.a_rows - 1;
      }
    }
    a_off[i] = src * lda * 4;
  }
  const __amdgpu_buffer_rsrc_t wrs =
      __builtin_amdgcn_make_buffer_rsrc((void *)P.Bp, 0, tilesN * TB * KSp * 1024, 0x00020000);
  const int wvo = lane * 16;
  const int wb0 = (n0 >> 4) * KSp * 1024;
  const int kslast = KSp - 1;

  struct Slot {
    u32x4 a[TA], b[TB];
  };
  Slot ring[D];
  auto fetch = [&](int ks, Slot &r) {
    const int kc = ks < kslast ? ks : kslast;  // clamped: in bounds, never used
    int k = kc * 16 + lk;
    k = k < K ? k : K - 4;  // past K: the row's last vector (it meets zero weights)
#pragma unroll
    for (int i = 0; i < TA; ++i) r.a[i] = __builtin_amdgcn_raw_buffer_load_b128(ars, a_off[i] + k * 4, 0, 0);
#pragma unroll
    for (int j = 0; j < TB; ++j) r.b[j] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo, wb0 + (j * KSp + kc) * 1024, 0);
  };
#pragma unroll
  for (int d = 0; d < D; ++d) fetch(d, ring[d]);

  f32x4 acc[TA][TB];
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // the ring index of step ks is ks % D; the loop advances U steps per iteration (KSp % U == 0,
  // U a multiple of D).  The compiler drains the memory counter at the loop header, so the
  // longer the body, the rarer the drain.
  for (int ks0 = 0; ks0 < KSp; ks0 += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int d = u % D;
      float fa[TA][4], fb[TB][4];
#pragma unroll
      for (int i = 0; i < TA; ++i) __builtin_memcpy(fa[i], &ring[d].a[i], 16);
#pragma unroll
      for (int j = 0; j < TB; ++j) __builtin_memcpy(fb[j], &ring[d].b[j], 16);
      // element e of every vector feeds MFMA e; the TA x TB accumulators alternate between
      // dependent MFMAs
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < TA; ++i)
#pragma unroll
          for (int j = 0; j < TB; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i][e], fb[j][e], acc[i][j], 0, 0, 0);
      // the refill of a slot goes behind the MFMAs that read it (hoisted above them, its loads
      // would need fresh registers and a wait for every load in flight)
      __builtin_amdgcn_sched_barrier(0);
      fetch(ks0 + u + D, ring[d]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // ---- epilogue: lane holds D[row = 4 * (lane / 16) + r][col = lane % 16] of each 16x16 block;
  // the bias values are loaded before any store and waited for once ----
  const int obf = pin_s(P.out_bf16);
  const float *const biasp = pin_s(P.bias);
  char *const outp = (char *)pin_s(P.out);
  float bias[TB];
#pragma unroll
  for (int j = 0; j < TB; ++j) {
    const int col = n0 + 16 * j + lr;
    bias[j] = biasp ? ((const __attribute__((address_space(1))) float *)biasp)[col < N ? col : N - 1] : 0.f;
  }
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  auto epilogue = [&](auto bf) {
#pragma unroll
    for (int j = 0; j < TB; ++j) {
      const int col = n0 + 16 * j + lr;
      if (col >= N) continue;
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m0 + 16 * i + (lane >> 4) * 4 + r;
          if (row >= M) continue;
          float v = acc[i][j][r] + bias[j];
          if (EPI == EPI_TANH) v = tanh_fast(v);
          if constexpr (decltype(bf)::value)
            ((__attribute__((address_space(1))) bf16 *)outp)[(size_t)row * ldc + col] = to_bf16(v);
          else
            ((__attribute__((address_space(1))) float *)outp)[(size_t)row * ldc + col] = v;
        }
    }
  };
  if (obf)
    epilogue(std::integral_constant<bool, true>{});
  else
    epilogue(std::integral_constant<bool, false>{});
}

template <int TA, int TB, int EPI>
static hipError_t go_f32_t(const Problems &ps, int nprob, hipStream_t st) {
  int maxw = 0;
  bool deep = TA + TB <= 4;  // ring depth in 16-k steps: 8 for small tiles when it divides the steps
  bool long16 = true;        // 16 steps per loop iteration
  for (int i = 0; i < nprob; ++i) {
    const int w = ((ps.p[i].M + 16 * TA - 1) / (16 * TA)) * ((ps.p[i].N + 16 * TB - 1) / (16 * TB));
    maxw = w > maxw ? w : maxw;
    deep = deep && (ps.p[i].ldb / 16) % 8 == 0;
    long16 = long16 && (ps.p[i].ldb / 16) % 16 == 0;
  }
  if (maxw == 0) return hipSuccess;
  const dim3 grid((maxw + 3) / 4, 1, nprob);
  if constexpr (TA + TB <= 4) {
    if (deep && long16) hipLaunchKernelGGL((gemm_f32_kernel<TA, TB, EPI, 8, 16>), grid, dim3(256), 0, st, ps);
    else if (deep) hipLaunchKernelGGL((gemm_f32_kernel<TA, TB, EPI, 8, 8>), grid, dim3(256), 0, st, ps);
    else hipLaunchKernelGGL((gemm_f32_kernel<TA, TB, EPI, 4, 4>), grid, dim3(256), 0, st, ps);
  } else {
    if (long16) hipLaunchKernelGGL((gemm_f32_kernel<TA, TB, EPI, 4, 16>), grid, dim3(256), 0, st, ps);
    else hipLaunchKernelGGL((gemm_f32_kernel<TA, TB, EPI, 4, 4>), grid, dim3(256), 0, st, ps);
  }
  return hipGetLastError();
}

// Tile choice: the fewest rounds of waves over the chip's SIMDs, each round costing the tile's
// MFMA count (TA x TB blocks), among a few shapes with enough accumulators per wave to keep the
// matrix core busy.
template <int EPI>
static hipError_t go_f32(const Problems &ps, int nprob, hipStream_t st) {
  for (int i = 0; i < nprob; ++i) {
    const GemmProblem &p = ps.p[i];
    if (p.ldb % 64 != 0 || p.K > p.ldb || p.K % 4 != 0 || p.lda % 4 != 0) return hipErrorInvalidValue;
  }
  static const int shapes[][2] = {{3, 3}, {3, 4}, {3, 5}, {3, 2}, {2, 4}, {4, 4}, {2, 2}, {1, 2}};
  constexpr int kSimds = 1024;
  long best = -1;
  int bi = 0;
  for (int s = 0; s < 8; ++s) {
    long w = 0;
    for (int i = 0; i < nprob; ++i)
      w += (long)((ps.p[i].M + 16 * shapes[s][0] - 1) / (16 * shapes[s][0])) *
           ((ps.p[i].N + 16 * shapes[s][1] - 1) / (16 * shapes[s][1]));
    const long cost = ((w + kSimds - 1) / kSimds) * shapes[s][0] * shapes[s][1];
    if (best < 0 || cost < best) {
      best = cost;
      bi = s;
    }
  }
  switch (bi) {
    case 0: return go_f32_t<3, 3, EPI>(ps, nprob, st);
    case 1: return go_f32_t<3, 4, EPI>(ps, nprob, st);
    case 2: return go_f32_t<3, 5, EPI>(ps, nprob, st);
    case 3: return go_f32_t<3, 2, EPI>(ps, nprob, st);
    case 4: return go_f32_t<2, 4, EPI>(ps, nprob, st);
    case 5: return go_f32_t<4, 4, EPI>(ps, nprob, st);
    case 6: return go_f32_t<2, 2, EPI>(ps, nprob, st);
    default: return go_f32_t<1, 2, EPI>(ps, nprob, st);
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
  // CUs idle, else 64 x 64 (at these shapes the time follows the number of tiles per CU, and
  // 64 x 128 tiles divide worse over 256 CUs)
  long t128 = 0, t64 = 0;
  for (int i = 0; i < nprob; ++i) {
    t128 += (long)((ps.p[i].M + 127) / 128) * ((ps.p[i].N + 127) / 128);
    t64 += (long)((ps.p[i].M + 63) / 64) * ((ps.p[i].N + 63) / 64);
  }
  if (t128 >= 512) return go<CT, AT, EPI, 128, 128>(ps, nprob, st);
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
  if (!bf16_mma) return epi == EPI_TANH ? go_f32<EPI_TANH>(ps, nprob, st) : go_f32<EPI_STORE>(ps, nprob, st);
  if (probs[0].a_bf16)
    return epi == EPI_TANH ? go_wd<bf16, EPI_TANH>(ps, nprob, st) : go_wd<bf16, EPI_STORE>(ps, nprob, st);
  return epi == EPI_TANH ? go_wd<float, EPI_TANH>(ps, nprob, st) : go_wd<float, EPI_STORE>(ps, nprob, st);
}

}  // namespace mt
