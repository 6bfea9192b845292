// Matrix products of the decoder step on CDNA4 matrix cores:
// out[m, n] = sum_k A[m, k] * W[k, n] (+ bias[n]), tanh optional, fp32 or bf16 output.
// The A operand may be gathered by a row index (token -> embedding row, backpointer -> state
// row); every problem of one launch has the same A element type.  W is packed at load time
// (mt_load_weights) in the MFMA fragment order of its kernel, zero padded to [K_pad][N_pad]:
//  * fp32 (gemm_f32_kernel): 16 x 16 x 4 MFMAs, both operands straight from global memory;
//  * bf16 (gemm_wd_kernel): 32 x 32 x 16 MFMAs, weights straight from global memory and the
//    activations through a small LDS ring.
// Loads are unconditional and nothing is masked: a row past M reads row 0 and its output row is
// never stored, and a vector past K reads the row's last in-range vector, which meets the zero
// padding of the packed weights (finite x 0 adds nothing).  Epilogues load the bias before any
// store and read the problem fields into scalar registers once: a load between the stores
// would make every store wait for all earlier ones (the memory counter counts both).
#include "mt_internal.h"

namespace mt {

template <typename T>
__device__ __forceinline__ T pin_s(T x) {  // keep a uniform value in a scalar register
  asm volatile("" : "+s"(x));
  return x;
}

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
  // rows counted on the device, when given, bound the rows read and stored
  const int *const mdp = pin_s(P.m_dev);
  int Mv = M;
  if (mdp) {
    const int md = *(const __attribute__((address_space(1))) int *)mdp;
    Mv = md < M ? md : M;
  }
  if (m0 >= Mv) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- activation staging: thread t owns 8-k vector c = t % 16 of rows t / 16 + 8 p ----
  const int c = tid & 15;
  const char *a_src[RP];
#pragma unroll
  for (int p = 0; p < RP; ++p) {
    const int m = m0 + (tid >> 4) + 8 * p;
    int src = m < Mv ? m : 0;  // rows past the count read row 0 and are never stored
    if (P.a_idx && m < Mv) {
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
  // EPI_SCATTER: the output row of each stored row is its (clamped) gather row
  int orow[EPI == EPI_SCATTER ? MB : 1][16];
  if constexpr (EPI == EPI_SCATTER) {
    const int32_t *const aix = pin_s(P.a_idx);
    const int arows = pin_s(P.a_rows);
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int g = row < Mv ? ((const __attribute__((address_space(1))) int32_t *)aix)[row] : 0;
        orow[i][r] = g < 0 ? 0 : g >= arows ? arows - 1 : g;
      }
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
          if (row >= Mv) continue;
          float v = acc[i][j][r] + bias[j];
          if (EPI == EPI_TANH) v = tanh_fast(v);
          int orw = row;
          if constexpr (EPI == EPI_SCATTER) orw = orow[i][r];
          if constexpr (decltype(bf)::value)
            ((__attribute__((address_space(1))) bf16 *)outp)[(size_t)orw * ldc + col] = to_bf16(v);
          else
            ((__attribute__((address_space(1))) float *)outp)[(size_t)orw * ldc + col] = v;
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
// fp32 operands: (BLK TA) x (BLK TB) output tiles, each computed by S waves of one workgroup that
// split its k-steps and add their partial sums through LDS; both operands straight from global
// memory (at fp32 rates the MFMAs need only a few bytes per cycle, so no LDS staging).
//
// BLK = 16: v_mfma_f32_16x16x4_f32 takes one fp32 per lane per operand, A lane l holding row
// l % 16 and k (l / 16), B lane l column l % 16 and k (l / 16).  A 16-byte vector per lane holds
// the k quadruple 4 (l / 16) + e, e < 4, of one 16-k step and feeds MFMA e, so the four MFMAs of
// a step cover its 16 k once (the same assignment on both operands).
// BLK = 32: v_mfma_f32_32x32x2f32, A lane l holding row l % 32 and k (l / 32); a 16-byte vector
// holds k = 4 (l / 32) + e of one 8-k step, again feeding MFMA e.  This form sustains a higher
// fraction of the matrix core's rate (86% against 74% in pure-MFMA loops, about 5% more in this
// kernel), at the price of coarser tiles.
// The weights are packed in the order of their form (mt_load_weights picks it per matrix): for
// BLK-column block nb and step ks, 64 lanes x 16 bytes at ((nb * KS + ks) * 64 + lane) * 16
// (KS = K_pad / (256 / BLK)).  The activation vector of lane l is A[row][step k0 + its k
// quadruple], one 16-byte load.  Both come through a register ring refilled D steps ahead.
//
// Tile shape and split are chosen per launch (go_f32) so that the waves spread evenly over the
// chip's 1024 SIMDs: at these shapes the time is set by the SIMD with the most work.
template <int BLK>
struct F32Form {
  static constexpr int KSTEP = 256 / BLK;   // k per step (one 16-byte vector per lane)
  static constexpr int NACC = BLK * BLK / 64;  // accumulator registers per lane per block
  static constexpr int HALF = 64 / BLK;     // lane groups of the k quadruples
};

template <int BLK, int TA, int TB, int S, int EPI, int D, int U>
__global__ __launch_bounds__(256) void gemm_f32_kernel(Problems probs) {
  using F = F32Form<BLK>;
  typedef __attribute__((__vector_size__(F::NACC * sizeof(float)))) float accv;
  constexpr int TPB = 4 / S;  // tiles per workgroup (four waves)
  __shared__ __attribute__((aligned(16))) float red[S > 1 ? TPB * (S - 1) * TA * TB * F::NACC * 64 : 1];
  const GemmProblem &P = probs.p[blockIdx.z];
  const int M = pin_s(P.M), N = pin_s(P.N), K = pin_s(P.K), lda = pin_s(P.lda), ldc = pin_s(P.ldc);
  const int KSp = pin_s(P.ldb) / F::KSTEP;
  const int tilesM = (M + BLK * TA - 1) / (BLK * TA);
  const int tilesN = (N + BLK * TB - 1) / (BLK * TB);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int part = wave % S, slot_t = wave / S;
  const int tile = xcd_remap(blockIdx.x, gridDim.x) * TPB + slot_t;
  // rows counted on the device, when given, bound the rows read and stored
  const int *const mdp = pin_s(P.m_dev);
  int Mv = M;
  if (mdp) {
    const int md = *(const __attribute__((address_space(1))) int *)mdp;
    Mv = md < M ? md : M;
  }
  // a wave without a tile still takes part in the workgroup's barrier below
  const bool has_tile = tile < tilesM * tilesN;
  const int tl = has_tile ? tile : 0;
  const int tm = tl % tilesM, tn = tl / tilesM;  // neighbours share a weight panel
  const int m0 = tm * BLK * TA, n0 = tn * BLK * TB;
  const bool live = has_tile && m0 < Mv;
  // without a split there is no barrier, so a wave without a tile (or whose rows all lie past
  // the device count) ends here; with one it computes a stand-in tile for the barrier's sake
  if constexpr (S == 1)
    if (!live) return;
  const int lr = lane & (BLK - 1), lk = (lane / BLK) * 4;
  const int ks_begin = part * (KSp / S), ks_end = ks_begin + KSp / S;

  // activation rows of this lane (gathered, clamped; rows past M read row 0, never stored), as
  // byte offsets into a buffer view of A
  const __amdgpu_buffer_rsrc_t ars =
      __builtin_amdgcn_make_buffer_rsrc((void *)P.A, 0, P.a_rows * lda * 4, 0x00020000);
  int a_off[TA];
#pragma unroll
  for (int i = 0; i < TA; ++i) {
    const int m = m0 + BLK * i + lr;
    int src = m < Mv ? m : 0;
    if (live && P.a_idx && m < Mv) {
      src = P.a_idx[m];
      if (src < 0 || src >= P.a_rows) {
        if (P.err) atomicOr(P.err, 1 << P.err_bit);
        src = src < 0 ? 0 : P.a_rows - 1;
      }
    }
    a_off[i] = src * lda * 4;
  }
  // the view covers the column blocks that exist (the packing pads N further, to N_pad, but a
  // tile may reach past even that): fragments of blocks beyond N read as zero and their
  // columns are never stored
  const __amdgpu_buffer_rsrc_t wrs =
      __builtin_amdgcn_make_buffer_rsrc((void *)P.Bp, 0, (N + BLK - 1) / BLK * KSp * 1024, 0x00020000);
  const int wvo = lane * 16;
  const int wb0 = (n0 / BLK) * KSp * 1024;
  const int kslast = ks_end - 1;

  struct Slot {
    u32x4 a[TA], b[TB];
  };
  Slot ring[D];
  auto fetch = [&](int ks, Slot &r) {
    const int kc = ks < kslast ? ks : kslast;  // clamped: in bounds, never used
    int k = kc * F::KSTEP + lk;
    k = k < K ? k : K - 4;  // past K: the row's last vector (it meets zero weights)
#pragma unroll
    for (int i = 0; i < TA; ++i) r.a[i] = __builtin_amdgcn_raw_buffer_load_b128(ars, a_off[i] + k * 4, 0, 0);
#pragma unroll
    for (int j = 0; j < TB; ++j) r.b[j] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo, wb0 + (j * KSp + kc) * 1024, 0);
  };
#pragma unroll
  for (int d = 0; d < D; ++d) fetch(ks_begin + d, ring[d]);

  accv acc[TA][TB];
#pragma unroll
  for (int i = 0; i < TA; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j)
#pragma unroll
      for (int r = 0; r < F::NACC; ++r) acc[i][j][r] = 0.f;

  // the ring index of step ks is (ks - ks_begin) % D; the loop advances U steps per iteration
  // ((KSp / S) % U == 0, U a multiple of D).  The compiler drains the memory counter at the loop
  // header, so the longer the body, the rarer the drain.
  for (int ks0 = ks_begin; ks0 < ks_end; ks0 += U) {
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
          for (int j = 0; j < TB; ++j) {
            if constexpr (BLK == 16)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i][e], fb[j][e], acc[i][j], 0, 0, 0);
            else
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[i][e], fb[j][e], acc[i][j], 0, 0, 0);
          }
      // the refill of a slot goes behind the MFMAs that read it (hoisted above them, its loads
      // would need fresh registers and a wait for every load in flight)
      __builtin_amdgcn_sched_barrier(0);
      fetch(ks0 + u + D, ring[d]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // ---- the split's partial sums: parts 1.. write theirs, part 0 adds them in part order ----
  if constexpr (S > 1) {
    constexpr int PER = TA * TB * F::NACC;
    if (part > 0) {
      float *mine = red + (size_t)((slot_t * (S - 1) + part - 1) * PER) * 64;
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j)
#pragma unroll
          for (int r = 0; r < F::NACC; ++r) mine[((i * TB + j) * F::NACC + r) * 64 + lane] = acc[i][j][r];
    }
    __syncthreads();
    if (part > 0) return;
#pragma unroll
    for (int q = 1; q < S; ++q) {
      const float *o = red + (size_t)((slot_t * (S - 1) + q - 1) * PER) * 64;
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int j = 0; j < TB; ++j)
#pragma unroll
          for (int r = 0; r < F::NACC; ++r) acc[i][j][r] += o[((i * TB + j) * F::NACC + r) * 64 + lane];
    }
  }
  if (!live) return;

  // ---- epilogue: lane holds D[row][col = lane % BLK] of each block, row = 4 * (lane / 16) + r
  // (BLK 16) or 8 * (r / 4) + 4 * (lane / 32) + r % 4 (BLK 32); the bias values are loaded before
  // any store and waited for once ----
  const int obf = pin_s(P.out_bf16);
  const float *const biasp = pin_s(P.bias);
  char *const outp = (char *)pin_s(P.out);
  float bias[TB];
#pragma unroll
  for (int j = 0; j < TB; ++j) {
    const int col = n0 + BLK * j + lr;
    bias[j] = biasp ? ((const __attribute__((address_space(1))) float *)biasp)[col < N ? col : N - 1] : 0.f;
  }
  auto row_of = [&](int i, int r) {
    return m0 + BLK * i + (BLK == 16 ? (lane >> 4) * 4 + r : 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3));
  };
  // EPI_SCATTER: the output row of each stored row is its (clamped) gather row
  int orow[EPI == EPI_SCATTER ? TA : 1][EPI == EPI_SCATTER ? F::NACC : 1];
  if constexpr (EPI == EPI_SCATTER) {
    const int32_t *const aix = pin_s(P.a_idx);
    const int arows = pin_s(P.a_rows);
#pragma unroll
    for (int i = 0; i < TA; ++i)
#pragma unroll
      for (int r = 0; r < F::NACC; ++r) {
        const int row = row_of(i, r);
        const int g = row < Mv ? ((const __attribute__((address_space(1))) int32_t *)aix)[row] : 0;
        orow[i][r] = g < 0 ? 0 : g >= arows ? arows - 1 : g;
      }
  }
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  auto epilogue = [&](auto bf) {
#pragma unroll
    for (int j = 0; j < TB; ++j) {
      const int col = n0 + BLK * j + lr;
      if (col >= N) continue;
#pragma unroll
      for (int i = 0; i < TA; ++i)
#pragma unroll
        for (int r = 0; r < F::NACC; ++r) {
          const int row = row_of(i, r);
          if (row >= Mv) continue;
          float v = acc[i][j][r] + bias[j];
          if (EPI == EPI_TANH) v = tanh_fast(v);
          int orw = row;
          if constexpr (EPI == EPI_SCATTER) orw = orow[i][r];
          if constexpr (decltype(bf)::value)
            ((__attribute__((address_space(1))) bf16 *)outp)[(size_t)orw * ldc + col] = to_bf16(v);
          else
            ((__attribute__((address_space(1))) float *)outp)[(size_t)orw * ldc + col] = v;
        }
    }
  };
  if (obf)
    epilogue(std::integral_constant<bool, true>{});
  else
    epilogue(std::integral_constant<bool, false>{});
}

template <int BLK, int TA, int TB, int S, int EPI>
static hipError_t go_f32_t(const Problems &ps, int nprob, hipStream_t st) {
  int maxw = 0;
  bool deep = TA + TB <= 4;  // ring depth in steps: 8 for small tiles when it divides the steps
  bool long16 = true;        // 16 steps per loop iteration
  for (int i = 0; i < nprob; ++i) {
    const int w = ((ps.p[i].M + BLK * TA - 1) / (BLK * TA)) * ((ps.p[i].N + BLK * TB - 1) / (BLK * TB));
    maxw = w > maxw ? w : maxw;
    const int steps = ps.p[i].ldb / F32Form<BLK>::KSTEP / S;
    deep = deep && steps % 8 == 0;
    long16 = long16 && steps % 16 == 0;
  }
  if (maxw == 0) return hipSuccess;
  constexpr int TPB = 4 / S;
  const dim3 grid((maxw + TPB - 1) / TPB, 1, nprob);
  if constexpr (TA + TB <= 4) {
    if (deep && long16) hipLaunchKernelGGL((gemm_f32_kernel<BLK, TA, TB, S, EPI, 8, 16>), grid, dim3(256), 0, st, ps);
    else if (deep) hipLaunchKernelGGL((gemm_f32_kernel<BLK, TA, TB, S, EPI, 8, 8>), grid, dim3(256), 0, st, ps);
    else hipLaunchKernelGGL((gemm_f32_kernel<BLK, TA, TB, S, EPI, 4, 4>), grid, dim3(256), 0, st, ps);
  } else {
    if (long16) hipLaunchKernelGGL((gemm_f32_kernel<BLK, TA, TB, S, EPI, 4, 16>), grid, dim3(256), 0, st, ps);
    else hipLaunchKernelGGL((gemm_f32_kernel<BLK, TA, TB, S, EPI, 4, 4>), grid, dim3(256), 0, st, ps);
  }
  return hipGetLastError();
}

// Tile shapes per form: TA x TB blocks of BLK x BLK, k split S.
struct F32Shape {
  int ta, tb, s;
};
static const F32Shape kShapes16[] = {{3, 3, 1}, {3, 4, 1}, {3, 5, 1}, {3, 2, 1}, {2, 4, 1}, {1, 2, 1},
                                     {3, 3, 2}, {3, 4, 2}, {3, 5, 2}, {3, 2, 2}, {1, 2, 4}};
static const F32Shape kShapes32[] = {{1, 3, 1}, {2, 2, 1}, {1, 4, 1}, {2, 3, 1}, {1, 2, 1}, {1, 2, 2}};

// Cost of the best shape of a form for (rows, columns, k-steps): the SIMD with the most work
// receives ceil(waves / 1024) waves of TA * TB / S block-steps each, counted in 16x16x4 MFMA
// time (a 32 x 32 block-step is four 16 x 16 ones at the 32x32x2 form's better rate: 0.95 of
// their time in this kernel at the decoder's shapes).  Also measured there: a k split costs a little more than the same
// work unsplit (its partial sums and the second ring fill), fewer than 6 accumulators leave
// dependent 16x16x4 MFMAs too close together, and between equal costs the shape with more
// waves hides latency better.  A split needs at least 4 steps per part.
static double f32_best(int blk, const long *rows, const long *cols, int nprob, int steps, int *which) {
  const F32Shape *sh = blk == 16 ? kShapes16 : kShapes32;
  const int n = blk == 16 ? (int)(sizeof(kShapes16) / sizeof(kShapes16[0])) : (int)(sizeof(kShapes32) / sizeof(kShapes32[0]));
  double best = -1.0;
  long best_w = 0;
  *which = 0;
  for (int s = 0; s < n; ++s) {
    const F32Shape &h = sh[s];
    if (steps / h.s < 4 || steps % (4 * h.s) != 0) continue;
    long w = 0;
    for (int i = 0; i < nprob; ++i) w += ((rows[i] + blk * h.ta - 1) / (blk * h.ta)) * ((cols[i] + blk * h.tb - 1) / (blk * h.tb));
    w *= h.s;
    const long per = (w + 1023) / 1024;
    double cost = (double)per * h.ta * h.tb / h.s * (h.s > 1 ? 1.05 : 1.0);
    if (blk == 16) cost /= h.ta * h.tb >= 6 ? 1.0 : 0.6;
    else cost *= 4 * 0.95;
    if (best < 0 || cost < best - 1e-9 || (cost < best + 1e-9 && w > best_w)) {
      best = cost;
      best_w = w;
      *which = s;
    }
  }
  return best;
}

int gemm_f32_weight_block(long rows, long N, long K) {
  const long kp = (K + 63) / 64 * 64;
  int w16, w32;
  const double c16 = f32_best(16, &rows, &N, 1, (int)(kp / 16), &w16);
  const double c32 = f32_best(32, &rows, &N, 1, (int)(kp / 8), &w32);
  return (c32 >= 0 && c32 < c16) ? 32 : 16;
}

template <int EPI>
static hipError_t go_f32(const Problems &ps, int nprob, hipStream_t st) {
  const int blk = ps.p[0].wblk == 32 ? 32 : 16;
  int minsteps = 1 << 30;
  long rows[2], cols[2];
  for (int i = 0; i < nprob; ++i) {
    const GemmProblem &p = ps.p[i];
    if (p.ldb % 64 != 0 || p.K > p.ldb || p.K % 4 != 0 || p.lda % 4 != 0) return hipErrorInvalidValue;
    if ((p.wblk == 32 ? 32 : 16) != blk) return hipErrorInvalidValue;
    const int steps = p.ldb / F32Form<16>::KSTEP * (blk == 32 ? 2 : 1);
    minsteps = steps < minsteps ? steps : minsteps;
    rows[i] = p.M;
    cols[i] = p.N;
  }
  int bi = 0;
  if (f32_best(blk, rows, cols, nprob, minsteps, &bi) < 0) return hipErrorInvalidValue;
  if (blk == 32) {
    switch (bi) {
      case 0: return go_f32_t<32, 1, 3, 1, EPI>(ps, nprob, st);
      case 1: return go_f32_t<32, 2, 2, 1, EPI>(ps, nprob, st);
      case 2: return go_f32_t<32, 1, 4, 1, EPI>(ps, nprob, st);
      case 3: return go_f32_t<32, 2, 3, 1, EPI>(ps, nprob, st);
      case 4: return go_f32_t<32, 1, 2, 1, EPI>(ps, nprob, st);
      default: return go_f32_t<32, 1, 2, 2, EPI>(ps, nprob, st);
    }
  }
  switch (bi) {
    case 0: return go_f32_t<16, 3, 3, 1, EPI>(ps, nprob, st);
    case 1: return go_f32_t<16, 3, 4, 1, EPI>(ps, nprob, st);
    case 2: return go_f32_t<16, 3, 5, 1, EPI>(ps, nprob, st);
    case 3: return go_f32_t<16, 3, 2, 1, EPI>(ps, nprob, st);
    case 4: return go_f32_t<16, 2, 4, 1, EPI>(ps, nprob, st);
    case 5: return go_f32_t<16, 1, 2, 1, EPI>(ps, nprob, st);
    case 6: return go_f32_t<16, 3, 3, 2, EPI>(ps, nprob, st);
    case 7: return go_f32_t<16, 3, 4, 2, EPI>(ps, nprob, st);
    case 8: return go_f32_t<16, 3, 5, 2, EPI>(ps, nprob, st);
    case 9: return go_f32_t<16, 3, 2, 2, EPI>(ps, nprob, st);
    default: return go_f32_t<16, 1, 2, 4, EPI>(ps, nprob, st);
  }
}

hipError_t launch_gemm(int bf16_mma, const GemmProblem *probs, int nprob, Epilogue epi, hipStream_t st) {
  Problems ps{};
  for (int i = 0; i < nprob; ++i) {
    ps.p[i] = probs[i];
    if (probs[i].a_bf16 != probs[0].a_bf16 || (probs[i].a_bf16 && !bf16_mma)) return hipErrorInvalidValue;
    if (epi == EPI_SCATTER && !probs[i].a_idx) return hipErrorInvalidValue;
  }
  if (!bf16_mma) {
    if (epi == EPI_SCATTER) return go_f32<EPI_SCATTER>(ps, nprob, st);
    return epi == EPI_TANH ? go_f32<EPI_TANH>(ps, nprob, st) : go_f32<EPI_STORE>(ps, nprob, st);
  }
  if (epi == EPI_SCATTER)  // the keys precompute: bf16 context rows
    return probs[0].a_bf16 ? go_wd<bf16, EPI_SCATTER>(ps, nprob, st) : hipErrorInvalidValue;
  if (probs[0].a_bf16)
    return epi == EPI_TANH ? go_wd<bf16, EPI_TANH>(ps, nprob, st) : go_wd<bf16, EPI_STORE>(ps, nprob, st);
  return epi == EPI_TANH ? go_wd<float, EPI_TANH>(ps, nprob, st) : go_wd<float, EPI_STORE>(ps, nprob, st);
}

}  // namespace mt
