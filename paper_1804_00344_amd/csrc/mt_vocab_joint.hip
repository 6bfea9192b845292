// Output layer of a fused ensemble step: one pass over the vocabulary for all members
// (ensembling inside batched beam search, Section 2.3).
//
// The combined log-probability of entry v is sum_m w_m logit_m(v) - C with C = sum_m w_m LSE_m
// a per-row constant, so the beam needs, per row, every member's log-sum-exp and the
// combined value sum_m w_m logit_m(v) of its best entries; nothing of size [rows][V] has to
// exist.  A workgroup keeps the readout activations of every member resident in LDS and at
// each k-step runs the MFMAs of every member on the same vocabulary tile (the members' packed
// weights share one layout, so one fragment offset serves all of them).  The tile epilogue
// folds each member's logits into that member's log-sum-exp partials, forms the combined
// value, and collects it when it reaches the row's threshold, taken on the combined values
// of the first vocabulary entries.  Layouts, runs, candidate lists and partials are those of
// the single-model kernel; the k-loop reads the weights with buffer loads.
#include "mt_vocab_common.h"

#include <type_traits>

namespace mt {

struct VocabJointArgs {
  const void *t[kJointMax];     // [M][E] readout activations of member m (CT)
  const void *wp[kJointMax];    // packed Wo^T of member m
  const float *bias[kJointMax];  // [Vpad] output bias of member m, -inf beyond V
  float w[kJointMax];           // member weights
  float2 *part[kJointMax];      // [M][n_chunks] log-sum-exp partials of member m
  int M, V, E, KS, n_chunks, tiles_total;
  const float *thr;  // [M] threshold on the combined value
  int2 *cbuf;        // [M][cap][n_chunks][kLists] (combined value bits, token)
  int *ccnt;         // [M][n_chunks][kLists]
  int cap;
};

template <typename CT, int HB, int D, bool FIX, int NM>
__global__ __launch_bounds__((VShape<CT, HB>::NT)) void vocab_joint_kernel(VocabJointArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr int HBB = VShape<CT, HB>::HBW;
  constexpr int kVT = VShape<CT, HB>::NT;
  constexpr int KV = VCfg<CT>::KV;
  constexpr int es = (int)sizeof(CT);
  const int rowb = a.E * es + 16;  // LDS row stride of the resident activations
  const int mbytes = HB * rowb;    // LDS bytes of one member's rows

  const int nhb = (a.M + HB - 1) / HB;
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int chunk = L / nhb, hb = L % nhb;
  if (chunk >= a.n_chunks) return;
  const int h0 = hb * HB;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int run = wave & 3;
  const int hc0 = (wave >> 2) * VShape<CT, HB>::WH;

  // ---- resident activations of every member: rows h0..h0+HB-1 (zero beyond M) ----
  {
    const int vpr = a.E * es / 16;
#pragma unroll
    for (int mm = 0; mm < NM; ++mm) {
      const char *src = (const char *)a.t[mm];
      for (int idx = tid; idx < HB * vpr; idx += kVT) {
        const int r = idx / vpr, c = idx % vpr;
        v4u val = {0u, 0u, 0u, 0u};
        if (h0 + r < a.M) val = *(const v4u *)(src + ((size_t)(h0 + r) * a.E) * es + c * 16);
        *(v4u *)(lds + mm * mbytes + r * rowb + c * 16) = val;
      }
    }
  }
  __syncthreads();

  // ---- this wave's run of vocabulary tiles (as in the single-model kernel) ----
  const int slots = a.n_chunks * 4;
  const int slot = chunk * 4 + run;
  const int nblk = (a.V + 31) / 32;
  const int b_begin = (int)((long)nblk * slot / slots);
  const int b_end = (int)((long)nblk * (slot + 1) / slots);
  const int npair = (b_end - b_begin) >> 1;
  const int ntile = npair + ((b_end - b_begin) & 1);
  const int KS = a.KS;
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int src = run * 2 + lhalf;

  float lm[NM][HBB], ls[NM][HBB], th[HBB];
  const int nlr = a.n_chunks * kLists;
  const uint32_t lstep = (uint32_t)nlr * 8u;
  uint32_t loff[HBB], lend[HBB];
  char *const cbase = (char *)a.cbuf;
#pragma unroll
  for (int j = 0; j < HBB; ++j) {
    const int h = h0 + hc0 + j * 32 + lrow;
#pragma unroll
    for (int mm = 0; mm < NM; ++mm) {
      lm[mm][j] = FIX ? 0.f : -INFINITY;
      ls[mm][j] = 0.f;
    }
    th[j] = h < a.M ? a.thr[h] : __builtin_nanf("");  // rows past M: no value passes a NaN
    loff[j] = (uint32_t)(((size_t)(h < a.M ? h : 0) * a.cap * nlr + chunk * kLists + src) * sizeof(int2));
    lend[j] = loff[j] + (uint32_t)(a.cap - 1) * lstep;
  }

  if (ntile > 0) {
    const int kb = KS * 1024;  // bytes of one 32-row block's fragments
    __amdgpu_buffer_rsrc_t wrs[NM];
#pragma unroll
    for (int mm = 0; mm < NM; ++mm)
      wrs[mm] = __builtin_amdgcn_make_buffer_rsrc((void *)a.wp[mm], 0, a.tiles_total * kVRows * a.E * es, 0x00020000);
    const int wvo = lane * 16;
    // A tile's second fragment is the next 32-row block's; a single-block tile (the run's
    // last, when its block count is odd) reads its own block again, so no read leaves the run.
    v4u ring[D][NM][2];
    {
      const int tb0 = b_begin * kb, sec0 = 0 < npair ? kb : 0;
#pragma unroll
      for (int d = 0; d < D; ++d)
#pragma unroll
        for (int mm = 0; mm < NM; ++mm) {
          ring[d][mm][0] = __builtin_amdgcn_raw_buffer_load_b128(wrs[mm], wvo, tb0 + d * 1024, 0);
          ring[d][mm][1] = __builtin_amdgcn_raw_buffer_load_b128(wrs[mm], wvo, tb0 + d * 1024 + sec0, 0);
        }
    }
    // activation fragments: member mm, hypothesis block j, k-step ks; the next k-step's are
    // read before the current step's MFMAs (one wave per SIMD: nothing else covers the LDS
    // latency)
    const char *blb = lds + (hc0 + lrow) * rowb + lhalf * (KV / 2 * es);
    auto lds_frag = [&](int ks, v4u(&f)[NM][HBB]) {
#pragma unroll
      for (int mm = 0; mm < NM; ++mm)
#pragma unroll
        for (int j = 0; j < HBB; ++j) f[mm][j] = *(const v4u *)(blb + mm * mbytes + j * 32 * rowb + ks * (KV * es));
    };
    v4u bcur[NM][HBB], bnxt[NM][HBB];
    lds_frag(0, bcur);

    auto do_tile = [&](auto nbc, int ti) {
      constexpr int NB = decltype(nbc)::value;
      // the previous epilogue's candidate stores are a data-dependent count in the memory
      // counter: drain it once per tile so the ring waits in the k-loop stay exact
      __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
      f32x16 acc[NM][2][HBB];
#pragma unroll
      for (int mm = 0; mm < NM; ++mm)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < HBB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[mm][i][j][r] = 0.f;
      const int tb = (b_begin + 2 * ti) * kb;
      const int tnx = ti + 1 < ntile ? ti + 1 : ti;  // the last tile prefetches itself again
      const int tn = (b_begin + 2 * tnx) * kb;
      const int sec_cur = ti < npair ? kb : 0, sec_nxt = tnx < npair ? kb : 0;
      for (int ks0 = 0; ks0 < KS; ks0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
          const int ks = ks0 + d;
          lds_frag(ks + 1 < KS ? ks + 1 : 0, bnxt);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int mm = 0; mm < NM; ++mm) {
            const v4u c0 = ring[d][mm][0], c1 = ring[d][mm][1];
            if constexpr (es == 2) {
              bf16x8 a0, a1;
              __builtin_memcpy(&a0, &c0, 16);
              __builtin_memcpy(&a1, &c1, 16);
#pragma unroll
              for (int j = 0; j < HBB; ++j) {
                bf16x8 b;
                __builtin_memcpy(&b, &bcur[mm][j], 16);
                acc[mm][0][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b, acc[mm][0][j], 0, 0, 0);
                if constexpr (NB == 2) acc[mm][1][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b, acc[mm][1][j], 0, 0, 0);
              }
            } else {
              float fa0[4], fa1[4], fb[HBB][4];
              __builtin_memcpy(fa0, &c0, 16);
              __builtin_memcpy(fa1, &c1, 16);
#pragma unroll
              for (int j = 0; j < HBB; ++j) __builtin_memcpy(fb[j], &bcur[mm][j], 16);
#pragma unroll
              for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int j = 0; j < HBB; ++j) {
                  acc[mm][0][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa0[s], fb[j][s], acc[mm][0][j], 0, 0, 0);
                  if constexpr (NB == 2)
                    acc[mm][1][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa1[s], fb[j][s], acc[mm][1][j], 0, 0, 0);
                }
            }
          }
          // refill this slot with k-step ks + D (the next tile's first k-steps past the end)
          const bool same = ks + D < KS;
          const int so = same ? tb + (ks + D) * 1024 : tn + (ks + D - KS) * 1024;
          const int so2 = so + (same ? sec_cur : sec_nxt);
#pragma unroll
          for (int mm = 0; mm < NM; ++mm) {
            ring[d][mm][0] = __builtin_amdgcn_raw_buffer_load_b128(wrs[mm], wvo, so, 0);
            ring[d][mm][1] = __builtin_amdgcn_raw_buffer_load_b128(wrs[mm], wvo, so2, 0);
          }
#pragma unroll
          for (int mm = 0; mm < NM; ++mm)
#pragma unroll
            for (int j = 0; j < HBB; ++j) bcur[mm][j] = bnxt[mm][j];
          __builtin_amdgcn_sched_barrier(0);
        }
      }

      // ---- epilogue: biases, member log-sum-exp partials, combined-value candidates ----
      // lane holds rows v = v0 + 32*i + 8*(r/4) + 4*lhalf + r%4 of hypothesis column j*32 + lrow
      const int v0 = (b_begin + 2 * ti) * 32;
#pragma unroll
      for (int mm = 0; mm < NM; ++mm)
#pragma unroll
        for (int i = 0; i < NB; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float4 b4 = *(const float4 *)(a.bias[mm] + v0 + 32 * i + 8 * q + 4 * lhalf);
#pragma unroll
            for (int j = 0; j < HBB; ++j) {
              acc[mm][i][j][4 * q + 0] += b4.x; acc[mm][i][j][4 * q + 1] += b4.y;
              acc[mm][i][j][4 * q + 2] += b4.z; acc[mm][i][j][4 * q + 3] += b4.w;
            }
          }
      const int vlim = a.V - v0;  // entries at or past V are padding: never candidates
#pragma unroll
      for (int j = 0; j < HBB; ++j) {
#pragma unroll
        for (int mm = 0; mm < NM; ++mm) {
          if constexpr (FIX) {
            float se = 0.f;
#pragma unroll
            for (int i = 0; i < NB; ++i)
#pragma unroll
              for (int r = 0; r < 16; ++r) se += __builtin_amdgcn_exp2f(acc[mm][i][j][r] * kLog2e);
            ls[mm][j] += se;
          } else {
            float mt = -INFINITY;
#pragma unroll
            for (int i = 0; i < NB; ++i)
#pragma unroll
              for (int r = 0; r < 16; ++r) mt = fmaxf(mt, acc[mm][i][j][r]);
            if (mt != -INFINITY) {  // -inf only when the whole tile is padding
              const float mts = mt * kLog2e;
              float se = 0.f;
#pragma unroll
              for (int i = 0; i < NB; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r) se += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[mm][i][j][r], kLog2e, -mts));
              const float mn = fmaxf(lm[mm][j], mt);
              ls[mm][j] = ls[mm][j] * exp_fast(lm[mm][j] - mn) + se * exp_fast(mt - mn);
              lm[mm][j] = mn;
            }
          }
        }
#pragma unroll
        for (int i = 0; i < NB; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            float c = a.w[0] * acc[0][i][j][r];
#pragma unroll
            for (int mm = 1; mm < NM; ++mm) c += a.w[mm] * acc[mm][i][j][r];
            const int vo = 32 * i + 8 * (r >> 2) + 4 * lhalf + (r & 3);
            if (c >= th[j] && vo < vlim) {
              *(int2 *)(cbase + loff[j]) = make_int2(__float_as_int(c), v0 + vo);
              const uint32_t nx = loff[j] + lstep;
              loff[j] = nx < lend[j] ? nx : lend[j];
            }
          }
      }
    };
    for (int ti = 0; ti < npair; ++ti) do_tile(std::integral_constant<int, 2>{}, ti);
    if (ntile > npair) do_tile(std::integral_constant<int, 1>{}, npair);
  }  // ntile > 0

  // ---- candidate counts, then each member's 8 log-sum-exp partials per row merged via LDS ----
#pragma unroll
  for (int j = 0; j < HBB; ++j) {
    const int h = h0 + hc0 + j * 32 + lrow;
    if (h < a.M) {
      const uint32_t lstart = lend[j] - (uint32_t)(a.cap - 1) * lstep;
      const int n = (int)((loff[j] - lstart) / lstep);
      a.ccnt[((size_t)h * a.n_chunks + chunk) * kLists + src] = n >= a.cap - 1 ? a.cap + 1 : n;
    }
  }
  __syncthreads();  // the resident activations are no longer read
  float2 *lp = (float2 *)lds;  // [HB][kLists]
#pragma unroll
  for (int mm = 0; mm < NM; ++mm) {
#pragma unroll
    for (int j = 0; j < HBB; ++j) lp[(hc0 + j * 32 + lrow) * kLists + src] = make_float2(lm[mm][j], ls[mm][j]);
    __syncthreads();
    for (int hl = tid; hl < HB; hl += kVT) {
      const int h = h0 + hl;
      if (h >= a.M) continue;
      float m = -INFINITY;
      for (int s = 0; s < kLists; ++s) m = fmaxf(m, lp[hl * kLists + s].x);
      float sum = 0.f;
      if (m != -INFINITY)
        for (int s = 0; s < kLists; ++s) {
          const float2 q = lp[hl * kLists + s];
          if (q.x != -INFINITY) sum += q.y * exp_fast(q.x - m);
        }
      a.part[mm][(size_t)h * a.n_chunks + chunk] = make_float2(m, sum);
    }
    __syncthreads();
  }
}

// Threshold on the combined values of the first S vocabulary entries: x = sum_m w_m
// sample_m[v]; the K-th largest of the 64 lane maxima minus the rounding margin, as for a
// single model.  Block 0 also clears the B sentence arrival counters.
template <int R>
__global__ __launch_bounds__(256) void vocab_joint_threshold_kernel(int M, int S, int K, VocabJointSample smp,
                                                                    float *__restrict__ thr, int *scnt, int B) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (blockIdx.x == 0)
    for (int i = threadIdx.x; i < B; i += 256) __hip_atomic_store(scnt + i, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int m = blockIdx.x * 4 + w;
  if (m >= M) return;  // uniform per wave
  uint32_t um[1] = {0u};
#pragma unroll
  for (int s = 0; s < R; ++s) {
    const int v = s * 64 + lane;
    if (v < S) {
      float x = smp.w[0] * smp.sample[0][(size_t)m * smp.ld + v];
      for (int mm = 1; mm < smp.n; ++mm) x += smp.w[mm] * smp.sample[mm][(size_t)m * smp.ld + v];
      const uint32_t c = key_code(x);
      um[0] = c > um[0] ? c : um[0];
    }
  }
  float kth = -INFINITY;
  if (wave_count_ge<1>(um, 1, 1u) >= K) kth = key_from_code(wave_kth_code<1>(um, 1, K));
  if (lane == 0) thr[m] = kth - 1e-3f * (1.0f + fabsf(kth));
}

// ---------------------------------------------------------------------------------------

int vocab_joint_rows(int bf16_mma, int E, int n) {
  if (n < 2 || n > kJointMax) return 0;
  const int es = bf16_mma ? 2 : 4;
  const int KV = bf16_mma ? 16 : 8;
  if (E % (4 * KV) != 0) return 0;  // the ring is 4 k-steps deep and the k-loop steps by 4
  // 64 rows per workgroup only for two members (more would spill the accumulators)
  for (int hb = n == 2 ? 64 : 32; hb >= 32; hb /= 2)
    if ((size_t)n * hb * (E * es + 16) <= 160 * 1024 - 1024) return hb;
  return 0;
}

int vocab_joint_chunks(int bf16_mma, int M, int V, int E, int n, int num_cu) {
  const int HB = vocab_joint_rows(bf16_mma, E, n);
  if (HB == 0) return 0;
  const int nhb = (M + HB - 1) / HB;
  const int tiles = (V + kVRows - 1) / kVRows;
  int c = num_cu / nhb;
  if (c < 1) c = 1;
  if (c * 4 > tiles) c = (tiles + 3) / 4;
  return c;
}

template <typename CT, int HB, bool FIX, int NM>
static hipError_t vjgo(const VocabJointArgs &a, hipStream_t st) {
  constexpr int D = NM <= 3 ? 4 : 2;  // ring depth in k-steps (four members: registers)
  const int nhb = (a.M + HB - 1) / HB;
  const size_t tbytes = (size_t)NM * HB * (a.E * sizeof(CT) + 16);
  const size_t lbytes = (size_t)HB * kLists * 8;
  const size_t lds = tbytes > lbytes ? tbytes : lbytes;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void *)vocab_joint_kernel<CT, HB, D, FIX, NM>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((vocab_joint_kernel<CT, HB, D, FIX, NM>), dim3(nhb * a.n_chunks), dim3(VShape<CT, HB>::NT), lds,
                     st, a);
  return hipGetLastError();
}

template <typename CT, bool FIX>
static hipError_t vjgo_n(int n, int HB, const VocabJointArgs &a, hipStream_t st) {
  switch (n) {
    case 2: return HB == 64 ? vjgo<CT, 64, FIX, 2>(a, st) : vjgo<CT, 32, FIX, 2>(a, st);
    case 3: return vjgo<CT, 32, FIX, 3>(a, st);
    default: return vjgo<CT, 32, FIX, 4>(a, st);
  }
}

template <typename CT>
static hipError_t vjgo_ct(int n, int HB, bool fix, const VocabJointArgs &a, hipStream_t st) {
  return fix ? vjgo_n<CT, true>(n, HB, a, st) : vjgo_n<CT, false>(n, HB, a, st);
}

hipError_t launch_vocab_joint(const VocabJoint &j, hipStream_t st) {
  if (j.M == 0) return hipSuccess;
  const int HB = vocab_joint_rows(j.bf16_mma, j.E, j.n);
  if (HB == 0) return hipErrorInvalidValue;
  VocabJointArgs a{};
  for (int m = 0; m < j.n; ++m) {
    a.t[m] = j.t[m];
    a.wp[m] = j.wp[m];
    a.bias[m] = j.bias[m];
    a.w[m] = j.w[m];
    a.part[m] = j.part[m];
  }
  a.M = j.M;
  a.V = j.V;
  a.E = j.E;
  a.KS = j.E / (j.bf16_mma ? 16 : 8);
  a.n_chunks = j.n_chunks;
  a.tiles_total = (j.V + kVRows - 1) / kVRows;
  a.thr = j.thr;
  a.cbuf = j.cbuf;
  a.ccnt = j.ccnt;
  a.cap = j.cap;
  return j.bf16_mma ? vjgo_ct<bf16>(j.n, HB, j.fixed_ref, a, st) : vjgo_ct<float>(j.n, HB, j.fixed_ref, a, st);
}

hipError_t launch_vocab_joint_threshold(int M, int V, int K, const VocabJointSample &smp, float *thr, int *scnt,
                                        int B, hipStream_t st) {
  if (M == 0) return hipSuccess;
  const int S = vocab_sample_size(V);
  const int Sv = V < S ? V : S;  // entries >= V of the sample are padding
  hipLaunchKernelGGL((vocab_joint_threshold_kernel<kSampleMax / 64>), dim3((M + 3) / 4), dim3(256), 0, st, M, Sv, K,
                     smp, thr, scnt, B);
  return hipGetLastError();
}

}  // namespace mt
