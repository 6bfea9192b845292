// Output layer of the decoder step: logits = t Wo + bo over the whole target vocabulary,
// fused with the log-sum-exp partials of the log-softmax and the candidate collection of the
// beam top-K.  Logits are never written unless requested.
//
// Orientation: the product is computed transposed, logits^T = Wo^T t^T, so the MFMA's A
// operand is the weight (vocabulary rows) and its B operand the readout activations
// (hypothesis columns).  In the 32x32 MFMA output layout a lane owns one hypothesis column
// of each 32-column block, so the per-hypothesis running state (online log-sum-exp, candidate
// count) lives in the lane's registers while the vocabulary streams past.
//
// Work split: a workgroup owns HB hypothesis rows (their activations stay resident in LDS for
// the whole kernel) and one contiguous chunk of the vocabulary, split into 4 runs of 64-row
// vocabulary tiles (cut at 32-row boundaries, so a run may end with one 32-row tile).  Each wave covers WH <= 64 hypothesis columns of one run (HB/WH waves per
// run share its weight fragments) and streams the packed weights straight from global memory
// (fragment order, one coalesced 16-byte load per lane per MFMA operand), prefetching D
// k-steps ahead across tile boundaries, with no barrier in the main loop.
//
// Beam candidates without sorting: a row's K best logits are all >= the K-th best logit of
// any subset of that row.  A small first pass computes the logits of the first S vocabulary
// entries and takes their K-th best (minus a rounding margin) as the row's threshold; the main
// pass appends every logit at or above it to a per-lane buffer (one compare per logit, a
// store when it passes).  The row selection then takes the K best keys among the collected
// values; a row whose buffers overflowed is recomputed in full, so the result is exact.
//
// Packed weights (built at load time): for 32-row vocabulary block vb and k-step ks of KV
// k-values, 64 lanes x 16 bytes at ((vb * KS + ks) * 64 + lane) * 16, where lane l holds
// Wo^T[vb*32 + l%32][ks*KV + (l/32)*KV/2 + j], j < 16/sizeof(CT).  fp32 uses the 32x32x2
// MFMA with each 16-byte vector feeding 4 successive MFMAs (lane half g supplies k = 4g + s
// to MFMA s); bf16 uses 32x32x16 with one vector per MFMA.
#include "mt_vocab_common.h"

#include <type_traits>

namespace mt {

struct VocabArgs {
  const void *t;        // [M][E] activations in CT
  const void *wp;       // packed weights (see header comment)
  const float *bias;    // [Vpad] with -inf beyond V
  int M, V, E, KS;      // KS = E / KV
  int n_chunks;
  int tiles_total;      // 64-row tiles of the packed weights (the packed extent)
  float2 *part;         // [M][n_chunks] (max, sum exp(l - max)); NULL in the threshold pass
  const float *thr;     // [M] candidate threshold
  int2 *cbuf;           // [M][cap][n_chunks][kLists] (logit bits, token): entry-major per row
  int *ccnt;            // [M][n_chunks][kLists] values at or above the threshold
  int cap;
  float *logits;        // [M][logits_ld] or NULL
  int logits_ld;
  int logits_vec;       // 16-byte aligned rows (base aligned, logits_ld % 4 == 0): float4 stores
  float logits_w;       // the logits are stored multiplied by this weight (1: as they are)
  int logits_acc;       // 1: added to the values already stored (ensemble members after the first)
  int cap_stored;       // 1: candidates are the stored (weighted, accumulated) values, not the logits
                        // (a fused ensemble's last member: the combined values of all members)
  int fixed_ref;        // logits proven bounded: log-sum-exp without a running maximum
};

// FIX: the logits are bounded (|logit| <= 40, checked at load time), so the log-sum-exp is
// accumulated as sum exp(logit) directly: no tile maximum, no rescaling, and every partial
// carries the reference 0.
// LOG: the logits are also written (parity mode); a separate instance so that the timed
// path carries none of that path's registers.
// KSC > 0: the depth is the compile-time KSC k-steps (E = KSC * KV); each tile's k-loop is
// then unrolled and the weights are read with buffer loads at a scalar offset (tile base +
// constant), so a refill costs one scalar add instead of the flat-stream index update.
template <typename CT, int HB, int D, bool FIX, bool LOG, int KSC>
__global__ __launch_bounds__((VShape<CT, HB>::NT)) void vocab_kernel(VocabArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr int HBB = VShape<CT, HB>::HBW;
  constexpr int kVT = VShape<CT, HB>::NT;
  constexpr int KV = VCfg<CT>::KV;
  constexpr int es = (int)sizeof(CT);
  const int rowb = a.E * es + 16;  // LDS row stride of the resident activations

  const int nhb = (a.M + HB - 1) / HB;
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int chunk = L / nhb, hb = L % nhb;
  if (chunk >= a.n_chunks) return;
  const int h0 = hb * HB;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: keeps the stream scalar
  const int run = wave & 3;                                    // vocabulary run of this wave
  const int hc0 = (wave >> 2) * VShape<CT, HB>::WH;               // first hypothesis column of this wave

  // ---- resident activations: rows h0..h0+HB-1 (zero beyond M) ----
  {
    const int vecs_per_row = a.E * es / 16;
    for (int idx = tid; idx < HB * vecs_per_row; idx += kVT) {
      const int r = idx / vecs_per_row, c = idx % vecs_per_row;
      v4u val = {0u, 0u, 0u, 0u};
      if (h0 + r < a.M) val = *(const v4u *)((const char *)a.t + ((size_t)(h0 + r) * a.E) * es + c * 16);
      *(v4u *)(lds + r * rowb + c * 16) = val;
    }
  }
  __syncthreads();

  // ---- this wave's contiguous run of vocabulary tiles ----
  // Runs are cut at 32-row block boundaries (half a tile), which evens out the work of the
  // busiest wave: a run is a sequence of two-block tiles, then one single-block tile when its
  // block count is odd.
  const int slots = a.n_chunks * 4;
  const int slot = chunk * 4 + run;
  const int nblk = (a.V + 31) / 32;
  const int b_begin = (int)((long)nblk * slot / slots);
  const int b_end = (int)((long)nblk * (slot + 1) / slots);
  const int npair = (b_end - b_begin) >> 1;
  const int ntile = npair + ((b_end - b_begin) & 1);
  const int total = ntile * a.KS;  // flat (tile, k-step) stream, KS % D == 0
  const int KS = a.KS;
  const int lrow = lane & 31, lhalf = lane >> 5;
  const int src = run * 2 + lhalf;
  const bool collect = a.part != nullptr;

  float lm[HBB], ls[HBB], th[HBB];
  // A row's lists are stored entry-major (entry q of all its lists contiguous), so that the
  // selection reads the first entries of every list of a row with coalesced loads; successive
  // entries of one list are nlr * 8 bytes apart.
  const int nlr = a.n_chunks * kLists;
  const uint32_t lstep = (uint32_t)nlr * 8u;
  uint32_t loff[HBB];  // byte offset of this lane's next candidate slot in cbuf, per hypothesis block
  uint32_t lend[HBB];  // offset of the list's last slot (writes past capacity stay there)
  char *const cbase = (char *)a.cbuf;
#pragma unroll
  for (int j = 0; j < HBB; ++j) {
    const int h = h0 + hc0 + j * 32 + lrow;
    lm[j] = FIX ? 0.f : -INFINITY;
    ls[j] = 0.f;
    th[j] = (collect && a.thr && h < a.M) ? a.thr[h] : INFINITY;
    loff[j] = (uint32_t)(((size_t)(h < a.M ? h : 0) * a.cap * nlr + chunk * kLists + src) * sizeof(int2));
    lend[j] = loff[j] + (uint32_t)(a.cap - 1) * lstep;
  }

  // With two hypothesis groups (two waves per SIMD, same vocabulary tiles), both waves of a
  // SIMD would reach their VALU-heavy tile epilogues at the same moments and leave the
  // matrix core idle meanwhile.  Starting the second group about half a tile late puts one
  // wave's epilogue under the other's MFMAs.
  if (VShape<CT, HB>::NW > 4 && (wave >> 2) == 1) __builtin_amdgcn_s_sleep(32);

  if (ntile > 0) {
    // Weight fragments of step g of tile ti are vocabulary blocks b_begin+2*ti and +1 at
    // k-step ks, 1 KiB (64 lanes x 16 bytes) apart per k-step.  The ring is refilled right
    // after its slot is consumed, from a wave-uniform fragment index that advances without a
    // branch (clamped to the last step), so the loads stay in flight across k-steps: a
    // conditional refill would make the compiler wait for every outstanding load.
    const v4u *wb = (const v4u *)a.wp + (size_t)b_begin * KS * 64 + lane;
    int pf_k = 0, pf_n = 0, pf_t = 0;
    int poff = 0;  // fragment index of the next prefetch, in 1 KiB steps from wb
    auto fetch = [&](v4u(&slot)[2]) {
      slot[0] = wb[(size_t)poff * 64];
      // a single-block tile reads its one block twice (the next block may lie past the end)
      slot[1] = wb[(size_t)(poff + (pf_t < npair ? KS : 0)) * 64];
      const int more = pf_n + 1 < total ? 1 : 0;
      const int nk = pf_k + more;
      const int wrap = nk == KS ? 1 : 0;
      pf_n += more;
      pf_k = wrap ? 0 : nk;
      pf_t += wrap;
      poff += more + wrap * KS;
    };
    v4u ring[D][2];
    // buffer view of the packed weights (KSC > 0): fixed per-lane offset, scalar fragment
    // offsets.  A tile's second fragment is the next block's; a single-block tile reads its
    // own block again, so no read leaves the run.
    const __amdgpu_buffer_rsrc_t wrs =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.wp, 0, a.tiles_total * kVRows * a.E * es, 0x00020000);
    const int wvo = lane * 16;
    if constexpr (KSC > 0) {
      const int sec0 = 0 < npair ? KSC * 1024 : 0;
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int so = (b_begin * KSC + d) * 1024;
        ring[d][0] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo, so, 0);
        ring[d][1] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo, so + sec0, 0);
      }
    } else {
#pragma unroll
      for (int d = 0; d < D; ++d) fetch(ring[d]);
    }
    const v4u *bl = (const v4u *)lds + (size_t)(hc0 + lrow) * (rowb / 16) + lhalf * (KV / 2 * es / 16);

    // activation fragments of k-step ks (identical for every tile, so the sequence repeats
    // with period KS).  With one wave per SIMD (fp32) the fragments of the next k-step are
    // read before the current step's MFMAs so the LDS latency is not exposed; bf16 runs two
    // waves per SIMD, which cover it, and has no registers to spare for the second copy.
    constexpr bool kPrefetchLds = es == 4;
    auto lds_frag = [&](int ks, v4u(&f)[HBB]) {
#pragma unroll
      for (int j = 0; j < HBB; ++j) f[j] = bl[(size_t)j * 32 * (rowb / 16) + ks * (KV * es / 16)];
    };
    v4u bcur[HBB], bnxt[HBB];
    if constexpr (kPrefetchLds) lds_frag(0, bcur);

    // one tile of NB (2 or 1) 32-row blocks
    auto do_tile = [&](auto nbc, int ti) {
      constexpr int NB = decltype(nbc)::value;
      // Drain the memory counter once per tile (stores count in it too, and the previous
      // epilogue issued a data-dependent number of them; the ring loads have long arrived).
      // With nothing outstanding on entry, the compiler keeps exact, non-draining waits on
      // the ring inside the k-loop.
      __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
      f32x16 acc[2][HBB];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < HBB; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

      // one k-step: MFMAs on ring slot `slot`, then its refill (refill(slot) issues the loads)
      auto kstep = [&](int ks, v4u(&slot)[2], auto refill) {
        if constexpr (kPrefetchLds) {
          lds_frag(ks + 1 < KS ? ks + 1 : 0, bnxt);
          __builtin_amdgcn_sched_barrier(0);  // issue the reads before this step's MFMAs
        } else {
          lds_frag(ks, bcur);
        }
        const v4u c0 = slot[0], c1 = slot[1];
        if constexpr (es == 2) {
          bf16x8 a0, a1;
          __builtin_memcpy(&a0, &c0, 16);
          __builtin_memcpy(&a1, &c1, 16);
#pragma unroll
          for (int j = 0; j < HBB; ++j) {
            bf16x8 b;
            __builtin_memcpy(&b, &bcur[j], 16);
            acc[0][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b, acc[0][j], 0, 0, 0);
            if constexpr (NB == 2) acc[1][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b, acc[1][j], 0, 0, 0);
          }
        } else {
          float fa0[4], fa1[4], fb[HBB][4];
          __builtin_memcpy(fa0, &c0, 16);
          __builtin_memcpy(fa1, &c1, 16);
#pragma unroll
          for (int j = 0; j < HBB; ++j) __builtin_memcpy(fb[j], &bcur[j], 16);
#pragma unroll
          for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int j = 0; j < HBB; ++j) {
              acc[0][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa0[s], fb[j][s], acc[0][j], 0, 0, 0);
              if constexpr (NB == 2) acc[1][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa1[s], fb[j][s], acc[1][j], 0, 0, 0);
            }
        }
        refill(slot);
        if constexpr (kPrefetchLds) {
#pragma unroll
          for (int j = 0; j < HBB; ++j) bcur[j] = bnxt[j];
        }
        // keep each refill right behind the MFMAs that consumed its slot (left alone, the
        // scheduler sinks all refills to the end of the unrolled body, which shortens the
        // prefetch distance of the first slots to almost nothing)
        __builtin_amdgcn_sched_barrier(0);
      };
      if constexpr (KSC > 0) {
        // byte offsets of this tile's and the next tile's first fragment (the last tile
        // prefetches itself again) and of their second blocks
        const int tb = (b_begin + 2 * ti) * KSC * 1024;
        const int tnx = ti + 1 < ntile ? ti + 1 : ti;
        const int tn = (b_begin + 2 * tnx) * KSC * 1024;
        const int sec_cur = ti < npair ? KSC * 1024 : 0, sec_nxt = tnx < npair ? KSC * 1024 : 0;
#pragma unroll
        for (int ks = 0; ks < KSC; ++ks)
          kstep(ks, ring[ks % D], [&](v4u(&r)[2]) {
            const int so = ks + D < KSC ? tb + (ks + D) * 1024 : tn + (ks + D - KSC) * 1024;
            r[0] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo, so, 0);
            r[1] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo, so + (ks + D < KSC ? sec_cur : sec_nxt), 0);
          });
      } else {
        for (int ks0 = 0; ks0 < KS; ks0 += D) {
#pragma unroll
          for (int d = 0; d < D; ++d) kstep(ks0 + d, ring[d], fetch);
        }
      }

      // ---- epilogue of this tile: bias, online log-sum-exp, threshold-filtered candidates ----
      // lane holds rows v = v0 + 32*i + 8*(r/4) + 4*lhalf + r%4 of hypothesis column j*32 + lrow
      const int v0 = (b_begin + 2 * ti) * 32;
#pragma unroll
      for (int i = 0; i < NB; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 b4 = *(const float4 *)(a.bias + v0 + 32 * i + 8 * q + 4 * lhalf);
#pragma unroll
          for (int j = 0; j < HBB; ++j) {
            acc[i][j][4 * q + 0] += b4.x; acc[i][j][4 * q + 1] += b4.y;
            acc[i][j][4 * q + 2] += b4.z; acc[i][j][4 * q + 3] += b4.w;
          }
        }
#pragma unroll
      for (int j = 0; j < HBB; ++j) {
        const int h = h0 + hc0 + j * 32 + lrow;
        // candidate capture: store the (logit, token) pair at the lane's next slot and advance;
        // the offset sticks at the list's last slot, and a list that reaches it is reported as
        // overflowed (its row is recomputed exactly)
        auto capture = [&](float x, int i, int r) {
          *(int2 *)(cbase + loff[j]) = make_int2(__float_as_int(x), v0 + 32 * i + 8 * (r >> 2) + 4 * lhalf + (r & 3));
          const uint32_t nx = loff[j] + lstep;
          loff[j] = nx < lend[j] ? nx : lend[j];
        };
        if (collect) {
          if constexpr (FIX) {
            float se = 0.f;
#pragma unroll
            for (int i = 0; i < NB; ++i)
#pragma unroll
              for (int r = 0; r < 16; ++r) {
                const float x = acc[i][j][r];
                se += __builtin_amdgcn_exp2f(x * kLog2e);
                if (!(LOG && a.cap_stored) && x >= th[j]) capture(x, i, r);
              }
            ls[j] += se;
          } else {
            float mt = -INFINITY;
#pragma unroll
            for (int i = 0; i < NB; ++i)
#pragma unroll
              for (int r = 0; r < 16; ++r) mt = fmaxf(mt, acc[i][j][r]);
            if (mt != -INFINITY) {  // -inf only when the whole tile is padding
              const float mts = mt * kLog2e;
              float se = 0.f;
#pragma unroll
              for (int i = 0; i < NB; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                  const float x = acc[i][j][r];
                  se += __builtin_amdgcn_exp2f(__builtin_fmaf(x, kLog2e, -mts));
                  if (!(LOG && a.cap_stored) && x >= th[j]) capture(x, i, r);
                }
              const float mn = fmaxf(lm[j], mt);
              ls[j] = ls[j] * exp_fast(lm[j] - mn) + se * exp_fast(mt - mn);
              lm[j] = mn;
            }
          }
        }
        if (LOG && h < a.M) {
          // a lane's four consecutive entries v..v+3 go out as one 16-byte store where the
          // row layout allows it
          float *lrowp = a.logits + (size_t)h * a.logits_ld;
#pragma unroll
          for (int i = 0; i < NB; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int vb = v0 + 32 * i + 8 * q + 4 * lhalf;
              if (a.logits_vec && vb + 3 < a.V) {
                float4 val = make_float4(a.logits_w * acc[i][j][4 * q], a.logits_w * acc[i][j][4 * q + 1],
                                         a.logits_w * acc[i][j][4 * q + 2], a.logits_w * acc[i][j][4 * q + 3]);
                if (a.logits_acc) {
                  const float4 o = *(const float4 *)(lrowp + vb);
                  val.x += o.x; val.y += o.y; val.z += o.z; val.w += o.w;
                }
                if (a.cap_stored) {
                  if (val.x >= th[j]) capture(val.x, i, 4 * q + 0);
                  if (val.y >= th[j]) capture(val.y, i, 4 * q + 1);
                  if (val.z >= th[j]) capture(val.z, i, 4 * q + 2);
                  if (val.w >= th[j]) capture(val.w, i, 4 * q + 3);
                }
                *(float4 *)(lrowp + vb) = val;
              } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  if (vb + e < a.V && vb + e < a.logits_ld) {
                    float val = a.logits_w * acc[i][j][4 * q + e];
                    if (a.logits_acc) val += lrowp[vb + e];
                    if (a.cap_stored && val >= th[j]) capture(val, i, 4 * q + e);
                    lrowp[vb + e] = val;
                  }
              }
            }
        }
      }
    };
    for (int ti = 0; ti < npair; ++ti) do_tile(std::integral_constant<int, 2>{}, ti);
    if (ntile > npair) do_tile(std::integral_constant<int, 1>{}, npair);
  }  // ntile > 0

  if (!collect) return;
  // ---- candidate counts, and the 8 log-sum-exp partials of each hypothesis merged via LDS ----
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
  for (int j = 0; j < HBB; ++j) lp[(hc0 + j * 32 + lrow) * kLists + src] = make_float2(lm[j], ls[j]);
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
    a.part[(size_t)h * a.n_chunks + chunk] = make_float2(m, sum);
  }
}

// Threshold of each row: a value with at least K of the first S logits at or above it, lowered
// by a margin that covers the rounding difference between this pass's logits and the main
// pass's (the two sum the same products in different orders).  The row's K best are all at or
// above it, whatever the distribution of the logits.  Each lane takes the maximum of its S/64
// sampled logits and the threshold is the K-th largest of the 64 lane maxima (exact, by
// bisection over order-preserving codes): K different lanes reach it, so K sampled logits do.
// Against the K-th best of the whole sample it is lower only when two of the sample's best
// share a lane, at a small fraction of the cost.
// A fused ensemble's last member thresholds the combined values instead: cw * sample[m][v],
// plus comb[m][v] (the earlier members' weighted logits, row stride V) when there are any.
template <int R, bool COMB>
__global__ __launch_bounds__(256) void vocab_threshold_kernel(int M, int S, int K, const float *__restrict__ sample,
                                                              int ld, float *__restrict__ thr, int *scnt, int B,
                                                              const float *__restrict__ comb, int V, float cw) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (blockIdx.x == 0)
    for (int i = threadIdx.x; i < B; i += 256) __hip_atomic_store(scnt + i, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int m = blockIdx.x * 4 + w;
  if (m >= M) return;  // uniform per wave
  const float *row = sample + (size_t)m * ld;
  float x[R];
#pragma unroll
  for (int s = 0; s < R; ++s) {
    const int v = s * 64 + lane;
    if constexpr (COMB)
      x[s] = v < S ? cw * row[v] + (comb ? comb[(size_t)m * V + v] : 0.f) : -INFINITY;
    else
      x[s] = v < S ? row[v] : -INFINITY;
  }
  uint32_t um[1] = {0u};
#pragma unroll
  for (int s = 0; s < R; ++s) {
    const uint32_t c = key_code(x[s]);
    um[0] = c > um[0] ? c : um[0];
  }
  float kth = -INFINITY;
  if (wave_count_ge<1>(um, 1, 1u) >= K) kth = key_from_code(wave_kth_code<1>(um, 1, K));
  if (lane == 0) thr[m] = kth - 1e-3f * (1.0f + fabsf(kth));
}

// ---------------------------------------------------------------------------------------

int vocab_rows_per_block(int bf16_mma, int E) {
  const int es = bf16_mma ? 2 : 4;
  const int want = bf16_mma ? 128 : 64;
  for (int hb = want; hb >= 32; hb /= 2)
    if ((size_t)hb * (E * es + 16) <= 160 * 1024 - 1024) return hb;
  return 0;
}

size_t vocab_pack_bytes(int bf16_mma, int V, int E) {
  const int Vpad = (V + kVRows - 1) / kVRows * kVRows;
  return (size_t)Vpad * E * (bf16_mma ? 2 : 4);
}

int vocab_sample_size(int V) {
  const int s = V < kSampleMax ? V : kSampleMax;
  return (s + kVRows - 1) / kVRows * kVRows;
}

int vocab_lists() { return kLists; }

// packed[((vb * KS + ks) * 64 + lane) * 16 bytes] from Wo^T rows (row v = column v of Wo)
void vocab_pack_host(int bf16_mma, int V, int E, const float *src, int src_is_emb, void *out) {
  const int KV = bf16_mma ? 16 : 8, epv = bf16_mma ? 8 : 4;
  const int KS = E / KV;
  const int Vpad = (V + kVRows - 1) / kVRows * kVRows;
  for (int vb = 0; vb < Vpad / 32; ++vb)
    for (int ks = 0; ks < KS; ++ks)
      for (int l = 0; l < 64; ++l)
        for (int j = 0; j < epv; ++j) {
          const int v = vb * 32 + (l & 31);
          const int k = ks * KV + (l >> 5) * (KV / 2) + j;
          float x = 0.f;
          if (v < V) x = src_is_emb ? src[(size_t)v * E + k] : src[(size_t)k * V + v];
          const size_t o = (((size_t)vb * KS + ks) * 64 + l) * epv + j;
          if (bf16_mma) {
            ((uint16_t *)out)[o] = bf16_rne_bits(x);
          } else {
            ((float *)out)[o] = x;
          }
        }
}

// prefetch depth in k-steps: a bf16 k-step is 16x shorter in MFMA time than an fp32 one, so it
// needs a deeper ring to cover the same memory latency
static int ring_depth(int bf16_mma, int KS) {
  if (bf16_mma && KS % 8 == 0) return 8;
  return KS % 4 == 0 ? 4 : KS % 2 == 0 ? 2 : 1;
}

template <typename CT, int HB, int D, bool FIX, bool LOG, int KSC>
static hipError_t vgo(const VocabArgs &a, hipStream_t st) {
  const int nhb = (a.M + HB - 1) / HB;
  const size_t tbytes = (size_t)HB * (a.E * sizeof(CT) + 16);
  const size_t lbytes = (size_t)HB * kLists * 8;
  const size_t lds = tbytes > lbytes ? tbytes : lbytes;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void *)vocab_kernel<CT, HB, D, FIX, LOG, KSC>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((vocab_kernel<CT, HB, D, FIX, LOG, KSC>), dim3(nhb * a.n_chunks), dim3(VShape<CT, HB>::NT), lds,
                     st, a);
  return hipGetLastError();
}

template <typename CT, int HB, int D, int KSC>
static hipError_t vgo_k(const VocabArgs &a, hipStream_t st) {
  if (a.logits) return a.fixed_ref ? vgo<CT, HB, D, true, true, KSC>(a, st) : vgo<CT, HB, D, false, true, KSC>(a, st);
  return a.fixed_ref ? vgo<CT, HB, D, true, false, KSC>(a, st) : vgo<CT, HB, D, false, false, KSC>(a, st);
}

// E = 512 (bf16: 32 k-steps, fp32: 64) takes the unrolled form
template <typename CT, int HB, int D>
static hipError_t vgo_f(const VocabArgs &a, hipStream_t st) {
  if (sizeof(CT) == 2 && a.KS == 32 && 32 % D == 0) return vgo_k<CT, HB, D, 32>(a, st);
  if (sizeof(CT) == 4 && a.KS == 64 && 64 % D == 0) return vgo_k<CT, HB, D, 64>(a, st);
  return vgo_k<CT, HB, D, 0>(a, st);
}

template <typename CT, int HB>
static hipError_t vgo_d(const VocabArgs &a, hipStream_t st) {
  switch (ring_depth(sizeof(CT) == 2, a.KS)) {
    case 8: return vgo_f<CT, HB, 8>(a, st);
    case 4: return vgo_f<CT, HB, 4>(a, st);
    case 2: return vgo_f<CT, HB, 2>(a, st);
    default: return vgo_f<CT, HB, 1>(a, st);
  }
}

static hipError_t vgo_any(int bf16_mma, const VocabArgs &a, hipStream_t st) {
  const int HB = vocab_rows_per_block(bf16_mma, a.E);
  if (bf16_mma) {
    if (HB == 128) return vgo_d<bf16, 128>(a, st);
    if (HB == 64) return vgo_d<bf16, 64>(a, st);
    return vgo_d<bf16, 32>(a, st);
  }
  if (HB == 64) return vgo_d<float, 64>(a, st);
  return vgo_d<float, 32>(a, st);
}

int vocab_chunks(int bf16_mma, int M, int V, int E, int num_cu) {
  const int HB = vocab_rows_per_block(bf16_mma, E);
  const int nhb = (M + HB - 1) / HB;
  const int tiles = (V + kVRows - 1) / kVRows;
  int n = num_cu / nhb;
  if (n < 1) n = 1;
  if (n * 4 > tiles) n = (tiles + 3) / 4;
  return n;
}

static VocabArgs base_args(int bf16_mma, const void *t, const void *wp, const float *bias_pad, int M, int V,
                           int E) {
  VocabArgs a{};
  a.t = t;
  a.wp = wp;
  a.bias = bias_pad;
  a.M = M;
  a.V = V;
  a.E = E;
  a.KS = E / (bf16_mma ? 16 : 8);
  return a;
}

hipError_t launch_vocab_threshold(int M, int V, int K, const float *sample, float *thr, int *scnt, int B,
                                  hipStream_t st, const float *comb, float w) {
  if (M == 0) return hipSuccess;
  const int S = vocab_sample_size(V);
  const int Sv = V < S ? V : S;  // entries >= V of the sample are padding
  // a fused ensemble's last member (weight w, earlier members' values comb) takes the combined
  // form; a single model's the plain one
  if (comb || w != 1.f)
    hipLaunchKernelGGL((vocab_threshold_kernel<kSampleMax / 64, true>), dim3((M + 3) / 4), dim3(256), 0, st, M, Sv,
                       K, sample, S, thr, scnt, B, comb, V, w);
  else
    hipLaunchKernelGGL((vocab_threshold_kernel<kSampleMax / 64, false>), dim3((M + 3) / 4), dim3(256), 0, st, M, Sv,
                       K, sample, S, thr, scnt, B, comb, V, w);
  return hipGetLastError();
}

hipError_t launch_vocab(int bf16_mma, const void *t, const void *wp, const float *bias_pad, int M, int V,
                        int E, int n_chunks, const float *thr, float2 *part, int2 *cbuf, int *ccnt, int cap,
                        float *logits, int fixed_ref, hipStream_t st, float logits_w, int logits_acc,
                        int cap_stored) {
  if (M == 0) return hipSuccess;
  VocabArgs a = base_args(bf16_mma, t, wp, bias_pad, M, V, E);
  a.tiles_total = (V + kVRows - 1) / kVRows;
  a.n_chunks = n_chunks;
  a.part = part;
  a.thr = thr;
  a.cbuf = cbuf;
  a.ccnt = ccnt;
  a.cap = cap;
  a.logits = logits;
  a.logits_ld = V;
  a.logits_vec = logits && ((uintptr_t)logits & 15) == 0 && V % 4 == 0;
  a.logits_w = logits_w;
  a.logits_acc = logits_acc;
  a.cap_stored = logits && cap_stored;
  a.fixed_ref = fixed_ref;
  return vgo_any(bf16_mma, a, st);
}

}  // namespace mt
