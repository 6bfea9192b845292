// Translation bookkeeping after a beam selection (batched beam search decoding to an n-best
// list as large as the beam): finished hypotheses on EOS, beam shrink, compaction of the
// surviving hypotheses into the leading slots, and the per-step record for backtracking; at
// the end, the n-best lists ranked and backtracked from those records.
// One 64-lane wave per sentence; lane r holds ranked result r (K <= 16).  Every lane loads its
// result before any lane stores, so the permutation can be done in place.
#include "mt_internal.h"

namespace mt {

__global__ __launch_bounds__(64) void beam_finish_kernel(BeamFinish a) {
  const int b = blockIdx.x, r = threadIdx.x, K = a.K;
  const int m = b * K + r;
  const int beam = a.beam[b];
  const int fbase = a.fin_count[b];
  int tk = 0, pv = 0, rw = 0;
  float sc = -INFINITY;
  if (r < K) {
    tk = a.tok[m];
    pv = a.bp[m];
    rw = a.row[m];
    sc = a.score[m];
  }
  // a hypothesis: within the sentence's beam and with a finite score
  const bool hyp = r < K && r < beam && sc > -INFINITY && sc < INFINITY;
  const bool fin = hyp && (a.final || tk == a.eos);
  const bool keep = hyp && !fin;
  const unsigned long long bf = __ballot(fin), bk = __ballot(keep);
  const unsigned long long lt = (1ull << r) - 1ull;
  const int nfin = __popcll(bf), nkeep = __popcll(bk);
  __builtin_amdgcn_s_waitcnt(0);  // the loads above have completed before the stores below
  if (fin) {
    const int j = fbase + __popcll(bf & lt);
    if (j < K) {
      const int f = b * K + j;
      a.fin_score[f] = sc;
      a.fin_norm[f] = sc / powf((float)(a.step + 1), a.alpha);
      a.fin_step[f] = a.step;
      a.fin_parent[f] = pv;
      a.fin_tok[f] = tk;
    }
  }
  if (keep) {
    const int d = b * K + __popcll(bk & lt);
    a.tok[d] = tk;
    a.bp[d] = pv;
    a.row[d] = rw;
    a.score[d] = sc;
    a.hist_tok[d] = tk;
    a.hist_bp[d] = pv;
  }
  if (r < K && r >= nkeep) {  // dead slot: never extends, reads a valid state row
    a.tok[m] = a.eos;
    a.bp[m] = 0;
    a.row[m] = b * K;
    a.score[m] = -INFINITY;
    a.hist_tok[m] = a.eos;
    a.hist_bp[m] = 0;
  }
  if (r == 0) {
    a.beam[b] = beam - nfin;
    a.fin_count[b] = fbase + nfin;
  }
}

// n-best lists from the records: one 64-lane wave per sentence.  Lane e < fin_count[b] holds
// finished entry e, counts the entries that rank before it (larger normalised score, or an
// equal one at a smaller index: the counts are a permutation), writes its index at its rank,
// and walks its hypothesis back through the per-step records (token and backpointer of the
// parent at each earlier step, one dependent round of loads per step) into the sequence row
// of its rank.  Unused ranks get order -1 and a row of -1.
__global__ __launch_bounds__(64) void beam_nbest_kernel(BeamNbest a) {
  const int b = blockIdx.x, e = threadIdx.x, K = a.K;
  const int base = b * K;
  const int fc = min(a.fin_count[b], K);
  const bool mine = e < fc;
  const float nv = mine ? a.fin_norm[base + e] : -INFINITY;
  int rank = 0;
  for (int o = 0; o < fc; ++o) {
    const float ov = __shfl(nv, o, 64);
    rank += (ov > nv || (ov == nv && o < e)) ? 1 : 0;
  }
  if (mine) {
    a.order[base + rank] = e;
    int32_t *row = a.seq + (size_t)(base + rank) * a.ld_seq;
    const int last = max(0, min(a.fin_step[base + e], a.steps - 1));
    row[last] = a.fin_tok[base + e];
    int p = a.fin_parent[base + e];
    for (int s = last - 1; s >= 0; --s) {
      const int m = base + min(max(p, 0), K - 1);
      const size_t o = (size_t)s * a.ld_hist + m;
      row[s] = a.hist_tok[o];
      p = a.hist_bp[o];
    }
    for (int s = last + 1; s < a.ld_seq; ++s) row[s] = -1;
  } else if (e < K) {
    a.order[base + e] = -1;
    int32_t *row = a.seq + (size_t)(base + e) * a.ld_seq;
    for (int s = 0; s < a.ld_seq; ++s) row[s] = -1;
  }
}

hipError_t launch_beam_nbest(const BeamNbest &a, int B, hipStream_t st) {
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(beam_nbest_kernel, dim3(B), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_beam_finish(const BeamFinish &a, int B, hipStream_t st) {
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(beam_finish_kernel, dim3(B), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace mt
