/*
 * mtref — CPU oracle for one beam-search step of a shallow attentional
 * cGRU decoder (Marian, arXiv 1804.00344: the Nematus-compatible shallow
 * model of Section 1 and Section 2.1; the encoder/decoder interface of
 * Section 2.2; batched beam search of Section 2.3).
 *
 * TEST INFRASTRUCTURE ONLY.  This code exists to check the GPU library.
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load it.  It shares no code, header, table or helper with the GPU path.
 *
 * Conventions: row-major, "x W" with W stored [in x out]; C = 2H.
 * Storage is fp32; every dot product, sum, max and transcendental is
 * evaluated in double and rounded to fp32 at stage boundaries (P, s0, s1,
 * q, alpha, c, s, t, logp).  Single-threaded, no BLAS, no fast-math.
 */
#ifndef MTREF_H
#define MTREF_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t E, H, A, V;   /* embedding, state, attention, vocabulary; C = 2H */
  int32_t layer_norm;   /* 1: LN on every gate block of both paths and the readout */
  int32_t tied_output;  /* 1: output matrix is emb transposed */
  double ln_eps;
  int32_t transitions;  /* recurrent-only GRU blocks after GRU 2 (deep transition); 0: shallow */
} mtref_dims;

typedef struct {
  const float *emb;                 /* [V,E] */
  const float *W1, *U1, *b1;        /* [E,3H], [H,3H], [3H]; gate blocks r,z,h */
  const float *Ua, *ba, *Wa, *va;   /* [C,A], [A], [H,A], [A] */
  const float *W2, *U2, *b2;        /* [C,3H], [H,3H], [3H] */
  const float *Wt_s, *Wt_y, *Wt_c, *bt; /* [H,E], [E,E], [C,E], [E] */
  const float *Wo, *bo;             /* [E,V], [V] */
  const float *Wi, *bi;             /* [C,H], [H] */
  /* layer norm (only read if layer_norm): gain/shift per path, [3H] each; readout [E] */
  const float *g1a, *be1a, *g1u, *be1u, *g2a, *be2a, *g2u, *be2u, *gt, *bet;
  /* transition blocks j < transitions, stacked: Ut [T][H,3H], btr [T][3H]; layer norm of
   * their recurrent products (only read if layer_norm): gtu, betu [T][3H] */
  const float *Ut, *btr, *gtu, *betu;
  /* second source (dual-source models): Ua2 [C,A], ba2 [A], Wa2 [H,A], va2 [A]; W2 and
   * Wt_c then have 2C rows (the two contexts side by side) */
  const float *Ua2, *ba2, *Wa2, *va2;
} mtref_weights;

/* status: 0 ok, -1 bad argument, -2 index out of range */

/* ---- stage functions (double in / double out) ---------------------------------- */

/* y = gamma * (x - mean) / sqrt(var + eps) + beta over n features; biased variance. */
void mtref_layer_norm(int n, const double *x, const float *gamma, const float *beta,
                      double eps, double *y);

/* One GRU block with reset-after-matmul:
 *   a = x W + b, u = h U, (optionally LN on each H-block of a and of u),
 *   r = sig(a_r + u_r), z = sig(a_z + u_z), hh = tanh(a_h + r * u_h),
 *   out = (1 - z) * hh + z * h.
 * ln_* may be NULL when no layer norm is applied. */
void mtref_gru(int in_dim, int H, const double *x, const double *h,
               const float *W, const float *U, const float *b,
               const float *ln_ga, const float *ln_ba, const float *ln_gu, const float *ln_bu,
               double eps, double *out);

/* One transition block of a deep-transition decoder cell: a GRU block with no
 * external input, so its input path is the bias alone:
 *   u = h U, (optionally LN on each H-block of u),
 *   r = sig(b_r + u_r), z = sig(b_z + u_z), hh = tanh(b_h + r * u_h),
 *   out = (1 - z) * hh + z * h. */
void mtref_gru_transition(int H, const double *h, const float *U, const float *b,
                          const float *ln_gu, const float *ln_bu, double eps, double *out);

/* Additive attention over S positions of one sentence for one query q[A]:
 *   e_i = sum_a va[a] tanh(P[i,a] + q[a]) for valid i (mask[i] != 0),
 *   alpha = softmax over valid positions (0 exactly elsewhere),
 *   ctx = sum_i alpha_i Cx[i,:].
 * Padded positions of P and Cx are never read.  With no valid position,
 * alpha and ctx are all zero. */
void mtref_attention(int S, int A, int Cdim, const double *q, const float *P, const float *Cx,
                     const float *mask, const float *va, double *alpha, double *ctx);

/* out = l - logsumexp(l); returns logsumexp(l). */
double mtref_log_softmax(int n, const double *l, double *out);

/* ---- batch and step ------------------------------------------------------------ */

/* Decoder start state and attention keys for B sentences:
 *   P[b,i,:] = ctx[b,i,:] Ua + ba for valid i (0 at padded i),
 *   s0[b,:] = tanh(mean_{valid i} ctx[b,i,:] Wi + bi). */
int mtref_precompute(const mtref_dims *d, const mtref_weights *w, int B, int S,
                     const float *ctx, const float *mask, float *P_out, float *s0_out);

/* One decoder step for M = B*K hypothesis rows (row m belongs to sentence m / K):
 *   x = emb[prev_tok[m]], h = state_in[src_row[m]]  (src_row < n_state_rows),
 *   s1 = GRU1(x, h), q = s1 Wa, (alpha, c) = attention(q), s = GRU2(c, s1),
 *   then s = transition_j(s) for j < transitions (deep transition),
 *   t = tanh(LN?(s Wt_s + x Wt_y + c Wt_c + bt)), logits = t Wo + bo,
 *   logp = log_softmax(logits).
 * Optional outputs (may be NULL): logp [M,V], alpha [M,S], s1/c/t taps. */
int mtref_step(const mtref_dims *d, const mtref_weights *w, int B, int K, int S,
               const int32_t *prev_tok, const int32_t *src_row, int n_state_rows,
               const float *state_in, const float *ctx, const float *P, const float *mask,
               float *state_out, float *logp_out, float *alpha_out,
               float *s1_out, float *c_out, float *t_out);

/* Encoder::build for the shallow model (Section 2.2; the Nematus-compatible encoder is a
 * bi-directional RNN, Section 3.1.1): ctx[b,i,:] = [f_i ; g_i] (C = 2H) with
 *   f_i = GRU(x_i, f_{i-1}; Wf, Uf, bf),  i = 0..S-1,  f_{-1} = 0,
 *   g_i = GRU(x_i, g_{i+1}; Wb, Ub, bb),  i = S-1..0,  g_S = 0,
 *   x_i = semb[src_tok[b,i]]; at a padded position (mask 0) a direction keeps its state
 *   (f_i = f_{i-1}, g_i = g_{i+1}).  No layer norm.  Every state stored in fp32. */
int mtref_encode(int E, int H, int Vs, int B, int S, const int32_t *src_tok, const float *mask,
                 const float *semb, const float *Wf, const float *Uf, const float *bf,
                 const float *Wb, const float *Ub, const float *bb, float *ctx_out);

/* The same with a deep-transition cell per direction (Section 3.1.1: the deep model's encoder
 * cell has four GRU blocks, with layer normalisation inside them): after the input block, T
 * recurrent-only transition blocks (mtref_gru_transition) with stacked Utf/btf (forward) and
 * Utb/btb (backward), [T,H,3H] and [T,3H]; a padded position carries the state over all
 * blocks.  Layer norm (lna_g NULL: none): the input block normalises both paths with
 * lna_g/lna_b (input path) and lnu_g/lnu_b (recurrent path), [2,3H] each, forward then
 * backward; transition block j of direction d normalises its recurrent path with
 * lnt_g/lnt_b[d][j], [2,T,3H]. */
int mtref_encode_deep(int E, int H, int Vs, int B, int S, const int32_t *src_tok, const float *mask,
                      const float *semb, const float *Wf, const float *Uf, const float *bf,
                      const float *Wb, const float *Ub, const float *bb, int T, const float *Utf,
                      const float *btf, const float *Utb, const float *btb, const float *lna_g,
                      const float *lna_b, const float *lnu_g, const float *lnu_b, const float *lnt_g,
                      const float *lnt_b, double eps, float *ctx_out);

/* Attention keys of the second source: P2 = ctx2 Ua2 + ba2 at valid positions, 0 elsewhere. */
int mtref_keys2(const mtref_dims *d, const mtref_weights *w, int B, int S, const float *ctx, const float *mask,
                float *P_out);

/* The step of a dual-source model: as mtref_step, and s1 also queries the second source
 * (S2 positions, ctx2 [B,S2,C], keys P2, mask2) through q2 = s1 Wa2 and va2; GRU 2 and the
 * readout take c = [c1 ; c2] (2C wide; the c tap is [M, 2C]); alpha is the first source's. */
int mtref_step_dual(const mtref_dims *d, const mtref_weights *w, int B, int K, int S,
                    const int32_t *prev_tok, const int32_t *src_row, int n_state_rows,
                    const float *state_in, const float *ctx, const float *P, const float *mask,
                    int S2, const float *ctx2, const float *P2, const float *mask2,
                    float *state_out, float *logp_out, float *alpha_out,
                    float *s1_out, float *c_out, float *t_out);

/* Beam selection: for each sentence b, candidates cand(k,v) = score[b*K+k] +
 * logp[b*K+k, v] evaluated in fp32; the K best by (cand descending, flat
 * index k*V+v ascending) give score_out, tok_out = v, bp_out = k. */
int mtref_topk(int B, int K, int V, const float *prev_score, const float *logp,
               int32_t *tok_out, int32_t *bp_out, float *score_out);

#ifdef __cplusplus
}
#endif
#endif
