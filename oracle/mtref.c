/*
 * mtref.c — CPU oracle for the decoder step (see mtref.h).
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
 * benchmark's CPU-baseline leg; never by the GPU library.
 *
 * The paper (Marian, arXiv 1804.00344) names the operators of the step —
 * fused GRU cells, attention, layer normalisation (Section 2.1) — and the
 * encoder/decoder interface it fits in (Section 2.2, Decoder::startState and
 * Decoder::step), but prints no equations.  The shallow model is stated to
 * be binary-compatible with Nematus (Section 1); the equations below are that
 * model's conditional GRU written out plainly.  Every reading taken where
 * the paper is silent is listed in the design notes; the ones that change
 * numbers are repeated at the function that applies them.
 *
 * Plain loops; double accumulation; fp32 storage at stage boundaries.
 */
#include "mtref.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* Layer normalisation (Ba et al., named in Section 2.1 and 3.1.1): biased
 * variance, eps inside the square root. */
void mtref_layer_norm(int n, const double *x, const float *gamma, const float *beta,
                      double eps, double *y) {
  double mean = 0.0;
  for (int i = 0; i < n; ++i) mean += x[i];
  mean /= n;
  double var = 0.0;
  for (int i = 0; i < n; ++i) var += (x[i] - mean) * (x[i] - mean);
  var /= n;
  double inv = 1.0 / sqrt(var + eps);
  for (int i = 0; i < n; ++i) y[i] = (double)gamma[i] * (x[i] - mean) * inv + (double)beta[i];
}

/* out[j] = bias[j] + sum_i in[i] * W[i*ld + j], j < n_out (bias may be NULL). */
static void vec_mat(int n_in, int n_out, int ld, const double *in, const float *W,
                    const float *bias, double *out) {
  for (int j = 0; j < n_out; ++j) out[j] = bias ? (double)bias[j] : 0.0;
  for (int i = 0; i < n_in; ++i) {
    double xi = in[i];
    const float *row = W + (size_t)i * ld;
    for (int j = 0; j < n_out; ++j) out[j] += xi * (double)row[j];
  }
}

/* GRU block (Section 2.1 "fused RNN cells"; Nematus cGRU sub-block).
 * Gate blocks are ordered r, z, h inside the 3H columns.  The reset gate
 * multiplies the recurrent product (h U_h), and z gates the previous state:
 * out = (1 - z) hh + z h.  Only the input path carries a bias.  With layer
 * normalisation, each H-block of each path is normalised on its own. */
void mtref_gru(int in_dim, int H, const double *x, const double *h,
               const float *W, const float *U, const float *b,
               const float *ln_ga, const float *ln_ba, const float *ln_gu, const float *ln_bu,
               double eps, double *out) {
  double *a = (double *)malloc(sizeof(double) * 3 * H);
  double *u = (double *)malloc(sizeof(double) * 3 * H);
  vec_mat(in_dim, 3 * H, 3 * H, x, W, b, a);
  vec_mat(H, 3 * H, 3 * H, h, U, NULL, u);
  if (ln_ga) {
    for (int g = 0; g < 3; ++g) {
      mtref_layer_norm(H, a + g * H, ln_ga + g * H, ln_ba + g * H, eps, a + g * H);
      mtref_layer_norm(H, u + g * H, ln_gu + g * H, ln_bu + g * H, eps, u + g * H);
    }
  }
  for (int j = 0; j < H; ++j) {
    double r = sigmoid(a[j] + u[j]);
    double z = sigmoid(a[H + j] + u[H + j]);
    double hh = tanh(a[2 * H + j] + r * u[2 * H + j]);
    out[j] = (1.0 - z) * hh + z * h[j];
  }
  free(a);
  free(u);
}

/* Transition block (Section 3.1.1: the deep-transition decoder cell stacks eight GRU
 * blocks per step, attention between the first and the second).  Blocks past the second
 * receive no external input, so their input path reduces to its bias; with layer
 * normalisation only the recurrent product's H-blocks are normalised (the input path has
 * no product to normalise).  Reading of the paper, which names the blocks only. */
void mtref_gru_transition(int H, const double *h, const float *U, const float *b,
                          const float *ln_gu, const float *ln_bu, double eps, double *out) {
  double *u = (double *)malloc(sizeof(double) * 3 * H);
  vec_mat(H, 3 * H, 3 * H, h, U, NULL, u);
  if (ln_gu)
    for (int g = 0; g < 3; ++g) mtref_layer_norm(H, u + g * H, ln_gu + g * H, ln_bu + g * H, eps, u + g * H);
  for (int j = 0; j < H; ++j) {
    double r = sigmoid((double)b[j] + u[j]);
    double z = sigmoid((double)b[H + j] + u[H + j]);
    double hh = tanh((double)b[2 * H + j] + r * u[2 * H + j]);
    out[j] = (1.0 - z) * hh + z * h[j];
  }
  free(u);
}

/* Additive (Bahdanau) attention with a masked softmax (Section 2.1 "attention
 * mechanisms"; Section 2.2: the encoder context and its mask live in the
 * EncoderState).  The maximum is taken over valid positions only; masked
 * weights are set to zero, never computed. */
void mtref_attention(int S, int A, int Cdim, const double *q, const float *P, const float *Cx,
                     const float *mask, const float *va, double *alpha, double *ctx) {
  double *e = (double *)malloc(sizeof(double) * (S > 0 ? S : 1));
  int any = 0;
  double mx = -INFINITY;
  for (int i = 0; i < S; ++i) {
    if (mask[i] == 0.0f) continue;
    double acc = 0.0;
    for (int k = 0; k < A; ++k) acc += (double)va[k] * tanh((double)P[(size_t)i * A + k] + q[k]);
    e[i] = acc;
    if (!any || acc > mx) mx = acc;
    any = 1;
  }
  double den = 0.0;
  for (int i = 0; i < S; ++i)
    if (mask[i] != 0.0f) den += exp(e[i] - mx);
  for (int i = 0; i < S; ++i) alpha[i] = (mask[i] != 0.0f) ? exp(e[i] - mx) / den : 0.0;
  for (int c = 0; c < Cdim; ++c) ctx[c] = 0.0;
  for (int i = 0; i < S; ++i) {
    if (mask[i] == 0.0f) continue;
    const float *row = Cx + (size_t)i * Cdim;
    for (int c = 0; c < Cdim; ++c) ctx[c] += alpha[i] * (double)row[c];
  }
  free(e);
}

double mtref_log_softmax(int n, const double *l, double *out) {
  double mx = l[0];
  for (int i = 1; i < n; ++i)
    if (l[i] > mx) mx = l[i];
  double s = 0.0;
  for (int i = 0; i < n; ++i) s += exp(l[i] - mx);
  double lse = mx + log(s);
  for (int i = 0; i < n; ++i) out[i] = l[i] - lse;
  return lse;
}

static void to_double(int n, const float *src, double *dst) {
  for (int i = 0; i < n; ++i) dst[i] = (double)src[i];
}
static void round_store(int n, const double *src, float *dst, double *keep) {
  /* store in fp32 and continue from the stored value */
  for (int i = 0; i < n; ++i) {
    float f = (float)src[i];
    dst[i] = f;
    if (keep) keep[i] = (double)f;
  }
}

/* Decoder::startState (Section 2.2): per-batch attention keys and the
 * initial state from the masked mean of the encoder context. */
int mtref_precompute(const mtref_dims *d, const mtref_weights *w, int B, int S,
                     const float *ctx, const float *mask, float *P_out, float *s0_out) {
  if (!d || !w || B < 0 || S < 1 || !ctx || !mask || !P_out || !s0_out) return -1;
  const int H = d->H, C = 2 * d->H, A = d->A;
  double *row = (double *)malloc(sizeof(double) * C);
  double *tmp = (double *)malloc(sizeof(double) * (A > H ? A : H));
  double *mean = (double *)malloc(sizeof(double) * C);
  for (int b = 0; b < B; ++b) {
    int n = 0;
    for (int c = 0; c < C; ++c) mean[c] = 0.0;
    for (int i = 0; i < S; ++i) {
      float *Pr = P_out + ((size_t)b * S + i) * A;
      if (mask[(size_t)b * S + i] == 0.0f) {
        for (int a = 0; a < A; ++a) Pr[a] = 0.0f;
        continue;
      }
      const float *cr = ctx + ((size_t)b * S + i) * C;
      to_double(C, cr, row);
      vec_mat(C, A, A, row, w->Ua, w->ba, tmp);
      round_store(A, tmp, Pr, NULL);
      for (int c = 0; c < C; ++c) mean[c] += row[c];
      ++n;
    }
    for (int c = 0; c < C; ++c) mean[c] = n ? mean[c] / n : 0.0;
    vec_mat(C, H, H, mean, w->Wi, w->bi, tmp);
    for (int j = 0; j < H; ++j) tmp[j] = tanh(tmp[j]);
    round_store(H, tmp, s0_out + (size_t)b * H, NULL);
  }
  free(row);
  free(tmp);
  free(mean);
  return 0;
}

/* Attention keys of a second source (dual-source models): P2 = ctx2 Ua2 + ba2 at valid
 * positions, 0 elsewhere. */
int mtref_keys2(const mtref_dims *d, const mtref_weights *w, int B, int S, const float *ctx, const float *mask,
                float *P_out) {
  if (!d || !w || !w->Ua2 || !w->ba2 || B < 0 || S < 1 || !ctx || !mask || !P_out) return -1;
  const int C = 2 * d->H, A = d->A;
  double *row = (double *)malloc(sizeof(double) * C);
  double *tmp = (double *)malloc(sizeof(double) * A);
  for (long i = 0; i < (long)B * S; ++i) {
    float *Pr = P_out + (size_t)i * A;
    if (mask[i] == 0.0f) {
      for (int a = 0; a < A; ++a) Pr[a] = 0.0f;
      continue;
    }
    to_double(C, ctx + (size_t)i * C, row);
    vec_mat(C, A, A, row, w->Ua2, w->ba2, tmp);
    round_store(A, tmp, Pr, NULL);
  }
  free(row);
  free(tmp);
  return 0;
}

/* Decoder::step for one batch of hypotheses (Section 2.2: consumes the target
 * part of the batch and produces the logits and the next state).  With a second
 * source (S2 > 0; dual-attention models of the post-editing systems in Section 3.2)
 * the intermediate state s1 also queries the second source through its own attention,
 * and GRU block 2 and the readout take the two contexts side by side. */
static int step_impl(const mtref_dims *d, const mtref_weights *w, int B, int K, int S,
                     const int32_t *prev_tok, const int32_t *src_row, int n_state_rows,
                     const float *state_in, const float *ctx, const float *P, const float *mask,
                     int S2, const float *ctx2, const float *P2, const float *mask2,
                     float *state_out, float *logp_out, float *alpha_out,
                     float *s1_out, float *c_out, float *t_out) {
  if (!d || !w || B < 0 || K < 1 || S < 1 || !prev_tok || !src_row || !state_in || !ctx ||
      !P || !mask || !state_out || d->transitions < 0 ||
      (d->transitions > 0 && (!w->Ut || !w->btr || (d->layer_norm && (!w->gtu || !w->betu)))) ||
      (S2 > 0 && (!ctx2 || !P2 || !mask2 || !w->Wa2 || !w->va2)))
    return -1;
  const int E = d->E, H = d->H, C1 = 2 * d->H, A = d->A, V = d->V;
  const int C = S2 > 0 ? 2 * C1 : C1;  /* width of the context fed to GRU 2 and the readout */
  const int M = B * K;
  for (int m = 0; m < M; ++m) {
    if (prev_tok[m] < 0 || prev_tok[m] >= V) return -2;
    if (src_row[m] < 0 || src_row[m] >= n_state_rows) return -2;
  }
  const int ln = d->layer_norm;
  double *x = (double *)malloc(sizeof(double) * E);
  double *h = (double *)malloc(sizeof(double) * H);
  double *s1 = (double *)malloc(sizeof(double) * H);
  double *q = (double *)malloc(sizeof(double) * A);
  double *al = (double *)malloc(sizeof(double) * (S > S2 ? S : S2));
  double *c = (double *)malloc(sizeof(double) * C);
  double *s = (double *)malloc(sizeof(double) * H);
  double *t = (double *)malloc(sizeof(double) * E);
  double *part = (double *)malloc(sizeof(double) * E);
  double *l = (double *)malloc(sizeof(double) * V);
  int fmax = H;
  if (A > fmax) fmax = A;
  if (C > fmax) fmax = C;
  if (E > fmax) fmax = E;
  float *f = (float *)malloc(sizeof(float) * (size_t)fmax);
  for (int m = 0; m < M; ++m) {
    const int b = m / K;
    to_double(E, w->emb + (size_t)prev_tok[m] * E, x);
    to_double(H, state_in + (size_t)src_row[m] * H, h);

    /* GRU block 1: input = previous target embedding, state = selected hypothesis state */
    mtref_gru(E, H, x, h, w->W1, w->U1, w->b1, ln ? w->g1a : NULL, ln ? w->be1a : NULL,
              ln ? w->g1u : NULL, ln ? w->be1u : NULL, d->ln_eps, s1);
    round_store(H, s1, f, s1);
    if (s1_out) memcpy(s1_out + (size_t)m * H, f, sizeof(float) * H);

    /* attention query from the intermediate state */
    vec_mat(H, A, A, s1, w->Wa, NULL, q);
    round_store(A, q, f, q);
    mtref_attention(S, A, C1, q, P + (size_t)b * S * A, ctx + (size_t)b * S * C1,
                    mask + (size_t)b * S, w->va, al, c);
    if (alpha_out)
      for (int i = 0; i < S; ++i) alpha_out[(size_t)m * S + i] = (float)al[i];
    if (S2 > 0) {  /* the second source: its own query projection, keys and va */
      vec_mat(H, A, A, s1, w->Wa2, NULL, q);
      round_store(A, q, f, q);
      mtref_attention(S2, A, C1, q, P2 + (size_t)b * S2 * A, ctx2 + (size_t)b * S2 * C1,
                      mask2 + (size_t)b * S2, w->va2, al, c + C1);
    }
    round_store(C, c, f, c);
    if (c_out) memcpy(c_out + (size_t)m * C, f, sizeof(float) * C);

    /* GRU block 2: input = attention context, state = s1 */
    mtref_gru(C, H, c, s1, w->W2, w->U2, w->b2, ln ? w->g2a : NULL, ln ? w->be2a : NULL,
              ln ? w->g2u : NULL, ln ? w->be2u : NULL, d->ln_eps, s);
    round_store(H, s, f, s);
    /* deep transition: recurrent-only blocks, each output stored in fp32 */
    for (int j = 0; j < d->transitions; ++j) {
      mtref_gru_transition(H, s, w->Ut + (size_t)j * H * 3 * H, w->btr + (size_t)j * 3 * H,
                           ln ? w->gtu + (size_t)j * 3 * H : NULL, ln ? w->betu + (size_t)j * 3 * H : NULL,
                           d->ln_eps, s1);
      round_store(H, s1, f, s);
    }
    memcpy(state_out + (size_t)m * H, f, sizeof(float) * H);

    /* deep-output readout: tanh of the sum of three projections to E */
    vec_mat(H, E, E, s, w->Wt_s, w->bt, t);
    vec_mat(E, E, E, x, w->Wt_y, NULL, part);
    for (int e = 0; e < E; ++e) t[e] += part[e];
    vec_mat(C, E, E, c, w->Wt_c, NULL, part);
    for (int e = 0; e < E; ++e) t[e] += part[e];
    if (ln) mtref_layer_norm(E, t, w->gt, w->bet, d->ln_eps, t);
    for (int e = 0; e < E; ++e) t[e] = tanh(t[e]);
    round_store(E, t, f, t);
    if (t_out) memcpy(t_out + (size_t)m * E, f, sizeof(float) * E);

    /* output layer and log-softmax over the target vocabulary */
    if (logp_out) {
      if (d->tied_output) {
        for (int v = 0; v < V; ++v) {
          double acc = (double)w->bo[v];
          const float *er = w->emb + (size_t)v * E;
          for (int e = 0; e < E; ++e) acc += t[e] * (double)er[e];
          l[v] = acc;
        }
      } else {
        vec_mat(E, V, V, t, w->Wo, w->bo, l);
      }
      mtref_log_softmax(V, l, l);
      for (int v = 0; v < V; ++v) logp_out[(size_t)m * V + v] = (float)l[v];
    }
  }
  free(x); free(h); free(s1); free(q); free(al); free(c); free(s); free(t); free(part);
  free(l); free(f);
  return 0;
}

int mtref_step(const mtref_dims *d, const mtref_weights *w, int B, int K, int S,
               const int32_t *prev_tok, const int32_t *src_row, int n_state_rows,
               const float *state_in, const float *ctx, const float *P, const float *mask,
               float *state_out, float *logp_out, float *alpha_out,
               float *s1_out, float *c_out, float *t_out) {
  return step_impl(d, w, B, K, S, prev_tok, src_row, n_state_rows, state_in, ctx, P, mask, 0, NULL, NULL, NULL,
                   state_out, logp_out, alpha_out, s1_out, c_out, t_out);
}

int mtref_step_dual(const mtref_dims *d, const mtref_weights *w, int B, int K, int S,
                    const int32_t *prev_tok, const int32_t *src_row, int n_state_rows,
                    const float *state_in, const float *ctx, const float *P, const float *mask,
                    int S2, const float *ctx2, const float *P2, const float *mask2,
                    float *state_out, float *logp_out, float *alpha_out,
                    float *s1_out, float *c_out, float *t_out) {
  if (S2 < 1) return -1;
  return step_impl(d, w, B, K, S, prev_tok, src_row, n_state_rows, state_in, ctx, P, mask, S2, ctx2, P2, mask2,
                   state_out, logp_out, alpha_out, s1_out, c_out, t_out);
}

/* Encoder::build for the shallow model (Section 2.2; bi-directional RNN encoder, Section
 * 3.1.1): a forward and a backward GRU block over the source embeddings, their states side by
 * side.  A padded position carries each direction's state over (reading of the paper, which
 * does not spell out the padding). */
int mtref_encode(int E, int H, int Vs, int B, int S, const int32_t *src_tok, const float *mask,
                 const float *semb, const float *Wf, const float *Uf, const float *bf,
                 const float *Wb, const float *Ub, const float *bb, float *ctx_out) {
  return mtref_encode_deep(E, H, Vs, B, S, src_tok, mask, semb, Wf, Uf, bf, Wb, Ub, bb, 0, NULL, NULL, NULL, NULL,
                           NULL, NULL, NULL, NULL, NULL, NULL, 0.0, ctx_out);
}

/* Deep-transition encoder cell (Section 3.1.1: four GRU blocks per encoder cell, layer
 * normalisation inside the blocks): the input block, then T blocks without external input,
 * each output stored in fp32. */
int mtref_encode_deep(int E, int H, int Vs, int B, int S, const int32_t *src_tok, const float *mask,
                      const float *semb, const float *Wf, const float *Uf, const float *bf,
                      const float *Wb, const float *Ub, const float *bb, int T, const float *Utf,
                      const float *btf, const float *Utb, const float *btb, const float *lna_g,
                      const float *lna_b, const float *lnu_g, const float *lnu_b, const float *lnt_g,
                      const float *lnt_b, double eps, float *ctx_out) {
  if (E < 1 || H < 1 || Vs < 1 || B < 0 || S < 1 || !src_tok || !mask || !semb || !Wf || !Uf || !bf ||
      !Wb || !Ub || !bb || !ctx_out || T < 0 || (T > 0 && (!Utf || !btf || !Utb || !btb)))
    return -1;
  const int ln = lna_g != NULL;
  if (ln && (!lna_b || !lnu_g || !lnu_b || (T > 0 && (!lnt_g || !lnt_b)))) return -1;
  for (long i = 0; i < (long)B * S; ++i)
    if (src_tok[i] < 0 || src_tok[i] >= Vs) return -2;
  const int C = 2 * H;
  double *x = (double *)malloc(sizeof(double) * E);
  double *h = (double *)malloc(sizeof(double) * H);
  double *hn = (double *)malloc(sizeof(double) * H);
  for (int b = 0; b < B; ++b) {
    for (int dir = 0; dir < 2; ++dir) {
      for (int j = 0; j < H; ++j) h[j] = 0.0;
      for (int n = 0; n < S; ++n) {
        const int i = dir == 0 ? n : S - 1 - n;
        float *out = ctx_out + ((size_t)b * S + i) * C + (size_t)dir * H;
        if (mask[(size_t)b * S + i] != 0.f) {
          to_double(E, semb + (size_t)src_tok[(size_t)b * S + i] * E, x);
          const size_t lo = (size_t)dir * 3 * H;
          mtref_gru(E, H, x, h, dir == 0 ? Wf : Wb, dir == 0 ? Uf : Ub, dir == 0 ? bf : bb,
                    ln ? lna_g + lo : NULL, ln ? lna_b + lo : NULL, ln ? lnu_g + lo : NULL, ln ? lnu_b + lo : NULL,
                    eps, hn);
          round_store(H, hn, out, h);
          for (int j = 0; j < T; ++j) {
            const float *U = (dir == 0 ? Utf : Utb) + (size_t)j * H * 3 * H;
            const float *bt = (dir == 0 ? btf : btb) + (size_t)j * 3 * H;
            const size_t to = ((size_t)dir * T + j) * 3 * H;
            mtref_gru_transition(H, h, U, bt, ln ? lnt_g + to : NULL, ln ? lnt_b + to : NULL, eps, hn);
            round_store(H, hn, out, h);
          }
        } else {
          for (int j = 0; j < H; ++j) out[j] = (float)h[j];
        }
      }
    }
  }
  free(x);
  free(h);
  free(hn);
  return 0;
}

typedef struct {
  float key;
  int32_t idx; /* k*V + v */
} cand_t;

static int cand_cmp(const void *pa, const void *pb) {
  const cand_t *a = (const cand_t *)pa, *b = (const cand_t *)pb;
  if (a->key > b->key) return -1;
  if (a->key < b->key) return 1;
  return (a->idx > b->idx) - (a->idx < b->idx);
}

/* Beam selection over the K x V extensions of each sentence (Section 2.2:
 * decoder states are used to select the next hypotheses; Section 2.3 batched
 * beam search).  A full sort of all candidates by (score desc, flat index
 * asc); the candidate score is summed in fp32, the precision the beam keeps
 * its scores in. */
int mtref_topk(int B, int K, int V, const float *prev_score, const float *logp,
               int32_t *tok_out, int32_t *bp_out, float *score_out) {
  if (B < 0 || K < 1 || V < 1 || !prev_score || !logp || !tok_out || !bp_out || !score_out)
    return -1;
  size_t n = (size_t)K * V;
  cand_t *cs = (cand_t *)malloc(sizeof(cand_t) * n);
  for (int b = 0; b < B; ++b) {
    for (int k = 0; k < K; ++k) {
      float sc = prev_score[b * K + k];
      const float *lp = logp + ((size_t)b * K + k) * V;
      for (int v = 0; v < V; ++v) {
        volatile float key = sc + lp[v];
        cs[(size_t)k * V + v].key = key;
        cs[(size_t)k * V + v].idx = k * V + v;
      }
    }
    qsort(cs, n, sizeof(cand_t), cand_cmp);
    for (int j = 0; j < K; ++j) {
      score_out[b * K + j] = cs[j].key;
      tok_out[b * K + j] = cs[j].idx % V;
      bp_out[b * K + j] = cs[j].idx / V;
    }
  }
  free(cs);
  return 0;
}
