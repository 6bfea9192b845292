/*
 * libmtstep — one batched beam-search step of a shallow attentional cGRU
 * decoder on an AMD Instinct MI355X (gfx950), behind a plain C ABI.
 *
 * The calls follow the encoder/decoder interface of Marian (arXiv
 * 1804.00344, Section 2.2): the encoder's output (context + mask, the
 * EncoderState) is an input here; mt_precompute_ctx plays
 * Decoder::startState (per-batch attention keys and the initial state);
 * mt_decoder_step plays Decoder::step (next state and the log-probabilities
 * over the target vocabulary); mt_beam_topk is the selection of the next
 * hypotheses from the decoder state (Section 2.2, last paragraphs; batched
 * beam search, Section 2.3).  The model is the shallow Nematus-compatible
 * RNN of Section 1 / Table 2 ("Shallow RNN"): conditional GRU with fused
 * gates and optional layer normalisation (Section 2.1), additive attention
 * with a masked softmax, a deep-output readout, the output projection and a
 * log-softmax.
 *
 * Model (row m = b*K + k of sentence b, all matrices stored [in x out]):
 *   x  = emb[prev_tok[m]],        h = state_in[src_row[m]]
 *   s1 = GRU(x, h; W1, U1, b1)    GRU(x,h): a = xW + b, u = hU, per-block LN
 *                                 (if enabled) on a_r,a_z,a_h,u_r,u_z,u_h,
 *                                 r = sig(a_r+u_r), z = sig(a_z+u_z),
 *                                 hh = tanh(a_h + r*u_h), out = (1-z)hh + z h
 *   q  = s1 Wa;  e_i = va . tanh(P[b,i] + q) for valid i;  alpha = softmax(e)
 *   c  = sum_i alpha_i ctx[b,i]
 *   s  = GRU(c, s1; W2, U2, b2)   -> state_out[m]
 *   t  = tanh(LN?(s Wt_s + x Wt_y + c Wt_c + bt))
 *   logp = log_softmax(t Wo + bo)
 * with P[b,i] = ctx[b,i] Ua + ba and s0[b] = tanh(mean_valid(ctx[b]) Wi + bi).
 *
 * Conventions for every call:
 *   - Device pointers unless stated otherwise; row-major; 16-byte aligned.
 *   - Calls are asynchronous on the given HIP stream (a hipStream_t passed as
 *     void*, NULL = the null stream) and never synchronise, except
 *     mt_load_weights, mt_free, mt_device_errors and mt_profile_query.
 *   - Every argument is validated on the host before anything is launched;
 *     a failed call launches nothing and returns a negative mt_status, with a
 *     message in mt_last_error().  Kernel faults surface at the caller's
 *     next synchronisation.
 *   - One model handle serves one stream at a time.  Callers own every
 *     activation buffer and the workspace; the library allocates only in
 *     mt_load_weights and never per step.
 */
#ifndef MTSTEP_H
#define MTSTEP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MT_OK = 0,
  MT_ERR_ARG = -1,       /* null/misaligned pointer, bad enum, bad flag */
  MT_ERR_SHAPE = -2,     /* a size out of its supported range */
  MT_ERR_DTYPE = -3,     /* unsupported dtype */
  MT_ERR_HIP = -4,       /* a HIP runtime call failed (message says which) */
  MT_ERR_OOM = -5,       /* device allocation failed in mt_load_weights */
  MT_ERR_STATE = -6,     /* call order violated (e.g. top-K without a step) */
  MT_ERR_WORKSPACE = -7  /* workspace too small */
} mt_status;

typedef enum { MT_F32 = 0, MT_BF16 = 1 } mt_dtype;

/* Model shape and options.
 *   E, H, A: multiples of 16 with 16 <= E, H <= 4096 and 16 <= A <= 4096;
 *   C = 2H (bi-directional encoder context); 2 <= V <= 2^24.
 *   gemm_dtype: operand type of every matrix product (accumulation is fp32).
 *     MT_BF16 also stores the encoder context and attention keys in bf16.
 *     Gates, layer norm, softmax, log-softmax, states and scores stay fp32.
 *   layer_norm: 0/1 — LN on each gate block of both paths of both GRUs and
 *     on the readout pre-activation (eps = ln_eps, biased variance).
 *   tied_output: 0/1 — the output matrix is emb transposed (Wo ignored).
 *   k_max: largest beam size the model will be called with, 1..16.
 *   dec_transitions: 0..16 — recurrent-only GRU blocks after GRU 2 (the
 *     deep-transition decoder cell of Section 3.1.1: eight blocks in all,
 *     attention between the first and the second, is 6); 0 is the shallow
 *     cGRU.  Such a block has no external input (its input path is its bias
 *     alone); with layer_norm its recurrent product is normalised per gate
 *     block.  The new state and the readout take the last block's output. */
typedef struct {
  int32_t E, H, A, V;
  int32_t layer_norm;
  int32_t tied_output;
  int32_t k_max;
  int32_t gemm_dtype;
  float ln_eps;
  int32_t dec_transitions;
  int32_t src_V;  /* source vocabulary of the encoder (mt_encode); 0: no encoder */
  int32_t dual_source;  /* 1: a second source with its own attention (mt_decoder_step_dual) */
  int32_t enc_transitions; /* 0..16: recurrent-only GRU blocks after the input block of each
                            * encoder direction (the deep-transition encoder cell of Section
                            * 3.1.1 has four blocks in all: 3); needs src_V > 0. */
  int32_t enc_layer_norm;  /* 0/1: layer norm inside the encoder's GRU blocks (eps = ln_eps):
                            * per gate block on both paths of each direction's input block and
                            * on the recurrent path of each transition block; needs src_V > 0 */
} mt_config;

/* Model parameters: HOST pointers to fp32, row-major logical [in x out]
 * (gate blocks of the [*, 3H] matrices in the order r, z, h).  Only read
 * during mt_load_weights; the caller may free them afterwards.
 *   emb[V,E]; W1[E,3H] U1[H,3H] b1[3H]; Ua[C,A] ba[A] Wa[H,A] va[A];
 *   W2[C,3H] U2[H,3H] b2[3H]; Wt_s[H,E] Wt_y[E,E] Wt_c[C,E] bt[E];
 *   Wo[E,V] bo[V]; Wi[C,H] bi[H];
 *   layer norm (read only if layer_norm): gain/shift of the input path (a)
 *   and recurrent path (u) of GRU 1 and 2, [3H] each; readout gt/bet [E];
 *   transition blocks (read only if dec_transitions = T > 0), stacked by
 *   block: Ut[T,H,3H] btr[T,3H], and with layer_norm gtu/betu[T,3H];
 *   encoder (read only if src_V > 0): semb[src_V,E], forward Wef[E,3H]
 *   Uef[H,3H] bef[3H], backward Web[E,3H] Ueb[H,3H] beb[3H];
 *   second source (read only if dual_source): Ua2[C,A] ba2[A] Wa2[H,A] va2[A],
 *   and W2 [2C,3H], Wt_c [2C,E] then take the two contexts side by side;
 *   encoder transition blocks (read only if enc_transitions = T > 0), stacked
 *   by block: forward Utef[T,H,3H] btef[T,3H], backward Uteb[T,H,3H] bteb[T,3H];
 *   encoder layer norm (read only if enc_layer_norm), forward then backward: gain/shift
 *   of the input blocks' input path gea/bea[2,3H] and recurrent path geu/beu[2,3H], and of
 *   the transition blocks' recurrent path gteu/beteu[2,T,3H]. */
typedef struct {
  const float *emb;
  const float *W1, *U1, *b1;
  const float *Ua, *ba, *Wa, *va;
  const float *W2, *U2, *b2;
  const float *Wt_s, *Wt_y, *Wt_c, *bt;
  const float *Wo, *bo;
  const float *Wi, *bi;
  const float *g1a, *be1a, *g1u, *be1u, *g2a, *be2a, *g2u, *be2u, *gt, *bet;
  const float *Ut, *btr, *gtu, *betu;
  const float *semb, *Wef, *Uef, *bef, *Web, *Ueb, *beb;
  const float *Ua2, *ba2, *Wa2, *va2;
  const float *Utef, *btef, *Uteb, *bteb;
  const float *gea, *bea, *geu, *beu, *gteu, *beteu;
} mt_weights;

typedef struct mt_model mt_model; /* opaque, library-owned */

/* Optional per-stage outputs of mt_decoder_step, each fp32 [B*K, n] or NULL:
 * s1 (n = H), c (n = 2H; 4H for dual-source models, both contexts), t (n = E).  For
 * stage-level checks. */
typedef struct {
  float *s1;
  float *c;
  float *t;
} mt_taps;

/* Copy, pack and convert the weights into library-owned device memory on
 * the current HIP device (fused gate layouts, K-contiguous transposes,
 * bf16 round-to-nearest-even when gemm_dtype is MT_BF16), and compute the
 * token-side table emb [W1 | Wt_y] + [b1 | 0] ([V, 3H+E] fp32, V(3H+E)*4
 * bytes of device memory) that the step gathers rows from.  Synchronous.
 * On success *out receives the handle; release it with mt_free. */
mt_status mt_load_weights(const mt_config *cfg, const mt_weights *w, mt_model **out);

/* Release a handle and its device memory (synchronises the device). */
mt_status mt_free(mt_model *model);

/* Workspace bytes that mt_precompute_ctx, mt_decoder_step and mt_beam_topk
 * need for B sentences, beam K and padded source length S; 0 on bad input.
 * The same workspace must be passed to a step and to the mt_beam_topk call
 * that consumes it (it carries the fused top-K candidates between them). */
size_t mt_workspace_bytes(const mt_model *model, int B, int K, int S);

/* Workspace bytes of mt_encode for B sentences of padded length S (0 on bad input or
 * when the model has no encoder). */
size_t mt_encode_workspace_bytes(const mt_model *model, int B, int S);

/* Encoder::build of the shallow model (Section 2.2; bi-directional RNN encoder):
 *   ctx_out [B,S,2H] in gemm dtype: ctx[b,i] = [f_i ; g_i], f the forward GRU over
 *   positions 0..S-1 and g the backward one over S-1..0 (zero initial states) on the
 *   source embeddings semb[src_tok[b,i]]; at a masked position each direction carries its
 *   state over (no layer norm).  Ready for mt_precompute_ctx and mt_decoder_step.
 *   src_tok [B,S] int32 in [0, src_V) (clamped, reported by mt_device_errors);
 *   mask [B,S] fp32 as for mt_precompute_ctx.  bf16 models keep the states in fp32 in the
 *   workspace and write their bf16 rounding (also the recurrent products' operand).
 * 1 <= S <= 1024; B*S <= 2^24.  One product for the input side of every position, then
 * one recurrent product and two cells per position: 3S launches. */
mt_status mt_encode(mt_model *model, int B, int S, const int32_t *src_tok, const float *mask, void *ctx_out,
                    void *ws, size_t ws_bytes, void *stream);

/* Decoder start state for B sentences (Section 2.2, Decoder::startState):
 *   ctx  [B,S,2H] in gemm dtype (fp32 or bf16) — the encoder context;
 *   mask [B,S] fp32, nonzero = valid position (any pattern; a row without a
 *        valid position yields zero context and zero attention);
 *   pctx_out [B,S,A] in gemm dtype — attention keys ctx Ua + ba, computed and
 *        written at valid positions only (masked rows are left as they were and
 *        never read);
 *   s0_out [B,H] fp32 — tanh(masked mean of ctx[b] times Wi + bi).
 * It also records in the model the order of the B sentences by length, which later steps
 * with the same B use to schedule their attention (the longest first); it decides
 * scheduling only, never results.
 * 1 <= S <= 1024; B*S <= 2^24. */
mt_status mt_precompute_ctx(mt_model *model, int B, int S, const void *ctx, const float *mask,
                            void *pctx_out, float *s0_out, void *ws, size_t ws_bytes,
                            void *stream);

/* One decoder step for M = B*K hypothesis rows (Section 2.2, Decoder::step):
 *   prev_tok [M] int32 in [0,V); src_row [M] int32 in [0,n_state_rows):
 *   row m reads h = state_in[src_row[m]] (at step 0 pass s0 with
 *   src_row[m] = m / K; later pass the previous state_out with row_out of
 *   mt_beam_topk).  Out-of-range indices are clamped and reported by
 *   mt_device_errors.  state_in [n_state_rows,H] fp32;
 *   ctx/pctx/mask as produced for mt_precompute_ctx;
 *   state_out [M,H] fp32 (must not alias state_in);
 *   logp_out [M,V] fp32 or NULL — materialised log-probabilities;
 *   attn_out [M,S] fp32 or NULL — attention weights (0 at masked positions);
 *   taps: NULL or optional stage outputs.
 * 1 <= K <= k_max, K <= V. */
mt_status mt_decoder_step(mt_model *model, int B, int K, int S, const int32_t *prev_tok,
                          const int32_t *src_row, int n_state_rows, const float *state_in,
                          const void *ctx, const void *pctx, const float *mask, float *state_out,
                          float *logp_out, float *attn_out, const mt_taps *taps, void *ws,
                          size_t ws_bytes, void *stream);

/* mt_precompute_ctx without a workspace argument, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid it): the
 * same kernels and results, with the workspace in a library-owned scratch array of 16 MiB
 * per GPU (a file-scope device array, allocated when the library's code is loaded on a GPU
 * and held until the process ends).  Calls no hipMalloc, hipFree or other allocating routine
 * and records no profiling events.  Needs rup256(B*2H*4) + rup256(B*S*4) + 256 bytes <= 16 MiB
 * (e.g. B <= 1900 at H = 1024, S = 80), else MT_ERR_WORKSPACE; the current device must be the
 * one the model was loaded on (MT_ERR_STATE otherwise).  Every call on a GPU shares that GPU's
 * scratch: calls that overlap on one GPU (other streams, other threads, other models) race.
 * Nothing in the scratch has to start at zero: every byte a call reads it first writes. */
mt_status mt_precompute_ctx_noalloc(mt_model *model, int B, int S, const void *ctx, const float *mask,
                                    void *pctx_out, float *s0_out, void *stream);

/* Dual-source models (the dual-attention post-editing models of Section 3.2: two encoders,
 * a decoder attending to both).  mt_precompute_keys2: the second source's attention keys
 * pctx2_out [B,S2,A] = ctx2 Ua2 + ba2 at its valid positions (ctx2 [B,S2,2H] and mask2
 * [B,S2] as for mt_precompute_ctx; workspace as mt_precompute_ctx needs for S2).
 * mt_decoder_step_dual: mt_decoder_step plus the second source: s1 also queries it (q2 =
 * s1 Wa2, va2, masked softmax over its S2 positions), and GRU 2 and the readout take the
 * two contexts side by side.  attn_out holds the first source's weights.  The start state
 * comes from the first source (mt_precompute_ctx).  mt_decoder_step on a dual-source
 * model (and these calls on another) return MT_ERR_STATE. */
mt_status mt_precompute_keys2(mt_model *model, int B, int S2, const void *ctx2, const float *mask2,
                              void *pctx2_out, void *ws, size_t ws_bytes, void *stream);
mt_status mt_decoder_step_dual(mt_model *model, int B, int K, int S, const int32_t *prev_tok,
                               const int32_t *src_row, int n_state_rows, const float *state_in,
                               const void *ctx, const void *pctx, const float *mask, int S2, const void *ctx2,
                               const void *pctx2, const float *mask2, float *state_out, float *logp_out,
                               float *attn_out, const mt_taps *taps, void *ws, size_t ws_bytes, void *stream);

/* Beam selection (Section 2.2: next hypotheses from the decoder state;
 * Section 2.3: batched beam search).  For sentence b the candidates are
 * cand(k,v) = prev_score[b*K+k] + logp[b*K+k, v], summed in fp32; the K best
 * by (cand descending, k*V + v ascending) are written as
 *   score_out[b*K+j] = cand, tok_out[b*K+j] = v, bp_out[b*K+j] = k,
 *   row_out[b*K+j] = b*K + k (NULL allowed) — the next step's src_row.
 * logp: [M,V] fp32 from any source, or NULL to use the candidates that the
 * preceding mt_decoder_step (same B, K, workspace) left in the workspace.
 * prev_score may alias score_out. */
mt_status mt_beam_topk(mt_model *model, int B, int K, const float *prev_score, const float *logp,
                       float *score_out, int32_t *tok_out, int32_t *bp_out, int32_t *row_out,
                       void *ws, size_t ws_bytes, void *stream);

/* Ensemble of n models decoding the same beams (Section 2.3: ensembling of models as a
 * meta-algorithm of batched beam search).  Each member runs its own mt_decoder_step on the
 * shared tokens and state rows (its own states) with logp_out given; this call combines
 * their log-probabilities for one mt_beam_topk (pass out as its logp):
 *   out[m, v] = sum_i weights[i] * logp[i][m, v],  m < M = B*K, v < V,
 * members summed in order, fp32.  logp: HOST array of n device pointers to fp32 [M, V]
 * (16-byte aligned); weights: HOST array of n finite floats; out: device fp32 [M, V],
 * may be one of the inputs.  model: any member (V = its vocabulary; profiling slot
 * MT_KERNEL_ENSEMBLE).  1 <= n <= 8.  Asynchronous on the stream. */
mt_status mt_ensemble_logp(mt_model *model, int n, const float *const *logp, const float *weights, int M,
                           float *out, void *stream);

/* Fused ensemble step (Section 2.3: ensembling inside batched beam search).  The combined
 * log-probability sum_i w_i logp_i(v) = sum_i w_i logit_i(v) - C, with C = sum_i w_i LSE_i a
 * per-row constant, so the members never materialise their log-probabilities:
 *   mt_ensemble_step: member `member` of n_members (called for 0, 1, ... in order) runs its
 *     decoder step (mt_decoder_step's arguments and state outputs) and writes weight * its
 *     logits (t Wo + bo) into comb_logits [B*K, V] fp32 device memory (member 0 stores, later
 *     members add, fp32, in member order); its log-sum-exp partials stay in its workspace ws.
 *     The last member (member = n_members - 1) also collects the beam candidates, on the
 *     combined values it stores; the others skip the candidate threshold.  weight finite and
 *     nonzero; 1 <= n_members <= 8; not for dual-source models (MT_ERR_STATE).
 *   mt_ensemble_topk: C[m] = sum_i weights[i] * LSE_i[m] (from the partials each member's
 *     mt_ensemble_step left in ws[i], which must be that call's workspace, of ws_bytes[i], and
 *     weights[i] that call's weight), then the beam selection of mt_beam_topk on the keys
 *     (prev_score - C) + comb_logits, from the last member's candidates (a row whose
 *     candidates overflow is selected from comb_logits): score_out = prev_score + sum_i w_i
 *     logp_i up to rounding.  models, weights, ws, ws_bytes: HOST arrays of the n members
 *     (same V, k_max >= K); row_const_out [B*K] or NULL receives C.  The selection's scratch
 *     lives in ws[n-1].  MT_ERR_STATE unless the members' last calls were exactly these
 *     ensemble steps.  1 <= n <= 8.  Asynchronous. */
/* Joint vocabulary pass (comb_logits = NULL in both calls): the members' steps stop after the
 * readout and the threshold sample, and mt_ensemble_topk runs one vocabulary kernel for all
 * members, which keeps every member's readout activations resident, forms the combined value
 * sum_i w_i logit_i(v) of each entry in registers and collects the beam candidates on it (a
 * row whose candidates overflow is recomputed from the members' weights); no [B*K, V] buffer
 * is written.  mt_ensemble_step fails with MT_ERR_SHAPE where the pass does not support the
 * member (see mt_ensemble_joint_ok). */
mt_status mt_ensemble_step(mt_model *model, int member, int n_members, float weight, int B, int K, int S,
                           const int32_t *prev_tok, const int32_t *src_row, int n_state_rows, const float *state_in,
                           const void *ctx, const void *pctx, const float *mask, float *state_out,
                           float *comb_logits, void *ws, size_t ws_bytes, void *stream);
mt_status mt_ensemble_topk(int n, mt_model *const *models, const float *weights, void *const *ws,
                           const size_t *ws_bytes, int B, int K, const float *prev_score, const float *comb_logits,
                           float *score_out, int32_t *tok_out, int32_t *bp_out, int32_t *row_out, float *row_const_out,
                           void *stream);
/* Recurrent-product operand reuse (bf16 models; Section 2.1: the step's fused kernels).  Every
 * step of a bf16 model leaves in its workspace the bf16 copy of state_out that the next
 * products read.  With on != 0, a step whose state_in is the state_out pointer of the
 * previous step on this model, with the same workspace and n_state_rows = that step's B*K,
 * gathers that copy for h U1 instead of rounding state_in again: the results are
 * bit-identical, PROVIDED the caller has not written to that state buffer since; a caller
 * that edits states between steps must leave this off (the default) for the step after the
 * edit.  Switching it does not forget the copy; any other call on the model (precompute,
 * encode, second-source keys) does.  fp32 models: no effect. */
mt_status mt_set_state_reuse(mt_model *model, int on);

/* 1 if the joint vocabulary pass supports these n members (2 <= n <= 4, single-source, equal V,
 * E and gemm dtype, the members' readout activations of one row block fitting one workgroup's
 * LDS together), else 0.  models: HOST array. */
int mt_ensemble_joint_ok(int n, mt_model *const *models);

/* Translation bookkeeping after mt_beam_topk of step `step` (batched beam search decoding
 * to an n-best list as large as the beam, Sections 2.3 and 3.1.3).  Per sentence b:
 *   beam[b] (device int32 [B], in/out): K minus the hypotheses b has finished (start: K);
 *   of b's K ranked results (tok, bp, row, score [B*K] as mt_beam_topk wrote them) the
 *   first beam[b] with a finite score are its new hypotheses.  Those whose token is eos
 *   (every one when final != 0) finish: entry fin_count[b] (+ rank among them) of b's list
 *   receives fin_score = score, fin_norm = score / (step+1)^alpha, fin_step = step,
 *   fin_parent = bp (slot in the previous beam), fin_tok = token; beam[b] shrinks by one
 *   each and fin_count[b] (device int32 [B], start 0) grows.  The other new hypotheses
 *   move, in rank order, to slots 0.. of tok/bp/row/score (in place); the remaining slots
 *   become dead (score -inf, token eos, bp 0, row b*K) and never extend.
 *   hist_tok, hist_bp (device int32 [B*K]) receive this step's compacted tok and bp, the
 *   record a caller backtracks through (finished entry -> fin_parent -> hist_* of the
 *   previous steps).
 *   fin_score, fin_norm [B*K] fp32, fin_step, fin_parent, fin_tok [B*K] int32: b's list at
 *   b*K..b*K+K-1 (at most K entries ever).
 * 1 <= K <= k_max, 0 <= eos < V, alpha finite.  Asynchronous on the stream. */
mt_status mt_beam_finish(mt_model *model, int B, int K, int step, int32_t eos, float alpha, int final_step,
                         int32_t *tok, int32_t *bp, int32_t *row, float *score, int32_t *beam,
                         int32_t *fin_count, int32_t *hist_tok, int32_t *hist_bp, float *fin_score,
                         float *fin_norm, int32_t *fin_step, int32_t *fin_parent, int32_t *fin_tok, void *stream);

/* The n-best lists of a finished translation batch from mt_beam_finish's records (decoding to
 * an n-best list as large as the beam, Sections 2.3 and 3.1.3), on the device.  Per sentence b
 * with fc = min(fin_count[b], K) finished entries (b*K + e, e < fc, as mt_beam_finish wrote
 * them):
 *   order[b*K + r] = the entry e of rank r (fin_norm descending, equal values by smaller e),
 *     -1 for r >= fc;
 *   seq[(b*K + r) * ld_seq + s] = token s of that hypothesis for s <= its fin_step (the last is
 *     its fin_tok, the earlier ones read back through hist_tok / hist_bp of steps fin_step-1 ..
 *     0, starting from fin_parent), -1 after it and in rows of unused ranks.
 * hist_tok, hist_bp: device int32 [steps][B*K], the records of steps 0 .. steps-1; fin_*: as
 * mt_beam_finish left them; order [B*K], seq [B*K][ld_seq] device int32, ld_seq >= steps.
 * 1 <= K <= 16.  Asynchronous on the stream. */
mt_status mt_beam_nbest(mt_model *model, int B, int K, int steps, const int32_t *hist_tok, const int32_t *hist_bp,
                        const int32_t *fin_count, const float *fin_norm, const int32_t *fin_step,
                        const int32_t *fin_parent, const int32_t *fin_tok, int32_t *order, int32_t *seq, int ld_seq,
                        void *stream);

/* Reads and clears the device-side error bits (synchronises the device):
 * bit 0 = a prev_tok out of range, bit 1 = a src_row out of range, bit 3 = a source token of
 * mt_encode out of range. */
mt_status mt_device_errors(mt_model *model, int32_t *flags);

/* Reads and clears (synchronises the device) the number of hypothesis rows that mt_beam_topk,
 * selecting from the candidates its preceding mt_decoder_step left in the workspace (logp =
 * NULL), recomputed exactly from the weights because their candidates did not fit the
 * workspace lists (or fell short of K), since the last call.  A diagnostic of the fused
 * selection (Section 2.3, batched beam search): the result is exact either way. */
mt_status mt_recomputed_rows(mt_model *model, int64_t *rows);

/* Kernel timing with HIP events recorded on the launch stream around each
 * launch of the selected kernel classes (bit k of kernel_mask selects
 * mt_kernel_id k; 0 turns timing off, the default; each timed launch costs
 * two event records).  mt_profile_query synchronises and returns the summed
 * duration in milliseconds and the number of timed launches since the last
 * reset. */
typedef enum {
  MT_KERNEL_GEMM_GRU1 = 0,  /* h U1 (the token side is a precomputed table) */
  MT_KERNEL_GRU_CELL = 1,   /* both GRU elementwise kernels */
  MT_KERNEL_GEMM_S1 = 2,    /* s1 [Wa|U2] */
  MT_KERNEL_ATTENTION = 3,
  MT_KERNEL_GEMM_CTX = 4,   /* c [W2|Wt_c] */
  MT_KERNEL_GEMM_READOUT = 5, /* s Wt_s */
  MT_KERNEL_READOUT = 6,    /* sum + LN + tanh */
  MT_KERNEL_VOCAB_GEMM = 7, /* t Wo + bo with fused LSE partials and beam candidates */
  MT_KERNEL_LSE = 8,        /* logits -> log-probabilities (only when logp_out is given) */
  MT_KERNEL_TOPK = 9,       /* all top-K kernels (row log-sum-exp merge included) */
  MT_KERNEL_PRECOMPUTE = 10,
  MT_KERNEL_VOCAB_THRESHOLD = 11, /* logits of the first vocabulary entries -> candidate threshold */
  MT_KERNEL_GEMM_TRANSITION = 12, /* s Ut_j of the transition blocks (dec_transitions > 0) */
  MT_KERNEL_ENSEMBLE = 13,  /* mt_ensemble_logp; the row constant of mt_ensemble_topk */
  MT_KERNEL_BEAM_FINISH = 14, /* mt_beam_finish */
  MT_KERNEL_ENCODE = 15,    /* every kernel of mt_encode */
  MT_KERNEL_COUNT = 16
} mt_kernel_id;

mt_status mt_profile_enable(mt_model *model, uint32_t kernel_mask);
/* Times one launch in `every` (>= 1, default 1) of each selected class, the first after a
 * reset included: an event record makes the stream wait for the work before it, which adds
 * a few microseconds around a timed launch, so sampling keeps a timed run's step time
 * representative while the average over the timed launches stays the class's. */
mt_status mt_profile_sample(mt_model *model, uint32_t every);
mt_status mt_profile_reset(mt_model *model);
mt_status mt_profile_query(mt_model *model, int kernel, double *total_ms, int64_t *launches);

/* The fp32 -> bf16 conversion that mt_load_weights applies to every matrix of a bf16 model
 * (gemm_dtype = MT_BF16): dst[i] = the bf16 bit pattern nearest to src[i], ties to even; a NaN
 * stays a quiet NaN, +-inf stay infinite, a value rounding past the largest finite bf16
 * becomes +-inf.  HOST pointers; needs no device; n = 0 or a NULL pointer does nothing. */
void mt_round_bf16(const float *src, uint16_t *dst, size_t n);

/* Message of the last failed call on this thread ("" if none). */
const char *mt_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
