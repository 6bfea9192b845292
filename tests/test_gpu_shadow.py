"""GPU path against the oracle at the inputs the benchmark times and over whole decodes.

* one step at the benchmark's own weights (zero output bias) at every workload size;
* bf16 models loaded from fp32 master weights and an unrounded context, so the library's own
  fp32 -> bf16 conversion is part of what is compared;
* shadow decodes: the whole fixed-step decode of a workload (start state, step 0 from it,
  then every step from the GPU's own beam) with the production configuration (no
  log-probabilities written: the selection works from the vocabulary pass's candidates); at
  every step the oracle takes the GPU step's inputs for the sampled sentences (tokens, state
  rows, previous state, scores) and its outputs are compared: new states, and the selected
  scores, tokens and backpointers under the gap rule.  Errors never accumulate and diverging
  beam decisions cannot desynchronise the comparison (the decode loop of Decoder::startState,
  Decoder::step and the selection of the next hypotheses, Sections 2.2 and 2.3).
"""
import concurrent.futures as cf
import sys

import numpy as np
import pytest

from oracle import mtref
from paper_1804_00344_amd import synth
from tests.parity_util import TOL, maxerr, oracle_model, oracle_sentences, sample_sentences, topk_gap_check

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU-only machines
    pytestmark = [pytest.mark.gpu, pytest.mark.skip(reason="no GPU")]
else:
    from paper_1804_00344_amd.runner import Decoder, Ensemble
    from paper_1804_00344_amd import mtstep as mt

DEV = "cuda:0"


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def T(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def check_step(p, dec, w, ctx, mask, lens, tok, src, state, nrows, score, n_sent, label, start=False):
    """One step with log-probabilities, then the fused selection and the candidates-only
    (production) step + selection, all against the oracle on sampled sentences."""
    M = p.M
    st_in = T(state)
    out_s = torch.empty((M, p.H), device=DEV)
    logp = torch.empty((M, p.V), device=DEV)
    dec.step(T(tok), T(src), st_in, nrows, out_s, logp=logp)
    sc, tk, bp, rw = [x.cpu().numpy() for x in dec.topk(T(score), None)]
    g_state, g_logp = out_s.cpu().numpy(), logp.cpu().numpy()
    mt.mt_recomputed_rows(dec.model)
    out_p = torch.empty((M, p.H), device=DEV)
    dec.step(T(tok), T(src), st_in, nrows, out_p)
    sc2, tk2, bp2, rw2 = [x.clone().cpu().numpy() for x in dec.topk(T(score), None)]
    torch.cuda.synchronize()
    n_rec = mt.mt_recomputed_rows(dec.model)
    assert mt.mt_device_errors(dec.model) == 0
    assert torch.equal(out_p, out_s)
    sents = sample_sentences(lens, n_sent)
    orc = oracle_sentences(oracle_model(p, w), p.K, sents, ctx, mask, tok, src, state, want_alpha=False,
                           taps=False, start="given" if start else False)
    tol = TOL[p.gemm]
    es = el = 0.0
    dec_n = tot = 0
    for b in sents:
        rows = slice(b * p.K, (b + 1) * p.K)
        es = max(es, maxerr(g_state[rows], orc[b]["state"]))
        el = max(el, maxerr(g_logp[rows], orc[b]["logp"]))
        for S_, T_, B_, R_ in ((sc, tk, bp, rw), (sc2, tk2, bp2, rw2)):
            d, n = topk_gap_check(p.K, score[rows], orc[b]["logp"], S_[rows], T_[rows], B_[rows], tol["logp"])
            assert np.array_equal(R_[rows], b * p.K + B_[rows])
        dec_n += d
        tot += n
    log(f"[{label}] state err {es:.3g}, logp err {el:.3g}; decided slots {dec_n}/{tot}; "
        f"rows recomputed exactly by the candidates-only selection: {n_rec} of {M}")
    assert es <= tol["state"] and el <= tol["logp"], (label, es, el)
    return es, el


# ------------------------------------------------------------------------------------------
# the benchmark's weights (zero output bias): nearly flat logits, so the candidate threshold,
# the list fill and the exact-recomputation fallback see what the timed runs see
# ------------------------------------------------------------------------------------------

BENCH_SETS = {"tiny_f32": 99, "nematus_f32": 4, "nematus_bf16_ln": 4, "vocab85k_bf16_ln": 4, "greedy_bf16_ln": 16}


@pytest.mark.parametrize("name", list(BENCH_SETS))
def test_step_parity_benchmark_weights(name):
    p = synth.PRESETS[name]
    log(f"\n[bench weights] {name}")
    w = synth.make_weights(p)
    assert not np.any(w["bo"])
    ctx, mask, lens = synth.make_source(p)
    dec = Decoder.from_preset(p, w)
    dec.set_batch(ctx, mask, p.K)
    dec.precompute()
    tok, src, state, score = synth.mid_decode_inputs(p, salt=21)
    check_step(p, dec, w, ctx, mask, lens, tok, src, state, p.M, score, BENCH_SETS[name], f"{name} mid-decode")
    # step 0 from the start state (src_row = m // K into the B rows of s0)
    tok0, src0, score0 = synth.start_beam(p)
    s0 = dec.s0.cpu().numpy()
    check_step(p, dec, w, ctx, mask, lens, tok0, src0, s0, p.B, score0, BENCH_SETS[name], f"{name} step 0",
               start=True)


# ------------------------------------------------------------------------------------------
# bf16 models from fp32 masters: the library converts (round to nearest even) every matrix
# itself; the oracle takes the unrounded masters and the bf16 tolerance covers the rounding
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name,n_sent", [("tiny_bf16_ln", 99), ("nematus_bf16_ln", 4), ("vocab85k_bf16_ln", 4),
                                         ("greedy_bf16_ln", 16)])
def test_step_parity_fp32_masters(name, n_sent):
    p = synth.PRESETS[name]
    log(f"\n[fp32 masters] {name}")
    w = synth.make_weights(p, peaked_bias=True, round_operands=False)
    ctx, mask, lens = synth.make_source(p, round_operands=False)
    assert np.any(synth.round_bf16(w["Wo"]) != w["Wo"]) and np.any(synth.round_bf16(ctx) != ctx)
    dec = Decoder.from_preset(p, w)
    dec.set_batch(ctx, mask, p.K)   # the context is handed over in bf16 (torch's conversion)
    dec.precompute()
    tok, src, state, score = synth.mid_decode_inputs(p, salt=22)
    check_step(p, dec, w, ctx, mask, lens, tok, src, state, p.M, score, n_sent, f"{name} fp32 masters")


# ------------------------------------------------------------------------------------------
# shadow decodes over the workload's full step count
# ------------------------------------------------------------------------------------------

SHADOW = {"tiny_f32": 99, "nematus_f32": 4, "nematus_bf16_ln": 4, "vocab85k_bf16_ln": 4, "greedy_bf16_ln": 16}


@pytest.mark.parametrize("name", list(SHADOW))
def test_shadow_decode(name):
    p = synth.PRESETS[name]
    log(f"\n[shadow] {name}: {p.steps} steps, B={p.B} K={p.K}")
    w = synth.make_weights(p)          # the benchmark's weights
    ctx, mask, lens = synth.make_source(p)
    dec = Decoder.from_preset(p, w)
    dec.set_batch(ctx, mask, p.K)
    om = oracle_model(p, w)
    tol = TOL[p.gemm]
    sents = sample_sentences(lens, SHADOW[name])
    # the oracle's per-sentence keys and start state, once
    with cf.ThreadPoolExecutor(8) as ex:
        pre = dict(zip(sents, ex.map(lambda b: om.precompute(ctx[b:b + 1], mask[b:b + 1]), sents)))
    dec.precompute()
    tok0, src0, score0 = synth.start_beam(p)
    dec.start(tok0, score0)
    g_s0 = dec.s0.cpu().numpy()
    es0 = max(maxerr(g_s0[b], pre[b][1][0]) for b in sents)
    assert es0 <= (1e-4 if p.gemm == "f32" else 5e-2), es0
    worst_s = 0.0
    decided = slots = 0
    n_rec = 0
    for t in range(p.steps):
        # the step's inputs, as the GPU holds them
        g_tok, g_row, g_score = dec.tok.cpu().numpy(), dec.row.cpu().numpy(), dec.score.cpu().numpy()
        first = dec.first
        g_in = (dec.s0 if first else dec.state[dec.cur]).cpu().numpy()
        state = dec.advance()   # production configuration: candidates only
        s_out = state.cpu().numpy()
        n_sc, n_tk, n_bp, n_rw = [x.cpu().numpy() for x in (dec.score, dec.tok, dec.bp, dec.row)]
        n_rec += mt.mt_recomputed_rows(dec.model)

        def one(b):
            rows = slice(b * p.K, (b + 1) * p.K)
            if first:
                st, sr = g_in[b:b + 1], (g_row[rows] - b).astype(np.int32)
            else:
                st, sr = g_in[rows], (g_row[rows] - b * p.K).astype(np.int32)
            P = pre[b][0]
            return b, om.step(p.K, g_tok[rows], sr, st, ctx[b:b + 1], P, mask[b:b + 1])

        with cf.ThreadPoolExecutor(8) as ex:
            orc = dict(ex.map(one, sents))
        for b in sents:
            rows = slice(b * p.K, (b + 1) * p.K)
            e = maxerr(s_out[rows], orc[b]["state"])
            assert e <= tol["state"], (name, t, b, e)
            worst_s = max(worst_s, e)
            d, n = topk_gap_check(p.K, g_score[rows], orc[b]["logp"], n_sc[rows], n_tk[rows], n_bp[rows],
                                  tol["logp"])
            assert np.array_equal(n_rw[rows], b * p.K + n_bp[rows])
            decided += d
            slots += n
    assert mt.mt_device_errors(dec.model) == 0
    log(f"[shadow] {name}: {p.steps} steps x {len(sents)} sentences, start state err {es0:.3g}, largest state "
        f"err {worst_s:.3g}, decided slots {decided}/{slots}, rows recomputed exactly {n_rec}")


def test_shadow_step0_all_sentences():
    """Step 0 of the Nematus fp32 workload for every sentence of the batch (the shadow above
    samples four): the start state, the step from it and the first selection."""
    p = synth.PRESETS["nematus_f32"]
    w = synth.make_weights(p)
    ctx, mask, lens = synth.make_source(p)
    dec = Decoder.from_preset(p, w)
    dec.set_batch(ctx, mask, p.K)
    dec.precompute()
    tok0, src0, score0 = synth.start_beam(p)
    check_step(p, dec, w, ctx, mask, lens, tok0, src0, dec.s0.cpu().numpy(), p.B, score0, p.B,
               "nematus_f32 step 0, all sentences", start=True)


# ------------------------------------------------------------------------------------------
# ensembles decoding from source tokens (each member encodes with its own encoder)
# ------------------------------------------------------------------------------------------

def test_ensemble_from_source_tokens():
    p = synth.PRESETS["tiny_f32"]
    src_V = 200
    members, decs = [], []
    _, mask, lens = synth.make_source(p)
    src = synth.source_tokens(p, src_V, lens, mask.shape[1])
    for i in range(2):
        q = synth.with_sizes(p, index=p.index + 100 * i, name=f"tiny_f32_m{i}")
        w = {**synth.make_weights(q, peaked_bias=True), **synth.make_encoder_weights(q, src_V)}
        members.append((q, w))
        decs.append(Decoder(q.E, q.H, q.A, q.V, w, k_max=q.K, src_V=src_V))
    ens = Ensemble(decs, [0.6, 0.4], joint=False)   # the per-member pass keeps the combined buffer
    ens.set_source(src, mask, p.K)
    ens.precompute()
    tok0, _, score0 = synth.start_beam(p)
    ens.start(tok0, score0)
    row_const = torch.empty(p.M, dtype=torch.float32, device="cuda")
    ens.advance(row_const=row_const)
    torch.cuda.synchronize()
    # the fused step leaves sum_i w_i logit_i; the combined logp is that minus the row constant
    g = ens.comb.cpu().numpy().astype(np.float64) - row_const.cpu().numpy()[:, None]
    sc, tk, bp = ens.lead.score.cpu().numpy(), ens.lead.tok.cpu().numpy(), ens.lead.bp.cpu().numpy()
    lps = []
    for (q, w), d in zip(members, decs):
        ctx_o = mtref.encode(src, mask, *[w[k] for k in synth.ENCODER_NAMES])
        om = oracle_model(q, w)
        P, s0 = om.precompute(ctx_o, mask)
        lps.append(om.step(p.K, tok0, (np.arange(p.M) // p.K).astype(np.int32), s0, ctx_o, P, mask)["logp"])
    ref = mtref.ensemble_logp(lps, [0.6, 0.4])
    err = maxerr(g, ref)
    log(f"[ensemble from source] combined logp error {err:.3g}")
    assert err <= TOL["f32"]["logp"]
    for b in range(p.B):
        rows = slice(b * p.K, (b + 1) * p.K)
        topk_gap_check(p.K, score0[rows], ref[rows], sc[rows], tk[rows], bp[rows], TOL["f32"]["logp"])
