"""GPU path (libmtstep through its C ABI) against the CPU oracle on seeded inputs."""
import dataclasses
import math
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
    from paper_1804_00344_amd.runner import Decoder
    from paper_1804_00344_amd import mtstep as mt

DEV = "cuda:0"


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def T(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x)).to(DEV)
    return t if dtype is None else t.to(dtype)


_cache = {}


def setup(name, peaked=False, nan_padding=False):
    key = (name, peaked, nan_padding)
    if key not in _cache:
        p = synth.PRESETS[name]
        w = synth.make_weights(p, peaked_bias=peaked)
        ctx, mask, lens = synth.make_source(p, nan_padding=nan_padding)
        dec = Decoder.from_preset(p, w)
        dec.set_batch(ctx, mask, p.K)
        dec.precompute()
        _cache.clear()
        _cache[key] = (p, w, ctx, mask, lens, dec)
    return _cache[key]


def run_step(dec, p, tok, src, state, nrows, logp=True, attn=True, taps=True):
    M = p.M
    out = {"state": torch.empty((M, p.H), device=DEV)}
    if logp:
        out["logp"] = torch.empty((M, p.V), device=DEV)
    if attn:
        out["alpha"] = torch.empty((M, dec.S), device=DEV)
    tp = None
    if taps:
        tp = {"s1": torch.empty((M, p.H), device=DEV), "c": torch.empty((M, p.C), device=DEV),
              "t": torch.empty((M, p.E), device=DEV)}
        out.update(tp)
    dec.step(T(tok), T(src), state, nrows, out["state"], logp=out.get("logp"), attn=out.get("alpha"), taps=tp)
    return out


def compare_rows(p, gpu, orc, sents, tol, label):
    K = p.K
    errs = {}
    for b in sents:
        rows = slice(b * K, (b + 1) * K)
        o = orc[b]
        for k, tk in (("state", "state"), ("logp", "logp"), ("alpha", "alpha"), ("s1", "s1"), ("c", "c"), ("t", "t")):
            if tk not in gpu or k not in o:
                continue
            g = gpu[tk][rows].float().cpu().numpy()
            errs[k] = max(errs.get(k, 0.0), maxerr(g, o[k]))
        if "alpha" in gpu:
            a = gpu["alpha"][rows].cpu().numpy()
            L = int((o["alpha"][0] != 0).sum()) if o["alpha"].size else 0
            assert np.all(np.abs(a.sum(1) - 1.0) <= 1e-5), (label, b, a.sum(1))
    log(f"[{label}] max errors over sentences {sents[:8]}{'...' if len(sents) > 8 else ''}: "
        + ", ".join(f"{k}={v:.3g}" for k, v in errs.items()))
    assert errs["state"] <= tol["state"], (label, errs)
    if "logp" in errs:
        assert errs["logp"] <= tol["logp"], (label, errs)
    if "alpha" in errs:
        assert errs["alpha"] <= tol["alpha"], (label, errs)
    for k in ("s1", "c", "t"):
        if k in errs:
            assert errs[k] <= tol["tap"], (label, k, errs)
    return errs


def masked_alpha_zero(p, gpu_alpha, mask):
    a = gpu_alpha.cpu().numpy().reshape(p.B, p.K, -1)
    m = mask[:, None, :] == 0
    assert np.all(a[np.broadcast_to(m, a.shape)] == 0.0)


# ------------------------------------------------------------------------------------------
# one step from a synthetic mid-decode beam: every preset
# ------------------------------------------------------------------------------------------

N_SAMPLE = {"tiny_f32": 99, "tiny_bf16_ln": 99, "nematus_f32": 4, "nematus_bf16_ln": 4,
            "vocab85k_bf16_ln": 4, "greedy_bf16_ln": 16,
            # deep-transition cell: six recurrent-only GRU blocks after GRU 2
            "tiny_deep_f32_ln": 99, "deep_f32_ln": 3, "deep_bf16_ln": 3}


# Nematus fp32 dimensions at other batch shapes: the fp32 products then run on the tile shapes
# and k-splits that 64 x 12 rows never pick (3x2, 3x3 and 3x5 blocks split over two waves, 2x4
# blocks, 32-wide 1x2 tiles with and without a split), and on row counts that are not a multiple
# of any tile (296).
BATCH_SHAPES = [(16, 12), (37, 8), (80, 8)]


@pytest.mark.parametrize("B,K", BATCH_SHAPES)
def test_step_parity_other_batch_shapes(B, K):
    p = dataclasses.replace(synth.PRESETS["nematus_f32"], name=f"nematus_f32_B{B}_K{K}", B=B, K=K)
    log(f"\n[step parity] {p.name} (M={p.M})")
    w = synth.make_weights(p, peaked_bias=True)
    ctx, mask, lens = synth.make_source(p)
    dec = Decoder.from_preset(p, w)
    dec.set_batch(ctx, mask, p.K)
    dec.precompute()
    tok, src, state, score = synth.mid_decode_inputs(p, salt=3)
    gpu = run_step(dec, p, tok, src, T(state), p.M)
    sc, tk, bp, rw = [x.cpu().numpy() for x in dec.topk(T(score), None)]
    torch.cuda.synchronize()
    assert mt.mt_device_errors(dec.model) == 0
    sents = sample_sentences(lens, 3)
    orc = oracle_sentences(oracle_model(p, w), p.K, sents, ctx, mask, tok, src, state)
    tol = TOL[p.gemm]
    compare_rows(p, gpu, orc, sents, tol, p.name)
    for b in sents:
        rows = slice(b * p.K, (b + 1) * p.K)
        topk_gap_check(p.K, score[rows], orc[b]["logp"], sc[rows], tk[rows], bp[rows], tol["logp"])
        assert np.array_equal(rw[rows], b * p.K + bp[rows])


# V = 1056 is 33 vocabulary blocks of 32 rows: the runs of the vocabulary pass are one or two
# blocks long, so most of them end with a single-block tile, the last one at the end of the range
@pytest.mark.parametrize("name", ["tiny_f32", "tiny_bf16_ln"])
def test_step_parity_single_block_vocab_tiles(name):
    p = dataclasses.replace(synth.PRESETS[name], name=f"{name}_V1056", V=1056)
    log(f"\n[step parity] {p.name} (M={p.M})")
    w = synth.make_weights(p, peaked_bias=True)
    ctx, mask, lens = synth.make_source(p)
    dec = Decoder.from_preset(p, w)
    dec.set_batch(ctx, mask, p.K)
    dec.precompute()
    tok, src, state, score = synth.mid_decode_inputs(p, salt=4)
    gpu = run_step(dec, p, tok, src, T(state), p.M)
    sc, tk, bp, rw = [x.cpu().numpy() for x in dec.topk(T(score), None)]
    torch.cuda.synchronize()
    assert mt.mt_device_errors(dec.model) == 0
    sents = sample_sentences(lens, 3)
    orc = oracle_sentences(oracle_model(p, w), p.K, sents, ctx, mask, tok, src, state)
    tol = TOL[p.gemm]
    compare_rows(p, gpu, orc, sents, tol, p.name)
    for b in sents:
        rows = slice(b * p.K, (b + 1) * p.K)
        topk_gap_check(p.K, score[rows], orc[b]["logp"], sc[rows], tk[rows], bp[rows], tol["logp"])
        assert np.array_equal(rw[rows], b * p.K + bp[rows])


@pytest.mark.parametrize("name", list(N_SAMPLE))
def test_step_parity_mid_decode(name):
    log(f"\n[step parity] preset={name}")
    p, w, ctx, mask, lens, dec = setup(name, peaked=True)
    tok, src, state, score = synth.mid_decode_inputs(p, salt=1)
    gpu = run_step(dec, p, tok, src, T(state), p.M)
    # fused top-K (candidates from the vocabulary GEMM epilogue)
    sc, tk, bp, rw = [x.cpu().numpy() for x in dec.topk(T(score), None)]
    # materialised top-K on the GPU's own log-probs
    sc2, tk2, bp2, _ = [x.cpu().numpy() for x in dec.topk(T(score), gpu["logp"], score_out=torch.empty_like(dec.score),
                                                          tok_out=torch.empty_like(dec.tok), bp_out=torch.empty_like(dec.bp),
                                                          row_out=torch.empty_like(dec.row))]
    torch.cuda.synchronize()
    assert mt.mt_device_errors(dec.model) == 0
    sents = sample_sentences(lens, N_SAMPLE[name])
    orc = oracle_sentences(oracle_model(p, w), p.K, sents, ctx, mask, tok, src, state)
    tol = TOL[p.gemm]
    compare_rows(p, gpu, orc, sents, tol, name)
    masked_alpha_zero(p, gpu["alpha"], mask)
    dec_slots = tot = 0
    for b in sents:
        rows = slice(b * p.K, (b + 1) * p.K)
        d, n = topk_gap_check(p.K, score[rows], orc[b]["logp"], sc[rows], tk[rows], bp[rows], tol["logp"])
        dec_slots += d
        tot += n
        assert np.array_equal(rw[rows], b * p.K + bp[rows])
    log(f"[{name}] top-K decided slots {dec_slots}/{tot}")
    # the materialised path is an exact sort of the GPU's own log-probs
    lp = gpu["logp"].cpu().numpy()
    t3, b3, s3 = mtref.topk(p.K, score, lp)
    assert np.array_equal(tk2, t3) and np.array_equal(bp2, b3) and np.array_equal(sc2, s3)
    # fused and materialised selections agree exactly: the GPU's keys are computed identically
    # (same log-sum-exp merge, same fp32 additions) and both levels break ties by flat index
    assert np.array_equal(sc, sc2) and np.array_equal(tk, tk2) and np.array_equal(bp, bp2)
    # the production configuration: no log-probs, attention or taps written (the vocabulary
    # pass then runs its candidates-only kernel)
    run_step(dec, p, tok, src, T(state), p.M, logp=False, attn=False, taps=False)
    sc4, tk4, bp4, rw4 = [x.cpu().numpy() for x in dec.topk(T(score), None, score_out=torch.empty_like(dec.score),
                                                            tok_out=torch.empty_like(dec.tok),
                                                            bp_out=torch.empty_like(dec.bp),
                                                            row_out=torch.empty_like(dec.row))]
    torch.cuda.synchronize()
    assert mt.mt_device_errors(dec.model) == 0
    dec_slots = 0
    for b in sents:
        rows = slice(b * p.K, (b + 1) * p.K)
        d, _ = topk_gap_check(p.K, score[rows], orc[b]["logp"], sc4[rows], tk4[rows], bp4[rows], tol["logp"])
        dec_slots += d
        assert np.array_equal(rw4[rows], b * p.K + bp4[rows])
    assert np.all(np.abs(sc4.astype(np.float64) - sc.astype(np.float64)) <= 2 * tol["logp"])
    same = np.mean((tk4 == tk) & (bp4 == bp))
    log(f"[{name}] candidates-only pass: decided slots {dec_slots}/{tot}, agreement with the logits pass {same:.4f}")


@pytest.mark.parametrize("name", list(N_SAMPLE))
def test_precompute_parity(name):
    log(f"\n[precompute parity] preset={name}")
    p, w, ctx, mask, lens, dec = setup(name, peaked=True)
    dec.precompute()
    P = dec.pctx.float().cpu().numpy()
    s0 = dec.s0.cpu().numpy()
    sents = sample_sentences(lens, N_SAMPLE[name])
    om = oracle_model(p, w)
    tol = 1e-4 if p.gemm == "f32" else 5e-2
    eP = es = 0.0
    for b in sents:
        Po, so = om.precompute(ctx[b:b + 1], mask[b:b + 1])
        L = int(lens[b])
        eP = max(eP, maxerr(P[b, :L], Po[0, :L]))
        es = max(es, maxerr(s0[b], so[0]))
    log(f"[{name}] P err {eP:.3g}  s0 err {es:.3g}")
    assert eP <= tol and es <= tol


# ------------------------------------------------------------------------------------------
# beam-search trajectories on the tiny preset: GPU and oracle run their own beams from the
# same start; each sentence is compared until its first undecided (near-tie) selection
# ------------------------------------------------------------------------------------------

# Anchored: every step the oracle continues from the GPU's beam (state, tokens, backpointers,
# scores), so each step is compared from identical inputs with the per-step tolerances, and
# errors never accumulate (with random weights a recurrent cell can amplify a state difference
# from step to step, so two free-running trajectories drift apart whatever the arithmetic).
# Every sentence is compared at every step; where a selection is undecided (a near-tie) the
# gap rule checks that the GPU's pick is a valid one.
@pytest.mark.parametrize("name", ["tiny_f32", "tiny_bf16_ln", "tiny_deep_f32_ln"])
def test_tiny_trajectory(name):
    log(f"\n[trajectory] preset={name}")
    p, w, ctx, mask, lens, dec = setup(name, peaked=True)
    tol = TOL[p.gemm]
    om = oracle_model(p, w)
    Po, _ = om.precompute(ctx, mask)
    tok0, src0, score0 = synth.start_beam(p)
    dec.precompute()
    dec.start(tok0, score0)
    # step 0 reads the GPU's start state too (its own parity is checked by the precompute test)
    o_tok, o_src, o_state, o_score = tok0.copy(), src0.copy(), dec.s0.cpu().numpy(), score0.copy()
    logp = torch.empty((p.M, p.V), device=DEV)
    worst_state = worst_logp = 0.0
    decided = slots = agree = 0
    for t in range(p.steps):
        state = dec.advance(logp=logp)
        g_score, g_tok, g_bp, g_row = [x.cpu().numpy() for x in (dec.score, dec.tok, dec.bp, dec.row)]
        g_state = state.cpu().numpy()
        g_logp = logp.cpu().numpy()
        out = om.step(p.K, o_tok, o_src, o_state, ctx, Po, mask)
        n_tok, n_bp, _ = mtref.topk(p.K, o_score, out["logp"])
        for b in range(p.B):
            rows = slice(b * p.K, (b + 1) * p.K)
            d, n = topk_gap_check(p.K, o_score[rows], out["logp"][rows], g_score[rows], g_tok[rows], g_bp[rows],
                                  tol["logp"])
            decided += d
            slots += n
            agree += int(np.array_equal(g_tok[rows], n_tok[rows]) and np.array_equal(g_bp[rows], n_bp[rows]))
        # the new states (state_out rows, before reordering) and log-probabilities, both sides from
        # the same inputs
        es, el = maxerr(g_state, out["state"]), maxerr(g_logp, out["logp"])
        assert es <= tol["state"] and el <= tol["logp"], (name, t, es, el)
        worst_state, worst_logp = max(worst_state, es), max(worst_logp, el)
        assert np.array_equal(g_row, (np.arange(p.M) // p.K) * p.K + g_bp)
        # the oracle continues from the GPU's beam
        o_tok, o_bp, o_score = g_tok.copy(), g_bp.copy(), g_score.copy()
        o_state = g_state.copy()
        o_src = ((np.arange(p.M) // p.K) * p.K + o_bp).astype(np.int32)
    log(f"[{name}] {p.steps} steps x {p.B} sentences: largest state error {worst_state:.3g}, logp {worst_logp:.3g}; "
        f"decided slots {decided}/{slots}; sentence-steps with identical selections {agree}/{p.steps * p.B}")


# ------------------------------------------------------------------------------------------
# top-K on given log-probabilities: bit-exact against the oracle's full sort
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("K,V", [(1, 16), (2, 7), (3, 1000), (5, 85000), (12, 50000), (16, 50000), (16, 16), (4, 2049),
                                 (2, 300000)])
def test_topk_given_logp_bit_exact(K, V):
    """V = 300000 makes the first level's chunks longer than its register-resident size."""
    log(f"\n[topk] K={K} V={V}")
    B = 6
    rng = np.random.default_rng(K * 1000 + V)
    p = synth.with_sizes(synth.PRESETS["tiny_f32"], V=max(V, 16), K=K, B=B)
    w = synth.make_weights(p)
    dec = Decoder(p.E, p.H, p.A, p.V, w, k_max=16)
    ctx, mask, _ = synth.make_source(p)
    dec.set_batch(ctx, mask, K)
    # heavy ties: values from a small set, plus some -inf scores
    logp = rng.choice(np.array([-1.0, -2.0, -2.5, -3.0, -7.25], np.float32), size=(B * K, p.V))
    logp[:, ::7] += rng.standard_normal((B * K, len(range(0, p.V, 7)))).astype(np.float32)
    score = rng.choice(np.array([0.0, -0.5, -1.0], np.float32), size=B * K)
    score[1] = -np.inf
    g = [x.cpu().numpy() for x in dec.topk(T(score), T(logp))]
    t, b, s = mtref.topk(K, score, logp)
    assert np.array_equal(g[1], t) and np.array_equal(g[2], b) and np.array_equal(g[0], s)
    assert np.array_equal(g[3], (np.arange(B * K) // K) * K + b)


# ------------------------------------------------------------------------------------------
# properties
# ------------------------------------------------------------------------------------------

def test_determinism_and_nan_padding():
    log("\n[determinism / NaN padding] nematus_bf16_ln")
    p, w, ctx, mask, lens, dec = setup("nematus_bf16_ln", peaked=True)
    tok, src, state, score = synth.mid_decode_inputs(p, salt=2)
    dec.precompute()
    outs = []
    for _ in range(3):
        o = run_step(dec, p, tok, src, T(state), p.M, taps=False)
        s = [x.clone() for x in dec.topk(T(score), None)]
        torch.cuda.synchronize()
        outs.append((o, s))
    for o, s in outs[1:]:
        for k in o:
            assert torch.equal(o[k], outs[0][0][k]), k
        for a, b in zip(s, outs[0][1]):
            assert torch.equal(a, b)
    # same inputs with NaN in every padded position of the context: nothing changes
    ctx_nan = ctx.copy()
    ctx_nan[mask == 0] = np.nan
    dec.set_batch(ctx_nan, mask, p.K)
    dec.precompute()
    o = run_step(dec, p, tok, src, T(state), p.M, taps=False)
    s = dec.topk(T(score), None)
    torch.cuda.synchronize()
    for k in o:
        assert torch.equal(o[k], outs[0][0][k]), k
    for a, b in zip(s, outs[0][1]):
        assert torch.equal(a, b)
    assert torch.isfinite(dec.s0).all()
    _cache.clear()


def test_out_of_range_indices_are_clamped_and_flagged():
    p, w, ctx, mask, lens, dec = setup("tiny_f32")
    tok, src, state, score = synth.mid_decode_inputs(p, salt=3)
    assert mt.mt_device_errors(dec.model) == 0
    bad_tok = tok.copy()
    bad_tok[3] = p.V + 5
    run_step(dec, p, bad_tok, src, T(state), p.M, taps=False)
    assert mt.mt_device_errors(dec.model) == 1
    bad_src = src.copy()
    bad_src[0] = -2
    run_step(dec, p, tok, bad_src, T(state), p.M, taps=False)
    assert mt.mt_device_errors(dec.model) == 2
    assert mt.mt_device_errors(dec.model) == 0


def test_abi_errors_on_gpu():
    p, w, ctx, mask, lens, dec = setup("tiny_f32")
    tok, src, state, score = synth.mid_decode_inputs(p, salt=4)
    st = T(state)
    out = torch.empty((p.M, p.H), device=DEV)
    small = torch.empty(256, dtype=torch.uint8, device=DEV)
    with pytest.raises(mt.MtError) as e:
        mt.mt_decoder_step(dec.model, p.B, p.K, dec.S, T(tok), T(src), p.M, st, dec.ctx, dec.pctx, dec.mask, out,
                           ws=small)
    assert e.value.status == mt.MT_ERR_WORKSPACE
    with pytest.raises(mt.MtError) as e:
        mt.mt_decoder_step(dec.model, p.B, p.K, dec.S, T(tok), T(src), p.M, st, dec.ctx, dec.pctx, dec.mask, st,
                           ws=dec.ws)
    assert e.value.status == mt.MT_ERR_ARG  # state_out aliases state_in
    with pytest.raises(mt.MtError) as e:
        mt.mt_decoder_step(dec.model, p.B, p.K + 1, dec.S, T(tok), T(src), p.M, st, dec.ctx, dec.pctx, dec.mask,
                           out, ws=dec.ws)
    assert e.value.status == mt.MT_ERR_SHAPE  # K > k_max
    # top-K from the workspace with a different workspace than the step's
    ws2 = torch.empty_like(dec.ws)
    with pytest.raises(mt.MtError) as e:
        mt.mt_beam_topk(dec.model, p.B, p.K, T(score), None, dec.score, dec.tok, dec.bp, dec.row, ws=ws2)
    assert e.value.status == mt.MT_ERR_STATE
    misaligned = dec.ws[1:]
    with pytest.raises(mt.MtError) as e:
        mt.mt_decoder_step(dec.model, p.B, p.K, dec.S, T(tok), T(src), p.M, st, dec.ctx, dec.pctx, dec.mask, out,
                           ws=misaligned)
    assert e.value.status == mt.MT_ERR_ARG


def test_candidate_buffer_overflow_falls_back_exactly():
    """A bias that makes the first vocabulary entries (the threshold sample, 2048 entries) very
    unlikely puts the candidate threshold far below the rest of the vocabulary, so the
    candidate buffers overflow; the row selection must then recompute the rows and still
    select exactly.  The recomputation sums each logit in another order than the matrix
    cores, so its scores match the materialised path to rounding, and its tokens exactly."""
    log("\n[overflow fallback]")
    p = synth.with_sizes(synth.PRESETS["tiny_f32"], V=85000, K=4, B=2)
    w = synth.make_weights(p)
    w["bo"] = np.zeros(p.V, np.float32)
    w["bo"][:2048] = -50.0
    dec = Decoder.from_preset(p, w)
    ctx, mask, lens = synth.make_source(p)
    dec.set_batch(ctx, mask, p.K)
    dec.precompute()
    tok, src, state, score = synth.mid_decode_inputs(p, salt=5)
    gpu = run_step(dec, p, tok, src, T(state), p.M, attn=False, taps=False)
    sc, tk, bp, _ = [x.cpu().numpy() for x in dec.topk(T(score), None)]
    lp = gpu["logp"].cpu().numpy()
    t2, b2, s2 = mtref.topk(p.K, score, lp)
    assert np.array_equal(tk, t2) and np.array_equal(bp, b2)
    assert np.all(np.abs(sc.astype(np.float64) - s2) <= 1e-5 * (1.0 + np.abs(s2)))
    orc = oracle_sentences(oracle_model(p, w), p.K, [0, 1], ctx, mask, tok, src, state, want_alpha=False, taps=False)
    for b in (0, 1):
        rows = slice(b * p.K, (b + 1) * p.K)
        assert maxerr(lp[rows], orc[b]["logp"]) <= 1e-3


@pytest.mark.parametrize("name", ["tiny_f32", "tiny_bf16_ln"])
def test_equal_logits_overflow_in_sentence_selection(name):
    """A zero output layer makes every logit of a row equal, so every vocabulary entry is a
    candidate: the row's candidates exceed what one wave stages and the selection must fall back
    to the exact recomputation.  At V = 2000 a row has at most 64 candidate lists, so the
    selection runs one workgroup per sentence, whose fallback is the row's own wave.  Equal keys
    rank by flat index: the K best of a sentence are the smallest tokens of its best previous
    hypotheses, checked against the oracle's brute-force top-K of the GPU's log-probabilities."""
    log(f"\n[equal-logit overflow] {name}")
    p = synth.with_sizes(synth.PRESETS[name], V=2000, K=4, B=2)
    w = synth.make_weights(p)
    w["Wo"] = np.zeros_like(w["Wo"])
    w["bo"] = np.zeros(p.V, np.float32)
    dec = Decoder.from_preset(p, w)
    ctx, mask, lens = synth.make_source(p)
    dec.set_batch(ctx, mask, p.K)
    dec.precompute()
    tok, src, state, score = synth.mid_decode_inputs(p, salt=7)
    mt.mt_recomputed_rows(dec.model)  # (the count restarts at every read)
    gpu = run_step(dec, p, tok, src, T(state), p.M, attn=False, taps=False)
    sc, tk, bp, _ = [x.cpu().numpy() for x in dec.topk(T(score), None)]
    assert mt.mt_recomputed_rows(dec.model) == p.M  # every row fell back
    lp = gpu["logp"].cpu().numpy()
    assert np.all(lp == lp[:, :1])
    t2, b2, s2 = mtref.topk(p.K, score, lp)
    assert np.array_equal(tk, t2) and np.array_equal(bp, b2)
    assert np.all(np.abs(sc.astype(np.float64) - s2) <= 1e-5 * (1.0 + np.abs(s2)))
    # materialised keys through the same selection (its lists never overflow)
    sc2, tk2, bp2, _ = [x.cpu().numpy() for x in dec.topk(T(score), gpu["logp"])]
    assert np.array_equal(tk2, t2) and np.array_equal(bp2, b2) and np.array_equal(sc2, sc)


@pytest.mark.parametrize("name", ["tiny_f32", "tiny_bf16_ln"])
def test_equal_logits_overflow_in_ensemble_selection(name):
    """The same fallback for a fused two-member ensemble: with both output layers zero every
    combined value of a row is equal and every row overflows, into the stored row's rescan (the
    per-member pass with a combined buffer) and into the recomputation from both members'
    weights (the joint pass, where the library supports it).  The beam is checked exactly
    against the brute-force top-K of the keys (prev - C) + combined value."""
    log(f"\n[equal-logit ensemble overflow] {name}")
    base = synth.with_sizes(synth.PRESETS[name], V=2000, K=4, B=2)
    members = [base, dataclasses.replace(base, name=f"{base.name}_m1", index=base.index + 100)]
    weights = [0.5, 0.5]
    ctx, mask, lens = synth.make_source(base)
    tok, src, state, score = synth.mid_decode_inputs(base, salt=9)
    decs = []
    for p in members:
        w = synth.make_weights(p)
        w["Wo"] = np.zeros_like(w["Wo"])
        w["bo"] = np.zeros(p.V, np.float32)
        dec = Decoder.from_preset(p, w)
        dec.set_batch(ctx, mask, p.K)
        dec.precompute()
        decs.append(dec)
    models = [d.model for d in decs]
    outs = [torch.empty((base.M, base.H), device=DEV) for _ in decs]
    sel = [torch.empty(base.M, device=DEV)] + [torch.empty(base.M, dtype=torch.int32, device=DEV) for _ in range(3)]
    cst = torch.empty(base.M, device=DEV)
    passes = [("per-member", torch.empty((base.M, base.V), device=DEV))]
    if mt.mt_ensemble_joint_ok(models):
        passes.append(("joint", None))
    for label, comb in passes:
        for i, dec in enumerate(decs):
            mt.mt_ensemble_step(dec.model, i, 2, weights[i], base.B, base.K, dec.S, T(tok), T(src), base.M, T(state),
                                dec.ctx, dec.pctx, dec.mask, outs[i], comb, dec.ws)
        for mdl in models:  # (the counts restart at every read)
            mt.mt_recomputed_rows(mdl)
        mt.mt_ensemble_topk(models, weights, [d.ws for d in decs], base.B, base.K, T(score), comb, *sel,
                            row_const_out=cst)
        torch.cuda.synchronize()
        assert sum(mt.mt_recomputed_rows(mdl) for mdl in models) == base.M, label
        for d in decs:
            assert mt.mt_device_errors(d.model) == 0
        values = comb.cpu().numpy() if comb is not None else np.zeros((base.M, base.V), np.float32)
        assert np.all(values == 0.0)
        keys = (score.astype(np.float32) - cst.cpu().numpy())[:, None] + values
        sc, tk, bp, rw = [x.cpu().numpy() for x in sel]
        exact_topk_check(base.B, base.K, keys, sc, tk, bp)
        log(f"[equal-logit ensemble overflow] {name}: {label} pass exact, all {base.M} rows recomputed")


# ------------------------------------------------------------------------------------------
# ensembles: two members (different seeded weights) decode the same beam, each with its own
# states; their log-probabilities are combined on the GPU and one selection extends the beam
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name,weights", [("tiny_f32", (0.6, 0.4)), ("nematus_f32", (0.5, 0.5)),
                                          ("nematus_bf16_ln", (0.7, 0.3))])
def test_ensemble_step_parity(name, weights):
    base = synth.PRESETS[name]
    members = [base, dataclasses.replace(base, name=f"{name}_m2", index=base.index + 100)]
    log(f"\n[ensemble] {name} weights={weights}")
    ctx, mask, lens = synth.make_source(base)
    tok, src, state, score = synth.mid_decode_inputs(base, salt=5)
    decs, ws, logps = [], [], []
    for p in members:
        w = synth.make_weights(p, peaked_bias=True)
        dec = Decoder.from_preset(p, w)
        dec.set_batch(ctx, mask, p.K)
        dec.precompute()
        gpu = run_step(dec, p, tok, src, T(state), p.M, attn=False, taps=False)
        decs.append(dec)
        ws.append(w)
        logps.append(gpu["logp"])
    out = torch.empty_like(logps[0])
    mt.mt_ensemble_logp(decs[0].model, logps, weights, base.M, out)
    sc, tk, bp, rw = [x.cpu().numpy() for x in decs[0].topk(T(score), out)]
    torch.cuda.synchronize()
    for d in decs:
        assert mt.mt_device_errors(d.model) == 0
    sents = sample_sentences(lens, N_SAMPLE[name])
    orcs = [oracle_sentences(oracle_model(p, w), base.K, sents, ctx, mask, tok, src, state, want_alpha=False,
                             taps=False) for p, w in zip(members, ws)]
    tol = TOL[base.gemm]
    g = out.cpu().numpy()
    worst = 0.0
    for b in sents:
        rows = slice(b * base.K, (b + 1) * base.K)
        ens = mtref.ensemble_logp([o[b]["logp"] for o in orcs], weights)
        worst = max(worst, maxerr(g[rows], ens))
        topk_gap_check(base.K, score[rows], ens, sc[rows], tk[rows], bp[rows], tol["logp"])
        assert np.array_equal(rw[rows], b * base.K + bp[rows])
    log(f"[ensemble] {name}: combined logp max error {worst:.3g}")
    assert worst <= tol["logp"]
    # the combination alone, aliased in place, against the GPU members' own sum
    ref = sum(float(np.float32(x)) * l.double() for l, x in zip(logps, weights))
    mt.mt_ensemble_logp(decs[0].model, logps, weights, base.M, logps[0])
    torch.cuda.synchronize()
    assert torch.max(torch.abs(logps[0].double() - ref)).item() <= 1e-4


@pytest.mark.parametrize("name", ["tiny_bf16_ln", "nematus_bf16_ln", "deep_bf16_ln"])
def test_state_reuse_is_bit_identical(name):
    """bf16 models: steps that gather the bf16 copy of the previous state from the workspace
    (mt_set_state_reuse, as the decode loop runs them) give bit-identical states, scores and
    beams to steps that round the fp32 state again, over several steps and a restart."""
    p = synth.PRESETS[name]
    w = synth.make_weights(p, peaked_bias=True)
    ctx, mask, _ = synth.make_source(p)
    dec = Decoder.from_preset(p, w)
    dec.set_batch(ctx, mask, p.K)
    tok0, _, score0 = synth.start_beam(p)
    runs = []
    for reuse in (True, False, True):
        dec.reuse_state = reuse
        rec = []
        for restart in range(2):
            dec.precompute()
            dec.start(tok0, score0)
            for _ in range(4):
                st = dec.advance()
                rec.append([x.clone() for x in (st, dec.score, dec.tok, dec.bp)])
        torch.cuda.synchronize()
        runs.append(rec)
    assert mt.mt_device_errors(dec.model) == 0
    for a, b in zip(runs[0], runs[1]):
        for x, y in zip(a, b):
            assert torch.equal(x, y)
    for a, b in zip(runs[0], runs[2]):
        for x, y in zip(a, b):
            assert torch.equal(x, y)
    log(f"[state reuse] {name}: 8 steps bit-identical with and without the bf16 state copy")


@pytest.mark.parametrize("name,fused", [("nematus_bf16_ln", True), ("tiny_f32", False)])
def test_ensemble_member_streams_identical(name, fused):
    """Members stepping on streams of their own (the joint pass, or materialised
    log-probabilities) give bit-identical beams and states to the same members stepping one
    after another on one stream, over a restart and several steps."""
    from paper_1804_00344_amd.runner import Ensemble
    base = synth.PRESETS[name]
    ctx, mask, _ = synth.make_source(base)
    tok0, _, score0 = synth.start_beam(base)
    decs = []
    for i in range(2):
        p = dataclasses.replace(base, name=f"{name}_m{i}", index=base.index + 100 * i)
        decs.append(Decoder.from_preset(p, synth.make_weights(p, peaked_bias=True)))
    runs = []
    for conc in (True, False):
        ens = Ensemble(decs, (0.6, 0.4), fused=fused, concurrent=conc)
        assert ens.concurrent == conc
        ens.set_batch(ctx, mask, base.K)
        rec = []
        for _ in range(2):
            ens.precompute()
            ens.start(tok0, score0)
            for _ in range(3):
                states = ens.advance()
                rec.append([x.clone() for x in states] + [decs[0].score.clone(), decs[0].tok.clone(),
                                                         decs[0].bp.clone()])
        torch.cuda.synchronize()
        runs.append(rec)
    for a, b in zip(*runs):
        for x, y in zip(a, b):
            assert torch.equal(x, y)
    log(f"[ensemble streams] {name} fused={fused}: 6 steps bit-identical on member streams and on one stream")


def exact_topk_check(B, K, keys, sc, tk, bp):
    """sc/tk/bp [B*K] are, per sentence, the K best of keys [B*K, V] (flattened k*V + v),
    larger key first, equal keys by smaller flat index; bit-exact."""
    V = keys.shape[1]
    for b in range(B):
        f = keys[b * K:(b + 1) * K].reshape(-1)
        kth = np.partition(f, f.size - K)[f.size - K]
        idx = np.nonzero(f >= kth)[0]
        order = idx[np.lexsort((idx, -f[idx].astype(np.float64)))][:K]
        rows = slice(b * K, (b + 1) * K)
        assert np.array_equal(sc[rows], f[order]), (b, sc[rows], f[order])
        assert np.array_equal(tk[rows], order % V) and np.array_equal(bp[rows], order // V), b


@pytest.mark.parametrize("name,weights,peaked", [("tiny_f32", (0.6, 0.4), True), ("nematus_f32", (0.5, 0.5), True),
                                                 ("nematus_bf16_ln", (0.7, 0.3), True),
                                                 ("tiny_bf16_ln", (0.2, 0.5, 0.3), True),
                                                 ("nematus_bf16_ln", (0.5, 0.5), False),
                                                 ("tiny_f32", (0.1, 0.2, 0.3, 0.4), False),
                                                 ("nematus_bf16_ln", (0.3, 0.3, 0.4), False)])
def test_fused_ensemble_step_parity(name, weights, peaked):
    """Fused ensemble: each member adds its weighted logits into one buffer and the selection
    subtracts the per-row constant sum_i w_i LSE_i; the combined log-probabilities (buffer minus
    the constant), the members' states and the beam against the oracle's ensemble."""
    base = synth.PRESETS[name]
    members = [base] + [dataclasses.replace(base, name=f"{name}_m{i}", index=base.index + 100 * i)
                        for i in range(1, len(weights))]
    log(f"\n[fused ensemble] {name} weights={weights} peaked_bias={peaked}")
    ctx, mask, lens = synth.make_source(base)
    tok, src, state, score = synth.mid_decode_inputs(base, salt=5)
    decs, ws = [], []
    comb = torch.empty((base.M, base.V), device=DEV)
    states = []
    for i, p in enumerate(members):
        w = synth.make_weights(p, peaked_bias=peaked)   # peaked=False: the benchmark's zero output bias
        dec = Decoder.from_preset(p, w)
        dec.set_batch(ctx, mask, p.K)
        dec.precompute()
        out = torch.empty((p.M, p.H), device=DEV)
        mt.mt_ensemble_step(dec.model, i, len(weights), weights[i], p.B, p.K, dec.S, T(tok), T(src), p.M, T(state),
                            dec.ctx, dec.pctx, dec.mask, out, comb, dec.ws)
        decs.append(dec)
        ws.append(w)
        states.append(out)
    cst = torch.empty(base.M, device=DEV)
    sc_t, tk_t, bp_t, rw_t = (torch.empty(base.M, device=DEV), torch.empty(base.M, dtype=torch.int32, device=DEV),
                              torch.empty(base.M, dtype=torch.int32, device=DEV),
                              torch.empty(base.M, dtype=torch.int32, device=DEV))
    mt.mt_ensemble_topk([d.model for d in decs], weights, [d.ws for d in decs], base.B, base.K, T(score), comb, sc_t,
                        tk_t, bp_t, rw_t, row_const_out=cst)
    torch.cuda.synchronize()
    for d in decs:
        assert mt.mt_device_errors(d.model) == 0
    g = (comb - cst[:, None]).cpu().numpy()
    sc, tk, bp, rw = [x.cpu().numpy() for x in (sc_t, tk_t, bp_t, rw_t)]
    # the selection from the last member's candidates is exactly the best K of the keys
    # (prev - C) + stored combined value over each sentence's whole K x V block (fp32, the
    # same two roundings), ties to the smaller flat index
    keys = (score.astype(np.float32) - cst.cpu().numpy())[:, None] + comb.cpu().numpy()
    exact_topk_check(base.B, base.K, keys, sc, tk, bp)
    sents = sample_sentences(lens, N_SAMPLE[name] if name in N_SAMPLE else 99)
    orcs = [oracle_sentences(oracle_model(p, w), base.K, sents, ctx, mask, tok, src, state, want_alpha=False,
                             taps=False) for p, w in zip(members, ws)]
    tol = TOL[base.gemm]
    worst = worst_s = 0.0
    dec_n = tot = 0
    for b in sents:
        rows = slice(b * base.K, (b + 1) * base.K)
        ens = mtref.ensemble_logp([o[b]["logp"] for o in orcs], weights)
        worst = max(worst, maxerr(g[rows], ens))
        for o, st in zip(orcs, states):
            worst_s = max(worst_s, maxerr(st[rows].cpu().numpy(), o[b]["state"]))
        d, n = topk_gap_check(base.K, score[rows], ens, sc[rows], tk[rows], bp[rows], tol["logp"])
        dec_n += d
        tot += n
        assert np.array_equal(rw[rows], b * base.K + bp[rows])
    log(f"[fused ensemble] {name}: combined logp max error {worst:.3g}, member state error {worst_s:.3g}, "
        f"decided slots {dec_n}/{tot}")
    assert worst <= tol["logp"] and worst_s <= tol["state"]

    # the joint vocabulary pass (one kernel for all members, nothing of size [rows][V] written)
    # on the same inputs: states equal to the per-member pass's, the row constant equal up to
    # the partials' chunking, the beam the oracle's under the gap rule and, against the
    # per-member pass's stored combined values (the same products summed in the same order),
    # exact where a gap of 1e-5 separates candidates
    if mt.mt_ensemble_joint_ok([d.model for d in decs]):
        comb_np = comb.cpu().numpy()
        cst_np = cst.cpu().numpy()
        states_j = []
        for i, dec in enumerate(decs):
            out = torch.empty((base.M, base.H), device=DEV)
            mt.mt_ensemble_step(dec.model, i, len(weights), weights[i], base.B, base.K, dec.S, T(tok), T(src), base.M,
                                T(state), dec.ctx, dec.pctx, dec.mask, out, None, dec.ws)
            states_j.append(out)
        cst_j = torch.empty(base.M, device=DEV)
        mt.mt_recomputed_rows(decs[0].model)
        mt.mt_ensemble_topk([d.model for d in decs], weights, [d.ws for d in decs], base.B, base.K, T(score), None,
                            sc_t, tk_t, bp_t, rw_t, row_const_out=cst_j)
        torch.cuda.synchronize()
        n_rec = mt.mt_recomputed_rows(decs[0].model)
        for a_, b_ in zip(states_j, states):
            assert torch.equal(a_, b_)
        cj = cst_j.cpu().numpy()
        assert np.max(np.abs(cj - cst_np) / (1.0 + np.abs(cst_np))) <= 1e-5
        scj, tkj, bpj, rwj = [x.cpu().numpy() for x in (sc_t, tk_t, bp_t, rw_t)]
        prev_j = score.astype(np.float32) - cj
        dj = 0
        for b in sents:
            rows = slice(b * base.K, (b + 1) * base.K)
            ens = mtref.ensemble_logp([o[b]["logp"] for o in orcs], weights)
            topk_gap_check(base.K, score[rows], ens, scj[rows], tkj[rows], bpj[rows], tol["logp"])
            assert np.array_equal(rwj[rows], b * base.K + bpj[rows])
        for b in range(base.B):
            rows = slice(b * base.K, (b + 1) * base.K)
            tau = 1e-5 * (1.0 + float(np.max(np.abs(scj[rows][np.isfinite(scj[rows])]), initial=0.0)))
            d, _ = topk_gap_check(base.K, prev_j[rows], comb_np[rows], scj[rows], tkj[rows], bpj[rows], tau)
            dj += d
        log(f"[fused ensemble] {name}: joint pass, decided slots against the stored combined values "
            f"{dj}/{base.M}, rows recomputed {n_rec}")
    # the same beam through the runner's fused and materialised ensembles agrees within the
    # rounding of the two forms
    from paper_1804_00344_amd.runner import Ensemble
    sel = {}
    for fused in (True, False):
        ens = Ensemble(decs, weights, fused=fused)
        ens.set_batch(ctx, mask, base.K)
        ens.precompute()
        tok0, _, score0 = synth.start_beam(base)
        ens.start(tok0, score0)
        ens.advance()
        torch.cuda.synchronize()
        sel[fused] = [x.cpu().numpy().copy() for x in (decs[0].score, decs[0].tok, decs[0].bp)]
    assert np.all(np.abs(sel[True][0] - sel[False][0]) <= 2 * tol["logp"])
    agree = np.mean((sel[True][1] == sel[False][1]) & (sel[True][2] == sel[False][2]))
    log(f"[fused ensemble] {name}: step-0 beam agreement fused vs materialised {agree:.4f}")


# ------------------------------------------------------------------------------------------
# translation bookkeeping (mt_beam_finish) and whole translations
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("B,K,steps", [(7, 12, 9), (3, 16, 1), (5, 1, 6), (64, 12, 40)])
def test_beam_nbest_bit_exact(B, K, steps):
    """mt_beam_nbest on random records (ties in the normalised scores, empty and full lists,
    hypotheses finished at every step) against a plain CPU ranking and walk back through the
    records: order and token rows equal."""
    p = synth.PRESETS["tiny_f32"]
    dec = Decoder(p.E, p.H, p.A, p.V, synth.make_weights(p), k_max=16)
    rng = np.random.default_rng(7 + B * K + steps)
    M = B * K
    ht = rng.integers(0, 1000, (steps, M)).astype(np.int32)
    hb = rng.integers(0, K, (steps, M)).astype(np.int32)
    fc = rng.integers(0, K + 1, B).astype(np.int32)
    fc[0], fc[-1] = K, 0
    fn = rng.choice(np.array([-1.5, -2.0, -0.25, -3.0], np.float32), M) + \
        (rng.random(M) < 0.5) * rng.standard_normal(M).astype(np.float32)
    fn = fn.astype(np.float32)
    fst = rng.integers(0, steps, M).astype(np.int32)
    fpa = rng.integers(0, K, M).astype(np.int32)
    fto = rng.integers(0, 1000, M).astype(np.int32)
    ld = steps + 3
    order = torch.full((M,), 77, dtype=torch.int32, device=DEV)
    seq = torch.full((M, ld), 77, dtype=torch.int32, device=DEV)
    mt.mt_beam_nbest(dec.model, B, K, steps, T(ht), T(hb), T(fc), T(fn), T(fst), T(fpa), T(fto), order, seq)
    torch.cuda.synchronize()
    g_order, g_seq = order.cpu().numpy(), seq.cpu().numpy()
    for b in range(B):
        ents = list(range(int(fc[b])))
        ents.sort(key=lambda e: (-float(fn[b * K + e]), e))
        for r in range(K):
            row = g_seq[b * K + r]
            if r >= len(ents):
                assert g_order[b * K + r] == -1 and np.all(row == -1), (b, r)
                continue
            e = ents[r]
            f = b * K + e
            assert g_order[b * K + r] == e, (b, r, g_order[b * K + r], e)
            toks = [int(fto[f])]
            par = int(fpa[f])
            for st in range(int(fst[f]) - 1, -1, -1):
                toks.append(int(ht[st, b * K + par]))
                par = int(hb[st, b * K + par])
            toks = toks[::-1]
            n = len(toks)
            assert row[:n].tolist() == toks, (b, r)
            assert np.all(row[n:] == -1), (b, r)


@pytest.mark.parametrize("B,K,final", [(5, 4, False), (7, 12, False), (3, 16, True), (4, 1, False)])
def test_beam_finish_bit_exact(B, K, final):
    """Random ranked beams (some EOS tokens, some -inf scores, beams already shrunk) through
    the C ABI against the oracle's bookkeeping: every output equal (the normalised score to
    a few ulps: the kernel raises to the power in fp32)."""
    p = synth.PRESETS["tiny_f32"]
    dec = Decoder(p.E, p.H, p.A, p.V, synth.make_weights(p), k_max=16)
    rng = np.random.default_rng(100 + B * K)
    M, eos, step, alpha = B * K, 7, 3, 0.6
    tok = rng.integers(0, 10, M).astype(np.int32)
    tok[rng.random(M) < 0.3] = eos
    bp = rng.integers(0, K, M).astype(np.int32)
    row = ((np.arange(M) // K) * K + bp).astype(np.int32)
    score = np.sort(-rng.random((B, K)) * 5, axis=1)[:, ::-1].reshape(-1).astype(np.float32)
    score[rng.random(M) < 0.15] = -np.inf
    beam = rng.integers(0, K + 1, B).astype(np.int32)
    fcount = (K - beam).astype(np.int32)
    o_tok, o_bp, o_row, o_score, o_beam, fin = mtref.beam_finish(K, step, eos, alpha, tok, bp, row, score, beam,
                                                                 final=final)
    g = {n: T(a) for n, a in dict(tok=tok, bp=bp, row=row, score=score, beam=beam, fc=fcount).items()}
    ht, hb = torch.empty(M, dtype=torch.int32, device=DEV), torch.empty(M, dtype=torch.int32, device=DEV)
    fs, fn = torch.full((M,), 9.0, device=DEV), torch.full((M,), 9.0, device=DEV)
    fst, fpa, fto = [torch.full((M,), -5, dtype=torch.int32, device=DEV) for _ in range(3)]
    mt.mt_beam_finish(dec.model, B, K, step, eos, alpha, final, g["tok"], g["bp"], g["row"], g["score"], g["beam"],
                      g["fc"], ht, hb, fs, fn, fst, fpa, fto)
    torch.cuda.synchronize()
    c = lambda x: x.cpu().numpy()
    assert np.array_equal(c(g["tok"]), o_tok) and np.array_equal(c(g["bp"]), o_bp)
    assert np.array_equal(c(g["row"]), o_row) and np.array_equal(c(g["score"]), o_score)
    assert np.array_equal(c(g["beam"]), o_beam) and np.array_equal(c(ht), o_tok) and np.array_equal(c(hb), o_bp)
    assert np.array_equal(c(g["fc"]), fcount + (beam - o_beam))
    seen = np.zeros(B, np.int32)
    for (b, sc, norm, st, par, tk) in fin:
        f = b * K + fcount[b] + seen[b]
        seen[b] += 1
        assert c(fs)[f] == np.float32(sc) and c(fst)[f] == st and c(fpa)[f] == par and c(fto)[f] == tk
        assert abs(c(fn)[f] - norm) <= 4e-7 * max(1.0, abs(norm))


# (tiny_f32, 0): every hypothesis ends in EOS within 3 steps; (tiny_f32, 3) and
# (tiny_deep_f32_ln, 1): some end in EOS mid-decode, the rest are finished at the last step
@pytest.mark.parametrize("name,eos", [("tiny_f32", 0), ("tiny_f32", 3), ("tiny_deep_f32_ln", 1)])
def test_translate_nbest_parity(name, eos):
    """Whole translations to n-best lists on the GPU (steps, selections, bookkeeping, host
    backtracking) against the oracle's translation loop on the same seeded inputs."""
    from paper_1804_00344_amd.runner import translate
    p, w, ctx, mask, lens, dec = setup(name, peaked=True)
    # EOS among the most probable tokens under the peaked output prior, so that hypotheses
    # finish at different steps and the beams shrink mid-decode
    alpha, steps = 0.6, 12
    tok0, _, score0 = synth.start_beam(p)
    nb, ran = translate(dec, tok0, score0, steps, eos, alpha)
    om = oracle_model(p, w)
    ref = mtref.translate(om, p.K, ctx, mask, tok0, score0, steps, eos, alpha)
    n_eos = 0
    for b in range(p.B):
        assert len(nb[b]) == len(ref[b]) == p.K, (b, len(nb[b]), len(ref[b]))
        for g, r in zip(nb[b], ref[b]):
            assert g[2] == r[2], (b, g, r)
            assert abs(g[1] - r[1]) <= TOL[p.gemm]["logp"] * len(r[2])
            n_eos += r[2][-1] == eos
    lens_ = sorted({len(r[2]) for b in range(p.B) for r in ref[b]})
    log(f"[translate] {name}: {p.B} sentences, {ran} steps, {n_eos} of {p.B * p.K} hypotheses end in EOS, "
        f"lengths {lens_}")


# ------------------------------------------------------------------------------------------
# encoder (mt_encode): bi-directional GRU over source tokens, then the decoder step on its
# context
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name,src_V,n_sent,enc_T,eln", [
    ("tiny_f32", 1000, 99, 0, False), ("tiny_bf16_ln", 1000, 6, 0, False), ("nematus_f32", 30000, 3, 0, False),
    ("nematus_bf16_ln", 30000, 3, 0, False), ("tiny_f32", 1000, 99, 3, False), ("tiny_bf16_ln", 1000, 6, 3, False),
    ("nematus_f32", 30000, 3, 3, False), ("nematus_bf16_ln", 30000, 3, 3, False), ("tiny_f32", 1000, 20, 1, False),
    ("tiny_f32", 1000, 99, 3, True), ("tiny_f32", 1000, 20, 0, True), ("tiny_bf16_ln", 1000, 6, 3, True),
    ("nematus_f32", 30000, 3, 3, True), ("nematus_bf16_ln", 30000, 3, 3, True)])
def test_encoder_parity(name, src_V, n_sent, enc_T, eln):
    """Encoded context against the oracle's encoder; enc_T > 0: deep-transition cells (an input
    block and enc_T recurrent-only blocks per direction; the deep model's cell has four); eln:
    layer norm inside the encoder's blocks."""
    p = synth.PRESETS[name]
    log(f"\n[encoder] {name} src_V={src_V} transitions={enc_T} layer_norm={eln}")
    w = synth.make_weights(p, peaked_bias=True)
    ew = synth.make_encoder_weights(p, src_V, transitions=enc_T, layer_norm=eln)
    _, mask, lens = synth.make_source(p)
    S = mask.shape[1]
    src = synth.source_tokens(p, src_V, lens, S)
    dec = Decoder(p.E, p.H, p.A, p.V, {**w, **ew}, gemm=p.gemm, layer_norm=p.layer_norm, k_max=max(p.K, 1),
                  src_V=src_V, enc_transitions=enc_T, enc_layer_norm=eln)
    trans = tuple(ew[k] for k in synth.ENCODER_TRANSITION_NAMES) if enc_T else None
    lnp = tuple(ew[k] for k in synth.ENCODER_LN_NAMES if k in ew) if eln else None
    dec.set_source(src, mask, p.K)
    dec.precompute()
    ctx_gpu = dec.ctx.float().cpu().numpy()
    assert mt.mt_device_errors(dec.model) == 0
    sents = sample_sentences(lens, n_sent)
    tol = TOL[p.gemm]["state"]
    worst = 0.0
    for b in sents:
        ref = mtref.encode(src[b:b + 1], mask[b:b + 1], *[ew[k] for k in synth.ENCODER_NAMES], transitions=trans,
                           ln=lnp, eps=1e-5)
        L = int(lens[b])
        worst = max(worst, maxerr(ctx_gpu[b, :L], ref[0, :L]))
    log(f"[encoder] {name} T={enc_T} LN={eln}: context max error {worst:.3g} over sentences {sents[:6]}")
    assert worst <= tol
    if name == "tiny_f32" and enc_T == 0 and not eln:
        # the step on the encoded context against the oracle's encoder + step
        ctx_o = mtref.encode(src, mask, *[ew[k] for k in synth.ENCODER_NAMES])
        tok, srow, state, score = synth.mid_decode_inputs(p, salt=6)
        gpu = run_step(dec, p, tok, srow, T(state), p.M)
        orc = oracle_sentences(oracle_model(p, w), p.K, sents, ctx_o, mask, tok, srow, state)
        compare_rows(p, gpu, orc, sents, TOL[p.gemm], name + "_encoded")


@pytest.mark.parametrize("S,lens,enc_T,eln", [(1, [1, 1, 1], 3, True), (7, [1, 7, 2, 5], 3, True),
                                               (7, [1, 7, 2, 5], 0, False), (5, [5], 1, False),
                                               (9, [3, 9, 1, 9, 4, 2], 2, True)])
def test_encoder_edge_shapes(S, lens, enc_T, eln):
    """Single-position sources, one-token sentences beside full ones, a single sentence:
    every position of the context, padded ones included (the forward state carried, the
    backward state zero), against the oracle's encoder."""
    p = synth.PRESETS["tiny_f32"]
    src_V = 50
    log(f"\n[encoder edge] S={S} lens={lens} transitions={enc_T} layer_norm={eln}")
    w = synth.make_weights(p, peaked_bias=True)
    ew = synth.make_encoder_weights(p, src_V, transitions=enc_T, layer_norm=eln)
    lens = np.asarray(lens)
    mask = (np.arange(S)[None, :] < lens[:, None]).astype(np.float32)
    src = synth.source_tokens(p, src_V, lens, S)
    dec = Decoder(p.E, p.H, p.A, p.V, {**w, **ew}, gemm=p.gemm, layer_norm=p.layer_norm, k_max=max(p.K, 1),
                  src_V=src_V, enc_transitions=enc_T, enc_layer_norm=eln)
    dec.set_source(src, mask, p.K)
    got = dec.ctx.float().cpu().numpy()
    assert mt.mt_device_errors(dec.model) == 0
    trans = tuple(ew[k] for k in synth.ENCODER_TRANSITION_NAMES) if enc_T else None
    lnp = tuple(ew[k] for k in synth.ENCODER_LN_NAMES if k in ew) if eln else None
    ref = mtref.encode(src, mask, *[ew[k] for k in synth.ENCODER_NAMES], transitions=trans, ln=lnp, eps=1e-5)
    err = maxerr(got, ref)
    log(f"[encoder edge] max error {err:.3g}")
    assert err <= TOL["f32"]["state"]
    assert np.all(got[:, :, p.H:][mask == 0] == 0)


# ------------------------------------------------------------------------------------------
# dual-source steps: a second source with its own attention; GRU 2 and the readout take both
# contexts
# ------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name,n_sent", [("tiny_f32", 99), ("tiny_bf16_ln", 6), ("nematus_f32", 3),
                                         ("nematus_bf16_ln", 3)])
def test_dual_source_step_parity(name, n_sent):
    p = synth.PRESETS[name]
    log(f"\n[dual] {name}")
    w = {**synth.make_weights(p, peaked_bias=True), **synth.make_dual_weights(p)}
    ctx, mask, lens = synth.make_source(p)
    ctx2, mask2, _ = synth.make_source2(p)
    dec = Decoder(p.E, p.H, p.A, p.V, w, gemm=p.gemm, layer_norm=p.layer_norm, k_max=max(p.K, 1), dual_source=True)
    dec.set_batch(ctx, mask, p.K)
    dec.set_second_source(ctx2, mask2)
    dec.precompute()
    tok, src, state, score = synth.mid_decode_inputs(p, salt=7)
    gpu = run_step(dec, p, tok, src, T(state), p.M, taps=False)
    sc, tk, bp, rw = [x.cpu().numpy() for x in dec.topk(T(score), None)]
    torch.cuda.synchronize()
    assert mt.mt_device_errors(dec.model) == 0
    sents = sample_sentences(lens, n_sent)
    orc = oracle_sentences(oracle_model(p, w, dual=True), p.K, sents, ctx, mask, tok, src, state, taps=False,
                           src2=(ctx2, mask2))
    tol = TOL[p.gemm]
    compare_rows(p, gpu, orc, sents, tol, name + "_dual")
    for b in sents:
        rows = slice(b * p.K, (b + 1) * p.K)
        topk_gap_check(p.K, score[rows], orc[b]["logp"], sc[rows], tk[rows], bp[rows], tol["logp"])
        assert np.array_equal(rw[rows], b * p.K + bp[rows])
    # a shallow call on a dual-source model is refused
    with pytest.raises(mt.MtError):
        mt.mt_decoder_step(dec.model, p.B, p.K, dec.S, T(tok), T(src), p.M, T(state), dec.ctx, dec.pctx, dec.mask,
                           torch.empty((p.M, p.H), device=DEV), ws=dec.ws)
