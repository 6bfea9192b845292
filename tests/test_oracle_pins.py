"""Pins for the CPU oracle: checks against what the mathematics and the paper fix.

Each test ties one part of the oracle to something other than itself:
library routines it must reduce to (torch.nn.GRUCell, F.layer_norm,
log_softmax), closed forms, invariants (normalisation, masking, scale and
permutation invariance, sentence independence), brute force on tiny inputs,
and the attention rows the paper prints in Figure 2.
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import mtref

GOLD = os.path.join(os.path.dirname(__file__), "golden")
rng0 = np.random.default_rng(1804)


def rnd(*shape, s=1.0, rng=rng0):
    return (rng.standard_normal(shape) * s).astype(np.float32)


# --------------------------------------------------------------------------------------
# GRU block: reduction to torch.nn.GRUCell (PyTorch's documented r, z, n equations with
# the reset gate applied to the recurrent product, h' = (1 - z) n + z h)
# --------------------------------------------------------------------------------------


def torch_gru(x, h, W, U, b):
    H = h.size
    cell = torch.nn.GRUCell(x.size, H, bias=True).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(W.astype(np.float64).T))
        cell.weight_hh.copy_(torch.from_numpy(U.astype(np.float64).T))
        cell.bias_ih.copy_(torch.from_numpy(b.astype(np.float64)))
        cell.bias_hh.zero_()
        out = cell(torch.from_numpy(x.astype(np.float64))[None], torch.from_numpy(h.astype(np.float64))[None])
    return out[0].numpy()


@pytest.mark.parametrize("in_dim,H", [(7, 5), (3, 9), (16, 16)])
def test_gru_equals_torch_grucell(in_dim, H):
    rng = np.random.default_rng(in_dim * 100 + H)
    x, h = rnd(in_dim, rng=rng), np.tanh(rnd(H, rng=rng))
    W, U, b = rnd(in_dim, 3 * H, s=0.7, rng=rng), rnd(H, 3 * H, s=0.7, rng=rng), rnd(3 * H, s=0.3, rng=rng)
    got = mtref.gru(x, h, W, U, b)
    ref = torch_gru(x, h, W, U, b)
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_gru_closed_forms():
    rng = np.random.default_rng(5)
    in_dim, H = 6, 4
    x, h = rnd(in_dim, rng=rng), np.tanh(rnd(H, rng=rng))
    b = rnd(3 * H, rng=rng)
    # all weights zero, b_z = 0 -> z = 1/2, hh = tanh(b_h): s = (tanh(b_h) + h) / 2
    bz = b.copy()
    bz[H:2 * H] = 0
    s = mtref.gru(x, h, np.zeros((in_dim, 3 * H), np.float32), np.zeros((H, 3 * H), np.float32), bz)
    assert np.max(np.abs(s - 0.5 * (np.tanh(bz[2 * H:].astype(np.float64)) + h))) <= 1e-15
    # b_z = +40: the update gate keeps the old state
    W, U = rnd(in_dim, 3 * H, s=0.3, rng=rng), rnd(H, 3 * H, s=0.3, rng=rng)
    bc = b.copy()
    bc[H:2 * H] = 40.0
    assert np.max(np.abs(mtref.gru(x, h, W, U, bc) - h)) <= 1e-15
    # b_z = -40 and U_h = 0: the state becomes tanh(x W_h + b_h)
    bn = b.copy()
    bn[H:2 * H] = -40.0
    U0 = U.copy()
    U0[:, 2 * H:] = 0
    want = np.tanh(x.astype(np.float64) @ W[:, 2 * H:].astype(np.float64) + bn[2 * H:])
    assert np.max(np.abs(mtref.gru(x, h, W, U0, bn) - want)) <= 1e-15


# --------------------------------------------------------------------------------------
# layer normalisation
# --------------------------------------------------------------------------------------


@pytest.mark.parametrize("n", [1, 5, 64, 1000])
def test_layer_norm_equals_torch(n):
    rng = np.random.default_rng(n)
    x = rng.standard_normal(n) * 3 + 1.5
    g, b = rnd(n, rng=rng), rnd(n, rng=rng)
    got = mtref.layer_norm(x, g, b, 1e-5)
    ref = F.layer_norm(torch.from_numpy(x)[None], (n,), torch.from_numpy(g.astype(np.float64)),
                       torch.from_numpy(b.astype(np.float64)), eps=1e-5)[0].numpy()
    assert np.max(np.abs(got - ref)) <= 1e-12


def test_layer_norm_closed_forms():
    n = 37
    g, b = rnd(n), rnd(n)
    # constant input: x - mean = 0 exactly, output = beta
    assert np.array_equal(mtref.layer_norm(np.full(n, 2.75), g, b), b.astype(np.float64))
    # unit gain, zero shift: mean 0 and variance var/(var + eps)
    x = np.random.default_rng(3).standard_normal(n) * 0.01
    y = mtref.layer_norm(x, np.ones(n, np.float32), np.zeros(n, np.float32), 1e-5)
    var = x.var()
    assert abs(y.mean()) <= 1e-12
    assert abs(y.var() - var / (var + 1e-5)) <= 1e-12


def test_ln_gru_gain_zero_gives_shifts_only():
    """gamma = 0 on every LN instance: each normalised block equals its shift beta,
    so the gates depend on the betas only (a check of which beta feeds which gate)."""
    rng = np.random.default_rng(11)
    in_dim, H = 5, 3
    x, h = rnd(in_dim, rng=rng), np.tanh(rnd(H, rng=rng))
    W, U, b = rnd(in_dim, 3 * H, rng=rng), rnd(H, 3 * H, rng=rng), rnd(3 * H, rng=rng)
    ba, bu = rnd(3 * H, rng=rng).astype(np.float64), rnd(3 * H, rng=rng).astype(np.float64)
    z0 = np.zeros(3 * H, np.float32)
    s = mtref.gru(x, h, W, U, b, ln=(z0, ba.astype(np.float32), z0, bu.astype(np.float32)))
    sig = lambda v: 1 / (1 + np.exp(-v))
    r = sig(ba[:H] + bu[:H])
    z = sig(ba[H:2 * H] + bu[H:2 * H])
    hh = np.tanh(ba[2 * H:] + r * bu[2 * H:])
    assert np.max(np.abs(s - ((1 - z) * hh + z * h))) <= 1e-15


def test_ln_gru_scale_invariance():
    """LN on each H-block of each path makes the block invariant to a positive
    rescaling of that block's weights (exact up to eps)."""
    rng = np.random.default_rng(12)
    in_dim, H = 8, 6
    x, h = rnd(in_dim, rng=rng), np.tanh(rnd(H, rng=rng))
    W, U, b = rnd(in_dim, 3 * H, rng=rng), rnd(H, 3 * H, rng=rng), rnd(3 * H, rng=rng)
    ln = tuple(rnd(3 * H, rng=rng) for _ in range(4))
    base = mtref.gru(x, h, W, U, b, ln=ln, eps=1e-12)
    for g in range(3):
        U2 = U.copy()
        U2[:, g * H:(g + 1) * H] *= 4.0  # powers of two: the scaled fp32 weights are exact
        W2, b2 = W.copy(), b.copy()
        W2[:, g * H:(g + 1) * H] *= 0.25
        b2[g * H:(g + 1) * H] *= 0.25
        assert np.max(np.abs(mtref.gru(x, h, W2, U2, b2, ln=ln, eps=1e-12) - base)) <= 1e-12
    # a scaling that mixes blocks is NOT an invariance (LN must be per block)
    U3 = U.copy()
    U3[:, :H] *= 3.5
    U3[:, H:] *= 1.0
    W3 = W.copy()
    W3[:, H] *= 5.0
    assert np.max(np.abs(mtref.gru(x, h, W3, U3, b, ln=ln, eps=1e-12) - base)) > 1e-6


# --------------------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------------------


def attn_case(S=9, A=6, Cd=10, lens=5, seed=0):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal(A)
    P, Cx = rnd(S, A, rng=rng), rnd(S, Cd, rng=rng)
    mask = (np.arange(S) < lens).astype(np.float32)
    va = rnd(A, rng=rng)
    return q, P, Cx, mask, va


@pytest.mark.parametrize("L", [1, 2, 5, 9])
def test_attention_normalised_and_masked(L):
    q, P, Cx, mask, va = attn_case(lens=L, seed=L)
    P[L:] = np.nan
    Cx[L:] = np.nan
    alpha, ctx = mtref.attention(q, P, Cx, mask, va)
    assert abs(alpha.sum() - 1.0) <= 1e-12
    assert np.all(alpha[L:] == 0.0) and np.all(np.isfinite(ctx))
    assert np.all(alpha[:L] > 0)
    if L == 1:
        assert alpha[0] == 1.0
        assert np.array_equal(ctx, Cx[0].astype(np.float64))


def test_attention_zero_va_is_uniform_mean():
    q, P, Cx, mask, va = attn_case(lens=6, seed=3)
    alpha, ctx = mtref.attention(q, P, Cx, mask, np.zeros_like(va))
    assert np.max(np.abs(alpha[:6] - 1 / 6)) <= 1e-15
    assert np.max(np.abs(ctx - Cx[:6].astype(np.float64).mean(0))) <= 1e-13


def test_attention_one_dim_reduces_to_softmax():
    """A = 1, va = 1: the scores are tanh(P_i + q) and alpha is scipy's softmax of them."""
    from scipy.special import softmax
    S = 11
    rng = np.random.default_rng(4)
    P = rnd(S, 1, rng=rng)
    q = np.array([0.3])
    mask = np.ones(S, np.float32)
    mask[[2, 7]] = 0  # not a prefix: positions 2 and 7 masked
    Cx = rnd(S, 3, rng=rng)
    alpha, ctx = mtref.attention(q, P, Cx, mask, np.ones(1, np.float32))
    keep = mask != 0
    e = np.tanh(P[keep, 0].astype(np.float64) + 0.3)
    assert np.max(np.abs(alpha[keep] - softmax(e))) <= 1e-15
    assert np.all(alpha[~keep] == 0)
    assert np.max(np.abs(ctx - softmax(e) @ Cx[keep].astype(np.float64))) <= 1e-14


def test_attention_all_masked_is_zero():
    q, P, Cx, mask, va = attn_case(lens=0, seed=5)
    alpha, ctx = mtref.attention(q, P, Cx, mask, va)
    assert np.all(alpha == 0) and np.all(ctx == 0)


def _load_fig2(name):
    rows = [l for l in open(os.path.join(GOLD, name)) if l[0].isdigit()]
    xs, ys, vs = zip(*[(int(a), int(b), float(c)) for a, b, c in (r.strip().split(",") for r in rows)])
    X, Y = max(xs) + 1, max(ys) + 1
    m = np.zeros((Y, X))
    for x, y, v in zip(xs, ys, vs):
        m[y, x] = v
    return m


@pytest.mark.parametrize("name", ["fig2_mt_to_pe_attention.csv", "fig2_src_to_pe_attention.csv"])
def test_attention_reproduces_paper_figure2_rows(name):
    """Figure 2 prints attention rows of a trained model to 4 decimals.

    Witness: every printed row sums to 1 within the rounding bound n * 5e-5.
    Reproduction: with A = 1 and keys chosen so that each score equals the log
    of the printed weight, the oracle's masked softmax returns the printed row
    (within rounding and the row's renormalisation)."""
    m = _load_fig2(name)
    n = m.shape[1]
    assert np.all(np.abs(m.sum(1) - 1.0) <= n * 5e-5)
    for row in m:
        logs = np.log(np.maximum(row, 2.5e-5))
        w = 2.0 * np.max(np.abs(logs - logs.mean()))
        P = np.arctanh((logs - logs.mean()) / w).astype(np.float32)[:, None]
        Cx = np.eye(n, dtype=np.float32)
        alpha, ctx = mtref.attention(np.zeros(1), P, Cx, np.ones(n, np.float32), np.array([w], np.float32))
        assert np.max(np.abs(alpha - row)) <= n * 5e-5 + 1e-4
        assert np.max(np.abs(ctx - alpha)) == 0.0  # identity context returns alpha itself


# --------------------------------------------------------------------------------------
# log-softmax
# --------------------------------------------------------------------------------------


@pytest.mark.parametrize("n", [1, 2, 1000, 50000])
def test_log_softmax(n):
    l = np.random.default_rng(n).standard_normal(n) * 5
    out, lse = mtref.log_softmax(l)
    assert abs(np.log(np.exp(out).sum())) <= 1e-12
    ref = torch.log_softmax(torch.from_numpy(l), 0).numpy()
    assert np.max(np.abs(out - ref)) <= 1e-12
    assert abs(lse - torch.logsumexp(torch.from_numpy(l), 0).item()) <= 1e-12


# --------------------------------------------------------------------------------------
# top-K beam selection: brute force
# --------------------------------------------------------------------------------------


def brute_topk(K, score, logp):
    M, V = logp.shape
    B = M // K
    tok, bp, sc = [], [], []
    for b in range(B):
        c = []
        for k in range(K):
            for v in range(V):
                c.append((-float(np.float32(score[b * K + k]) + np.float32(logp[b * K + k, v])), k * V + v))
        c.sort()
        for j in range(K):
            tok.append(c[j][1] % V)
            bp.append(c[j][1] // V)
            sc.append(np.float32(score[b * K + bp[-1]]) + np.float32(logp[b * K + bp[-1], tok[-1]]))
    return np.array(tok), np.array(bp), np.array(sc, np.float32)


@pytest.mark.parametrize("K", [1, 2, 3, 4])
@pytest.mark.parametrize("V", [4, 7, 20])
def test_topk_brute_force_with_ties(K, V):
    if V < K:
        pytest.skip("K > V")
    rng = np.random.default_rng(K * 31 + V)
    B = 3
    logp = rng.choice(np.array([-1.0, -2.0, -2.5, -3.0], np.float32), size=(B * K, V))
    score = rng.choice(np.array([0.0, -0.5, -1.0], np.float32), size=B * K)
    tok, bp, sc = mtref.topk(K, score, logp)
    t2, b2, s2 = brute_topk(K, score, logp)
    assert np.array_equal(tok, t2) and np.array_equal(bp, b2) and np.array_equal(sc, s2)


def test_topk_random_v1000():
    K, B, V = 4, 2, 1000
    rng = np.random.default_rng(9)
    logp = rnd(B * K, V, rng=rng)
    score = rnd(B * K, rng=rng)
    tok, bp, sc = mtref.topk(K, score, logp)
    t2, b2, s2 = brute_topk(K, score, logp)
    assert np.array_equal(tok, t2) and np.array_equal(bp, b2) and np.array_equal(sc, s2)


def test_topk_k1_is_argmax_smallest_index():
    logp = np.array([[0.5, 2.0, 2.0, 1.0], [3.0, -1.0, 3.0, 3.0]], np.float32)
    tok, bp, sc = mtref.topk(1, np.zeros(2, np.float32), logp)
    assert tok.tolist() == [1, 0] and bp.tolist() == [0, 0]
    assert np.array_equal(tok, np.argmax(logp, axis=1))  # numpy argmax takes the first maximum


def test_topk_bos_start_draws_from_hyp0():
    K, V = 4, 50
    rng = np.random.default_rng(2)
    logp = rnd(K, V, rng=rng)
    score = np.array([0, -np.inf, -np.inf, -np.inf], np.float32)
    tok, bp, sc = mtref.topk(K, score, logp)
    assert np.all(bp == 0)
    assert len(set(tok.tolist())) == K
    assert np.array_equal(tok, np.argsort(-logp[0], kind="stable")[:K])


# --------------------------------------------------------------------------------------
# whole step and precompute
# --------------------------------------------------------------------------------------

E_, H_, A_, V_ = 6, 5, 7, 23


def tiny_model(seed=0, layer_norm=False, **over):
    rng = np.random.default_rng(seed)
    E, H, A, V, C = E_, H_, A_, V_, 2 * H_
    w = dict(
        emb=rnd(V, E, s=0.5, rng=rng), W1=rnd(E, 3 * H, s=0.5, rng=rng), U1=rnd(H, 3 * H, s=0.5, rng=rng),
        b1=rnd(3 * H, s=0.1, rng=rng), Ua=rnd(C, A, s=0.4, rng=rng), ba=rnd(A, s=0.1, rng=rng),
        Wa=rnd(H, A, s=0.5, rng=rng), va=rnd(A, rng=rng), W2=rnd(C, 3 * H, s=0.4, rng=rng),
        U2=rnd(H, 3 * H, s=0.5, rng=rng), b2=rnd(3 * H, s=0.1, rng=rng), Wt_s=rnd(H, E, s=0.5, rng=rng),
        Wt_y=rnd(E, E, s=0.5, rng=rng), Wt_c=rnd(C, E, s=0.4, rng=rng), bt=rnd(E, s=0.1, rng=rng),
        Wo=rnd(E, V, rng=rng), bo=rnd(V, s=0.2, rng=rng), Wi=rnd(C, H, s=0.4, rng=rng), bi=rnd(H, s=0.1, rng=rng))
    if layer_norm:
        for n in ("g1a", "g1u", "g2a", "g2u"):
            w[n] = (1 + rnd(3 * H, s=0.1, rng=rng)).astype(np.float32)
        for n in ("be1a", "be1u", "be2a", "be2u"):
            w[n] = rnd(3 * H, s=0.1, rng=rng)
        w["gt"] = (1 + rnd(E, s=0.1, rng=rng)).astype(np.float32)
        w["bet"] = rnd(E, s=0.1, rng=rng)
    w.update(over)
    return mtref.Model(E, H, A, V, w, layer_norm=layer_norm), w


def tiny_batch(B=3, K=2, S=6, seed=1, lens=None):
    rng = np.random.default_rng(seed)
    C = 2 * H_
    lens = np.array(lens if lens is not None else rng.integers(1, S + 1, size=B))
    ctx = rnd(B, S, C, rng=rng)
    mask = (np.arange(S)[None] < lens[:, None]).astype(np.float32)
    M = B * K
    tok = rng.integers(0, V_, size=M).astype(np.int32)
    src = ((np.arange(M) // K) * K + rng.integers(0, K, size=M)).astype(np.int32)
    state = np.tanh(rnd(M, H_, rng=rng))
    return ctx, mask, lens, tok, src, state


def test_precompute_matches_library_matmul_and_masked_mean():
    model, w = tiny_model()
    ctx, mask, lens, *_ = tiny_batch(B=4, S=5, lens=[1, 5, 3, 2])
    ctx[mask == 0] = np.nan  # padded positions must never be read
    P, s0 = model.precompute(ctx, mask)
    for b, L in enumerate(lens):
        c = ctx[b, :L].astype(np.float64)
        assert np.max(np.abs(P[b, :L] - (c @ w["Ua"].astype(np.float64) + w["ba"]))) <= 1e-6
        want = np.tanh(c.mean(0) @ w["Wi"].astype(np.float64) + w["bi"])
        assert np.max(np.abs(s0[b] - want)) <= 1e-6
        assert np.all(P[b, L:] == 0)
    assert np.all(np.isfinite(s0))


def test_step_reduces_to_library_pieces_when_gru2_copies_and_readout_sees_x_only():
    """b2_z = +40 makes GRU block 2 a copy (state_out = s1 = GRUCell(x, h));
    Wt_s = Wt_c = 0 leaves logp = log_softmax(tanh(x Wt_y + bt) Wo + bo)."""
    H, E, C = H_, E_, 2 * H_
    b2 = np.zeros(3 * H, np.float32)
    b2[H:2 * H] = 40.0
    model, w = tiny_model(seed=4, b2=b2, Wt_s=np.zeros((H, E), np.float32), Wt_c=np.zeros((C, E), np.float32))
    ctx, mask, lens, tok, src, state = tiny_batch(seed=5)
    P, _ = model.precompute(ctx, mask)
    out = model.step(2, tok, src, state, ctx, P, mask, taps=True)
    for m in range(tok.size):
        g = torch_gru(w["emb"][tok[m]], state[src[m]], w["W1"], w["U1"], w["b1"])
        assert np.max(np.abs(out["s1"][m] - g)) <= 1e-6
        assert np.max(np.abs(out["state"][m] - out["s1"][m])) <= 1e-7
        x = torch.from_numpy(w["emb"][tok[m]].astype(np.float64))
        t = torch.tanh(x @ torch.from_numpy(w["Wt_y"].astype(np.float64)) + torch.from_numpy(w["bt"].astype(np.float64)))
        ref = torch.log_softmax(t @ torch.from_numpy(w["Wo"].astype(np.float64)) + torch.from_numpy(w["bo"].astype(np.float64)), 0)
        assert np.max(np.abs(out["logp"][m] - ref.numpy())) <= 2e-6


def test_step_zero_va_gives_masked_mean_context():
    model, w = tiny_model(seed=6, va=np.zeros(A_, np.float32))
    ctx, mask, lens, tok, src, state = tiny_batch(seed=7)
    P, _ = model.precompute(ctx, mask)
    out = model.step(2, tok, src, state, ctx, P, mask, want_alpha=True, taps=True)
    for m in range(tok.size):
        b = m // 2
        L = lens[b]
        assert np.allclose(out["alpha"][m, :L], 1.0 / L, atol=1e-7, rtol=0)
        assert np.all(out["alpha"][m, L:] == 0)
        assert np.max(np.abs(out["c"][m] - ctx[b, :L].astype(np.float64).mean(0))) <= 1e-6


def test_step_zero_wa_makes_attention_independent_of_state():
    model, w = tiny_model(seed=8, Wa=np.zeros((H_, A_), np.float32))
    ctx, mask, lens, tok, src, state = tiny_batch(seed=9)
    P, _ = model.precompute(ctx, mask)
    a1 = model.step(2, tok, src, state, ctx, P, mask, want_alpha=True)["alpha"]
    a2 = model.step(2, tok, src, np.tanh(state * 3 + 1).astype(np.float32), ctx, P, mask, want_alpha=True)["alpha"]
    assert np.array_equal(a1, a2)


@pytest.mark.parametrize("layer_norm", [False, True])
def test_step_invariants(layer_norm):
    model, w = tiny_model(seed=10, layer_norm=layer_norm)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=11)
    ctx[mask == 0] = np.nan
    P, _ = model.precompute(ctx, mask)
    out = model.step(2, tok, src, state, ctx, P, mask, want_alpha=True)
    assert np.all(np.isfinite(out["state"])) and np.all(np.isfinite(out["logp"]))
    assert np.max(np.abs(np.log(np.exp(out["logp"].astype(np.float64)).sum(1)))) <= 1e-6
    assert np.max(np.abs(out["alpha"].sum(1) - 1)) <= 1e-6
    for m in range(tok.size):
        assert np.all(out["alpha"][m, lens[m // 2]:] == 0)
    assert np.all(np.abs(out["state"]) < 1)


def test_step_zero_output_layer_gives_uniform():
    model, w = tiny_model(seed=12, Wo=np.zeros((E_, V_), np.float32), bo=np.zeros(V_, np.float32))
    ctx, mask, lens, tok, src, state = tiny_batch(seed=13)
    P, _ = model.precompute(ctx, mask)
    out = model.step(2, tok, src, state, ctx, P, mask)
    assert np.all(out["logp"] == np.float32(-math.log(V_)))


def test_tied_output_equals_explicit_transpose():
    model, w = tiny_model(seed=14)
    w2 = dict(w)
    w2["Wo"] = np.ascontiguousarray(w["emb"].T)
    m_exp = mtref.Model(E_, H_, A_, V_, w2)
    w3 = dict(w)
    del w3["Wo"]
    m_tied = mtref.Model(E_, H_, A_, V_, w3, tied_output=True)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=15)
    P, _ = m_exp.precompute(ctx, mask)
    a = m_exp.step(2, tok, src, state, ctx, P, mask)["logp"]
    b = m_tied.step(2, tok, src, state, ctx, P, mask)["logp"]
    assert np.array_equal(a, b)


def test_sentence_independence():
    model, w = tiny_model(seed=16, layer_norm=True)
    ctx, mask, lens, tok, src, state = tiny_batch(B=3, K=2, seed=17)
    P, _ = model.precompute(ctx, mask)
    o1 = model.step(2, tok, src, state, ctx, P, mask, want_alpha=True)
    ctx2, tok2, state2 = ctx.copy(), tok.copy(), state.copy()
    ctx2[1:] = rnd(*ctx2[1:].shape)
    tok2[2:] = (tok2[2:] + 5) % V_
    state2[2:] = 0.3
    P2, _ = model.precompute(ctx2, mask)
    o2 = model.step(2, tok2, src, state2, ctx2, P2, mask, want_alpha=True)
    for k in ("state", "logp", "alpha"):
        assert np.array_equal(o1[k][:2], o2[k][:2])
        assert not np.array_equal(o1[k][2:], o2[k][2:])


def test_full_step_equals_torch_reexpression():
    """Wiring check of the no-LN step against a float64 torch re-expression built on
    torch.nn.GRUCell, masked softmax and log_softmax."""
    model, w = tiny_model(seed=18)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=19)
    P, _ = model.precompute(ctx, mask)
    out = model.step(2, tok, src, state, ctx, P, mask, want_alpha=True)
    T = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    for m in range(tok.size):
        b = m // 2
        x = w["emb"][tok[m]]
        s1 = torch_gru(x, state[src[m]], w["W1"], w["U1"], w["b1"])
        q = T(s1) @ T(w["Wa"])
        e = torch.tanh(T(P[b]) + q) @ T(w["va"])
        e = e.masked_fill(T(mask[b]) == 0, -math.inf)
        al = torch.softmax(e, 0)
        c = al @ T(ctx[b])
        s = torch_gru(c.numpy(), s1, w["W2"], w["U2"], w["b2"])
        t = torch.tanh(T(s) @ T(w["Wt_s"]) + T(x) @ T(w["Wt_y"]) + c @ T(w["Wt_c"]) + T(w["bt"]))
        lp = torch.log_softmax(t @ T(w["Wo"]) + T(w["bo"]), 0)
        assert np.max(np.abs(out["alpha"][m] - al.numpy())) <= 1e-6
        assert np.max(np.abs(out["state"][m] - s)) <= 1e-6
        assert np.max(np.abs(out["logp"][m] - lp.numpy())) <= 1e-5


# --------------------------------------------------------------------------------------
# layer-norm wiring of the whole step (layer normalisation inside the GRU blocks and on the
# readout, Section 3.1.1): each gate block of each path of both GRUs is normalised with its
# own gain/shift set, and the summed readout pre-activation is normalised before the tanh
# --------------------------------------------------------------------------------------


def torch_ln_gru(x, h, W, U, b, ga, ba, gu, bu, eps=1e-5):
    """GRU block with per-gate-block layer norm on both paths, written with F.layer_norm in
    float64: a = LN_g(x W + b), u = LN_g(h U) per block g in (r, z, h), then the usual
    r, z, candidate and convex update."""
    T64 = lambda v: torch.from_numpy(np.asarray(v, np.float64))
    H = h.size
    a = T64(x) @ T64(W) + T64(b)
    u = T64(h) @ T64(U)
    an = [F.layer_norm(a[g * H:(g + 1) * H], (H,), T64(ga[g * H:(g + 1) * H]), T64(ba[g * H:(g + 1) * H]), eps)
          for g in range(3)]
    un = [F.layer_norm(u[g * H:(g + 1) * H], (H,), T64(gu[g * H:(g + 1) * H]), T64(bu[g * H:(g + 1) * H]), eps)
          for g in range(3)]
    r = torch.sigmoid(an[0] + un[0])
    z = torch.sigmoid(an[1] + un[1])
    n = torch.tanh(an[2] + r * un[2])
    return ((1 - z) * n + z * T64(h)).numpy()


def test_ln_step_equals_torch_reexpression():
    """The layer-norm step against float64 torch: F.layer_norm on each of the three gate blocks
    of the input and recurrent paths of GRU 1 (g1a/be1a, g1u/be1u) and GRU 2 (g2a/be2a,
    g2u/be2u), and on the summed readout pre-activation (gt/bet) before the tanh.  A swapped
    parameter set, a dropped readout norm or a norm after the tanh all fail it."""
    model, w = tiny_model(seed=90, layer_norm=True)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=91)
    P, _ = model.precompute(ctx, mask)
    out = model.step(2, tok, src, state, ctx, P, mask, want_alpha=True, taps=True)
    T64 = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    eps = 1e-5
    for m in range(tok.size):
        b = m // 2
        x = w["emb"][tok[m]]
        s1 = torch_ln_gru(x, state[src[m]], w["W1"], w["U1"], w["b1"], w["g1a"], w["be1a"], w["g1u"], w["be1u"])
        assert np.max(np.abs(out["s1"][m] - s1)) <= 1e-6
        q = T64(s1) @ T64(w["Wa"])
        e = torch.tanh(T64(P[b]) + q) @ T64(w["va"])
        e = e.masked_fill(T64(mask[b]) == 0, -math.inf)
        c = torch.softmax(e, 0) @ T64(ctx[b])
        s = torch_ln_gru(c.numpy(), s1, w["W2"], w["U2"], w["b2"], w["g2a"], w["be2a"], w["g2u"], w["be2u"])
        assert np.max(np.abs(out["state"][m] - s)) <= 1e-6
        pre = T64(s) @ T64(w["Wt_s"]) + T64(x) @ T64(w["Wt_y"]) + c @ T64(w["Wt_c"]) + T64(w["bt"])
        t = torch.tanh(F.layer_norm(pre, (E_,), T64(w["gt"]), T64(w["bet"]), eps))
        assert np.max(np.abs(out["t"][m] - t.numpy())) <= 1e-6
        lp = torch.log_softmax(t @ T64(w["Wo"]) + T64(w["bo"]), 0)
        assert np.max(np.abs(out["logp"][m] - lp.numpy())) <= 1e-5


def test_ln_step_zero_readout_gain_gives_tanh_of_shift():
    """gt = 0: the normalised readout pre-activation is exactly its shift, so every row's
    readout is t = tanh(bet), whatever the state, context and token."""
    _, w0 = tiny_model(seed=92, layer_norm=True)
    bet = w0["bet"]
    model, w = tiny_model(seed=92, layer_norm=True, gt=np.zeros(E_, np.float32))
    ctx, mask, lens, tok, src, state = tiny_batch(seed=93)
    P, _ = model.precompute(ctx, mask)
    out = model.step(2, tok, src, state, ctx, P, mask, taps=True)
    ref = np.tanh(bet.astype(np.float64)).astype(np.float32)
    for m in range(tok.size):
        assert np.max(np.abs(out["t"][m] - ref)) == 0.0
    # and the log-probabilities are then the same for every row
    assert np.max(np.abs(out["logp"] - out["logp"][0:1])) == 0.0


def test_ln_step_parameter_sets_are_not_interchangeable():
    """Exchanging GRU 1's layer-norm sets (g1a, be1a, g1u, be1u) with GRU 2's changes the new
    state, and so does exchanging the input-path and recurrent-path sets of one GRU: each of
    the four sets acts where the step says."""
    model, w = tiny_model(seed=94, layer_norm=True)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=95)
    P, _ = model.precompute(ctx, mask)
    ref = model.step(2, tok, src, state, ctx, P, mask)["state"]
    swaps = [{"g1a": "g2a", "be1a": "be2a", "g1u": "g2u", "be1u": "be2u"},
             {"g1a": "g1u", "be1a": "be1u"}, {"g2a": "g2u", "be2a": "be2u"}]
    for sw in swaps:
        w2 = dict(w)
        for a, b in sw.items():
            w2[a], w2[b] = w[b], w[a]
        m2 = mtref.Model(E_, H_, A_, V_, w2, layer_norm=True)
        got = m2.step(2, tok, src, state, ctx, P, mask)["state"]
        assert np.max(np.abs(got - ref)) > 1e-3, sw


def test_beam_k1_equals_greedy_decoding():
    model, w = tiny_model(seed=20, layer_norm=True)
    ctx, mask, lens, *_ = tiny_batch(B=3, K=1, seed=21)
    P, s0 = model.precompute(ctx, mask)
    tok = np.ones(3, np.int32)
    src = np.arange(3, dtype=np.int32)
    st = s0
    score = np.zeros(3, np.float32)
    for _ in range(6):
        out = model.step(1, tok, src, st, ctx, P, mask)
        t, bp, sc = mtref.topk(1, score, out["logp"])
        assert np.array_equal(t, np.argmax(out["logp"], 1))
        assert np.all(bp == 0)
        tok, st, score = t, out["state"], sc
        src = np.arange(3, dtype=np.int32)


def test_beam_permutation_invariance():
    """Permuting the hypotheses of a sentence (with their states and scores) leaves
    the selected (score, token, source state) multiset unchanged."""
    model, w = tiny_model(seed=22)
    K = 3
    ctx, mask, lens, tok, src, state = tiny_batch(B=2, K=K, seed=23)
    P, _ = model.precompute(ctx, mask)
    rng = np.random.default_rng(24)
    score = -rng.uniform(0, 3, size=2 * K).astype(np.float32)
    out = model.step(K, tok, src, state, ctx, P, mask)
    t1, b1, s1 = mtref.topk(K, score, out["logp"])
    perm = np.concatenate([b * K + rng.permutation(K) for b in range(2)])
    out2 = model.step(K, tok[perm], src[perm], state, ctx, P, mask)
    t2, b2, s2 = mtref.topk(K, score[perm], out2["logp"])
    for b in range(2):
        sl = slice(b * K, (b + 1) * K)
        a = sorted(zip(s1[sl].tolist(), t1[sl].tolist(), src[b * K + b1[sl]].tolist()))
        c = sorted(zip(s2[sl].tolist(), t2[sl].tolist(), src[perm][b * K + b2[sl]].tolist()))
        assert a == c


# --------------------------------------------------------------------------------------
# deep transition (Section 3.1.1: eight GRU blocks per decoder step, attention between
# the first and the second; the blocks past the second have no external input)
# --------------------------------------------------------------------------------------


def torch_transition(h, U, b):
    """A transition block is a GRU block whose input is zero: torch.nn.GRUCell with a
    zero input and bias_ih = b (the input path reduces to its bias)."""
    H = h.size
    cell = torch.nn.GRUCell(1, H, bias=True).double()
    with torch.no_grad():
        cell.weight_ih.fill_(0.37)  # multiplies the zero input: must not matter
        cell.weight_hh.copy_(torch.from_numpy(U.astype(np.float64).T))
        cell.bias_ih.copy_(torch.from_numpy(b.astype(np.float64)))
        cell.bias_hh.zero_()
        out = cell(torch.zeros(1, 1, dtype=torch.float64), torch.from_numpy(h.astype(np.float64))[None])
    return out[0].numpy()


@pytest.mark.parametrize("H", [1, 5, 16])
def test_transition_equals_torch_grucell_with_zero_input(H):
    rng = np.random.default_rng(300 + H)
    h = np.tanh(rnd(H, rng=rng))
    U, b = rnd(H, 3 * H, s=0.7, rng=rng), rnd(3 * H, s=0.5, rng=rng)
    assert np.max(np.abs(mtref.gru_transition(h, U, b) - torch_transition(h, U, b))) <= 1e-12


def test_transition_closed_forms():
    rng = np.random.default_rng(31)
    H = 6
    h = np.tanh(rnd(H, rng=rng))
    b = rnd(3 * H, rng=rng)
    sig = lambda v: 1.0 / (1.0 + np.exp(-v.astype(np.float64)))
    # U = 0: s = (1 - sig(b_z)) tanh(b_h) + sig(b_z) h
    z = sig(b[H:2 * H])
    want = (1 - z) * np.tanh(b[2 * H:].astype(np.float64)) + z * h
    assert np.max(np.abs(mtref.gru_transition(h, np.zeros((H, 3 * H), np.float32), b) - want)) <= 1e-15
    # b_z = +40: the block copies its state whatever U is
    b2 = b.copy()
    b2[H:2 * H] = 40.0
    got = mtref.gru_transition(h, rnd(H, 3 * H, rng=rng), b2)
    assert np.max(np.abs(got - h)) <= 1e-15


def test_ln_transition_zero_weights_gives_shift_gates():
    """u = 0 normalises to its shift beta: r = sig(b_r + beta_r), z = sig(b_z + beta_z),
    hh = tanh(b_h + r beta_h) (the bias stays outside the normalisation)."""
    rng = np.random.default_rng(32)
    H = 5
    h = np.tanh(rnd(H, rng=rng))
    b, g, be = rnd(3 * H, rng=rng), 1 + rnd(3 * H, s=0.2, rng=rng), rnd(3 * H, s=0.5, rng=rng)
    got = mtref.gru_transition(h, np.zeros((H, 3 * H), np.float32), b, ln=(g, be))
    sig = lambda v: 1.0 / (1.0 + np.exp(-v))
    b64, be64 = b.astype(np.float64), be.astype(np.float64)
    r = sig(b64[:H] + be64[:H])
    z = sig(b64[H:2 * H] + be64[H:2 * H])
    want = (1 - z) * np.tanh(b64[2 * H:] + r * be64[2 * H:]) + z * h
    assert np.max(np.abs(got - want)) <= 1e-15


def test_ln_transition_scale_invariance():
    """With layer norm only on the recurrent product, scaling U leaves the block unchanged
    (a normalisation that took the bias inside would not be)."""
    rng = np.random.default_rng(33)
    H = 16
    h = np.tanh(rnd(H, rng=rng))
    U, b = rnd(H, 3 * H, rng=rng), rnd(3 * H, s=0.5, rng=rng)
    g, be = 1 + rnd(3 * H, s=0.1, rng=rng), rnd(3 * H, s=0.1, rng=rng)
    a = mtref.gru_transition(h, U, b, ln=(g, be), eps=1e-12)
    c = mtref.gru_transition(h, (U * 8).astype(np.float32), b, ln=(g, be), eps=1e-12)
    assert np.max(np.abs(a - c)) <= 1e-9


def deep_model(T, seed=40, layer_norm=False, **over):
    rng = np.random.default_rng(seed + 1000)
    H = H_
    extra = dict(Ut=rnd(T, H, 3 * H, s=0.5, rng=rng), btr=rnd(T, 3 * H, s=0.3, rng=rng))
    if layer_norm:
        extra["gtu"] = (1 + rnd(T, 3 * H, s=0.1, rng=rng)).astype(np.float32)
        extra["betu"] = rnd(T, 3 * H, s=0.1, rng=rng)
    extra.update(over)
    _, w = tiny_model(seed=seed, layer_norm=layer_norm)
    w.update(extra)
    return mtref.Model(E_, H_, A_, V_, w, layer_norm=layer_norm, transitions=T), w


@pytest.mark.parametrize("layer_norm", [False, True])
def test_deep_step_with_copying_transitions_equals_shallow(layer_norm):
    T, H = 3, H_
    btr = np.zeros((T, 3 * H), np.float32)
    btr[:, H:2 * H] = 40.0  # z = 1: every transition block copies its state
    deep, w = deep_model(T, seed=41, layer_norm=layer_norm, btr=btr)
    shallow = mtref.Model(E_, H_, A_, V_, w, layer_norm=layer_norm)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=42)
    P, _ = shallow.precompute(ctx, mask)
    a = deep.step(2, tok, src, state, ctx, P, mask)
    b = shallow.step(2, tok, src, state, ctx, P, mask)
    assert np.array_equal(a["state"], b["state"]) and np.array_equal(a["logp"], b["logp"])


def test_deep_step_equals_torch_reexpression():
    """The transition blocks run after GRU block 2 in order, and the readout and the new
    state take the last block's output: the shallow step's state carried through
    torch.nn.GRUCell(0, .) T times, then tanh(s Wt_s + x Wt_y + c Wt_c + bt), log_softmax."""
    T = 2
    deep, w = deep_model(T, seed=43)
    shallow = mtref.Model(E_, H_, A_, V_, w)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=44)
    P, _ = shallow.precompute(ctx, mask)
    a = deep.step(2, tok, src, state, ctx, P, mask, taps=True)
    b = shallow.step(2, tok, src, state, ctx, P, mask, taps=True)
    Tt = lambda v: torch.from_numpy(np.asarray(v, np.float64))
    for m in range(tok.size):
        s = b["state"][m].astype(np.float64)
        for j in range(T):
            s = torch_transition(s, w["Ut"][j], w["btr"][j])
        assert np.max(np.abs(a["state"][m] - s)) <= 1e-6
        t = torch.tanh(Tt(s) @ Tt(w["Wt_s"]) + Tt(w["emb"][tok[m]]) @ Tt(w["Wt_y"]) + Tt(b["c"][m]) @ Tt(w["Wt_c"])
                       + Tt(w["bt"]))
        assert np.max(np.abs(a["t"][m] - t.numpy())) <= 1e-6
        lp = torch.log_softmax(t @ Tt(w["Wo"]) + Tt(w["bo"]), 0)
        assert np.max(np.abs(a["logp"][m] - lp.numpy())) <= 1e-5


# --------------------------------------------------------------------------------------
# ensembles (Section 2.3): the members' log-probabilities combined before one selection
# --------------------------------------------------------------------------------------


def test_ensemble_of_one_member_is_the_member():
    lp = rnd(6, 11)
    assert np.array_equal(mtref.ensemble_logp([lp], [1.0]), lp)


def test_ensemble_of_identical_members_with_unit_weights_is_the_member():
    lp = np.log(np.random.default_rng(50).dirichlet(np.ones(13), size=4)).astype(np.float32)
    out = mtref.ensemble_logp([lp, lp, lp, lp], [0.25] * 4)
    assert np.max(np.abs(out - lp)) == 0.0


def test_ensemble_is_the_weighted_sum_with_torch():
    rng = np.random.default_rng(51)
    lps = [rnd(5, 9, rng=rng) for _ in range(3)]
    w = [0.5, 0.3, 0.2]
    ref = sum(torch.from_numpy(l.astype(np.float64)) * float(np.float32(x)) for l, x in zip(lps, w))
    assert np.max(np.abs(mtref.ensemble_logp(lps, w) - ref.numpy())) <= 1e-6



def test_ensemble_is_log_linear_not_probability_averaging():
    """Two members over V = 3 where the two usual ways of combining disagree on the best token.
    Member 1 puts p = (0.9, 0.099, 0.001), member 2 p = (0.001, 0.5, 0.499); with weights 1/2
    the average of the probabilities, (0.4505, 0.2995, 0.25), prefers token 0, while the
    weighted sum of the log-probabilities, the log of the geometric mean (0.030, 0.222, 0.022)
    up to a constant, prefers token 1.  The combination is the log-linear one: its values are
    the closed forms (ln p1 + ln p2) / 2, and the beam step extends token 1."""
    p1 = np.array([[0.9, 0.099, 0.001]])
    p2 = np.array([[0.001, 0.5, 0.499]])
    lps = [np.log(p1).astype(np.float32), np.log(p2).astype(np.float32)]
    out = mtref.ensemble_logp(lps, [0.5, 0.5])
    closed = [0.5 * (math.log(0.9) + math.log(0.001)), 0.5 * (math.log(0.099) + math.log(0.5)),
              0.5 * (math.log(0.001) + math.log(0.499))]
    assert np.max(np.abs(out[0] - np.array(closed))) <= 1e-6
    averaged = np.log(0.5 * (p1 + p2))[0]
    assert np.min(np.abs(out[0] - averaged)) > 0.2
    tok, bp, sc = mtref.topk(1, np.zeros(1, np.float32), out)
    assert int(tok[0]) == 1 and int(np.argmax(averaged)) == 0


def test_ensemble_beam_of_two_copies_equals_single_model_beam():
    """An ensemble of two copies of one model (weights 1/2, 1/2) selects exactly the single
    model's beam at every step (the step of each member is the same)."""
    model, w = tiny_model(seed=52)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=53)
    P, _ = model.precompute(ctx, mask)
    score = np.zeros(tok.size, np.float32)
    for _ in range(4):
        out = model.step(2, tok, src, state, ctx, P, mask)
        ens = mtref.ensemble_logp([out["logp"], out["logp"]], [0.5, 0.5])
        a = mtref.topk(2, score, out["logp"])
        b = mtref.topk(2, score, ens)
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
        tok, bp, score = a
        src = ((np.arange(tok.size) // 2) * 2 + bp).astype(np.int32)
        state = out["state"]


# --------------------------------------------------------------------------------------
# translation bookkeeping: finished hypotheses on EOS, beam shrink, length-normalised n-best
# --------------------------------------------------------------------------------------


def test_translate_equals_exhaustive_search_when_the_beam_holds_everything():
    """V = 3 (EOS = 0) and K = 16 over 3 steps: the beam never has to drop a hypothesis
    (1 + 2 + 12 = 15 <= 16 sequences), so the n-best list must be every sequence that ends
    in EOS or reaches the last step, each scored path by path with one-row steps (the same
    fp32 additions of the step's log-probabilities), sorted by score / length ** alpha."""
    V, K, T, eos, alpha = 3, 16, 3, 0, 0.6
    rng = np.random.default_rng(60)
    E, H, A = E_, H_, A_
    C = 2 * H
    w = dict(
        emb=rnd(V, E, s=0.5, rng=rng), W1=rnd(E, 3 * H, s=0.5, rng=rng), U1=rnd(H, 3 * H, s=0.5, rng=rng),
        b1=rnd(3 * H, s=0.1, rng=rng), Ua=rnd(C, A, s=0.4, rng=rng), ba=rnd(A, s=0.1, rng=rng),
        Wa=rnd(H, A, s=0.5, rng=rng), va=rnd(A, rng=rng), W2=rnd(C, 3 * H, s=0.4, rng=rng),
        U2=rnd(H, 3 * H, s=0.5, rng=rng), b2=rnd(3 * H, s=0.1, rng=rng), Wt_s=rnd(H, E, s=0.5, rng=rng),
        Wt_y=rnd(E, E, s=0.5, rng=rng), Wt_c=rnd(C, E, s=0.4, rng=rng), bt=rnd(E, s=0.1, rng=rng),
        Wo=rnd(E, V, s=2.0, rng=rng), bo=rnd(V, s=0.5, rng=rng), Wi=rnd(C, H, s=0.4, rng=rng), bi=rnd(H, s=0.1, rng=rng))
    model = mtref.Model(E, H, A, V, w)
    B = 2
    ctx = rnd(B, 4, C, rng=rng)
    mask = np.ones((B, 4), np.float32)
    mask[1, 3] = 0
    tok0 = np.full(B * K, 1, np.int32)
    score0 = np.full(B * K, -np.inf, np.float32)
    score0[::K] = 0.0
    nbest = mtref.translate(model, K, ctx, mask, tok0, score0, T, eos, alpha)
    P, s0 = model.precompute(ctx, mask)
    for b in range(B):
        want = []

        def walk(prefix, tok, state, sc):
            out = model.step(1, np.array([tok], np.int32), np.array([0], np.int32), state[None], ctx[b:b + 1],
                             P[b:b + 1], mask[b:b + 1])
            for v in range(V):
                s = np.float32(sc + out["logp"][0, v])
                seq = prefix + [v]
                if v == eos or len(seq) == T:
                    want.append((float(s) / float(len(seq)) ** alpha, float(s), seq))
                else:
                    walk(seq, v, out["state"][0], s)

        walk([], 1, s0[b], np.float32(0.0))
        assert len(want) == 15 and len(nbest[b]) == 15
        key = lambda e: (-e[0], e[2])
        got, ref = sorted(nbest[b], key=key), sorted(want, key=key)
        for g, r in zip(got, ref):
            assert g[2] == r[2] and g[1] == r[1] and abs(g[0] - r[0]) <= 1e-6 * max(1.0, abs(r[0]))


def test_beam_finish_compacts_in_rank_order_and_shrinks_the_beam():
    K, eos = 5, 7
    tok = np.array([3, 7, 4, 7, 9, 1, 2, 7, 5, 6], np.int32)
    bp = np.array([0, 1, 2, 3, 4, 4, 3, 2, 1, 0], np.int32)
    row = (np.arange(10) // K * K + bp).astype(np.int32)
    score = np.array([-1, -2, -3, -4, -5, -1, -2, -3, -np.inf, -np.inf], np.float32)
    beam = np.array([4, 5], np.int32)  # sentence 0 had finished one hypothesis before
    t_, b_, r_, s_, beam2, fin = mtref.beam_finish(K, 2, eos, 1.0, tok, bp, row, score, beam)
    # sentence 0: ranks 0..3 are hypotheses; ranks 1 and 3 end in EOS; rank 4 is beyond the beam
    assert [f[:2] for f in fin[:2]] == [(0, -2.0), (0, -4.0)] and fin[0][2] == -2.0 / 3
    assert list(t_[:5]) == [3, 4, eos, eos, eos] and list(b_[:5]) == [0, 2, 0, 0, 0]
    assert list(r_[:5]) == [0, 2, 0, 0, 0] and list(s_[:2]) == [-1, -3] and np.all(np.isinf(s_[2:5]))
    # sentence 1: ranks 3, 4 have no finite score (fewer candidates than the beam); rank 2 is EOS
    assert [f[0] for f in fin[2:]] == [1] and fin[2][3] == 2 and fin[2][4] == 2
    assert list(t_[5:7]) == [1, 2] and list(r_[5:7]) == [9, 8] and np.all(np.isinf(s_[7:]))
    assert list(beam2) == [2, 4]
    # final step: every hypothesis finishes
    *_, beam3, fin3 = mtref.beam_finish(K, 2, eos, 1.0, tok, bp, row, score, beam, final=True)
    assert list(beam3) == [0, 2] and len(fin3) == 7


# --------------------------------------------------------------------------------------
# encoder (Encoder::build): bi-directional GRU over the source embeddings
# --------------------------------------------------------------------------------------


def enc_weights(E, H, Vs, seed):
    rng = np.random.default_rng(seed)
    return dict(semb=rnd(Vs, E, s=0.5, rng=rng), Wf=rnd(E, 3 * H, s=0.5, rng=rng), Uf=rnd(H, 3 * H, s=0.5, rng=rng),
                bf=rnd(3 * H, s=0.2, rng=rng), Wb=rnd(E, 3 * H, s=0.5, rng=rng), Ub=rnd(H, 3 * H, s=0.5, rng=rng),
                bb=rnd(3 * H, s=0.2, rng=rng))


def enc(tok, mask, w):
    return mtref.encode(tok, mask, w["semb"], w["Wf"], w["Uf"], w["bf"], w["Wb"], w["Ub"], w["bb"])


def test_encoder_equals_torch_bidirectional_gru():
    """Unpadded sentences: torch.nn.GRU(bidirectional=True) with the same reset-after-product
    cell (bias_ih = b, bias_hh = 0) gives the same context rows."""
    E, H, Vs, B, S = 6, 5, 11, 3, 7
    w = enc_weights(E, H, Vs, 70)
    tok = np.random.default_rng(71).integers(0, Vs, (B, S)).astype(np.int32)
    got = enc(tok, np.ones((B, S), np.float32), w)
    gru = torch.nn.GRU(E, H, batch_first=True, bidirectional=True).double()
    with torch.no_grad():
        for sfx, d in (("", "f"), ("_reverse", "b")):
            getattr(gru, "weight_ih_l0" + sfx).copy_(torch.from_numpy(w["W" + d].astype(np.float64).T))
            getattr(gru, "weight_hh_l0" + sfx).copy_(torch.from_numpy(w["U" + d].astype(np.float64).T))
            getattr(gru, "bias_ih_l0" + sfx).copy_(torch.from_numpy(w["b" + d].astype(np.float64)))
            getattr(gru, "bias_hh_l0" + sfx).zero_()
        ref, _ = gru(torch.from_numpy(w["semb"][tok].astype(np.float64)))
    assert np.max(np.abs(got - ref.numpy())) <= 2e-6


def test_encoder_padding_leaves_valid_rows_unchanged():
    """A sentence padded past its length encodes its valid positions exactly as unpadded
    (the backward direction starts from a zero state at its last valid position)."""
    E, H, Vs = 6, 5, 11
    w = enc_weights(E, H, Vs, 72)
    rng = np.random.default_rng(73)
    L, S = 4, 9
    tok = rng.integers(0, Vs, (1, S)).astype(np.int32)
    mask = (np.arange(S) < L).astype(np.float32)[None]
    a = enc(tok, mask, w)
    b = enc(tok[:, :L], np.ones((1, L), np.float32), w)
    assert np.array_equal(a[:, :L], b)
    # padded positions carry the forward state of the last valid position and the zero
    # backward state
    assert np.array_equal(a[0, L:, :H], np.repeat(b[0, L - 1:, :H], S - L, 0))
    assert np.all(a[0, L:, H:] == 0)


def test_encoder_reversal_swaps_directions():
    E, H, Vs, S = 6, 5, 11, 6
    w = enc_weights(E, H, Vs, 74)
    tok = np.random.default_rng(75).integers(0, Vs, (2, S)).astype(np.int32)
    one = np.ones((2, S), np.float32)
    a = enc(tok, one, w)
    sw = dict(w, Wf=w["Wb"], Uf=w["Ub"], bf=w["bb"], Wb=w["Wf"], Ub=w["Uf"], bb=w["bf"])
    b = enc(tok[:, ::-1].copy(), one, sw)
    assert np.array_equal(a[:, :, :H], b[:, ::-1, H:]) and np.array_equal(a[:, :, H:], b[:, ::-1, :H])


# --------------------------------------------------------------------------------------
# dual-source step (two encoders; the decoder attends to both)
# --------------------------------------------------------------------------------------


def dual_model(seed=80, **over):
    rng = np.random.default_rng(seed + 500)
    H, E, A = H_, E_, A_
    C = 2 * H
    _, w = tiny_model(seed=seed)
    w.update(Ua2=rnd(C, A, s=0.4, rng=rng), ba2=rnd(A, s=0.1, rng=rng), Wa2=rnd(H, A, s=0.5, rng=rng),
             va2=rnd(A, rng=rng), W2=rnd(2 * C, 3 * H, s=0.4, rng=rng), Wt_c=rnd(2 * C, E, s=0.4, rng=rng))
    w.update(over)
    return mtref.Model(E, H, A, V_, w, dual_source=True), w


def second_source(B, S2=5, seed=81):
    rng = np.random.default_rng(seed)
    lens2 = rng.integers(1, S2 + 1, size=B)
    ctx2 = rnd(B, S2, 2 * H_, rng=rng)
    mask2 = (np.arange(S2)[None] < lens2[:, None]).astype(np.float32)
    return ctx2, mask2, lens2


def test_dual_step_with_silent_second_context_equals_single_source():
    """Zero rows for the second context in W2 and Wt_c: the dual step must give the
    single-source step exactly (the second attention then feeds nothing)."""
    H, E = H_, E_
    C = 2 * H
    _, w1 = tiny_model(seed=82)
    dual, wd = dual_model(seed=82, W2=np.concatenate([w1["W2"], np.zeros((C, 3 * H), np.float32)]),
                          Wt_c=np.concatenate([w1["Wt_c"], np.zeros((C, E), np.float32)]))
    single = mtref.Model(E, H, A_, V_, w1)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=83)
    ctx2, mask2, _ = second_source(ctx.shape[0])
    P, _ = single.precompute(ctx, mask)
    P2 = dual.keys2(ctx2, mask2)
    a = dual.step(2, tok, src, state, ctx, P, mask, src2=(ctx2, P2, mask2))
    b = single.step(2, tok, src, state, ctx, P, mask)
    assert np.array_equal(a["state"], b["state"]) and np.array_equal(a["logp"], b["logp"])


def test_dual_zero_va2_gives_masked_mean_of_second_source():
    dual, w = dual_model(seed=84, va2=np.zeros(A_, np.float32))
    ctx, mask, lens, tok, src, state = tiny_batch(seed=85)
    ctx2, mask2, lens2 = second_source(ctx.shape[0], seed=86)
    P, _ = dual.precompute(ctx, mask)
    out = dual.step(2, tok, src, state, ctx, P, mask, taps=True, src2=(ctx2, dual.keys2(ctx2, mask2), mask2))
    C = 2 * H_
    for m in range(tok.size):
        b = m // 2
        want = ctx2[b, :lens2[b]].astype(np.float64).mean(0)
        assert np.max(np.abs(out["c"][m, C:] - want)) <= 1e-6


def test_dual_step_equals_torch_reexpression():
    dual, w = dual_model(seed=87)
    ctx, mask, lens, tok, src, state = tiny_batch(seed=88)
    ctx2, mask2, _ = second_source(ctx.shape[0], seed=89)
    P, _ = dual.precompute(ctx, mask)
    P2 = dual.keys2(ctx2, mask2)
    out = dual.step(2, tok, src, state, ctx, P, mask, src2=(ctx2, P2, mask2))
    Tt = lambda v: torch.from_numpy(np.asarray(v, np.float64))

    def att(q, Pb, Cb, mb, va):
        e = torch.tanh(Tt(Pb) + q) @ Tt(va)
        return torch.softmax(e.masked_fill(Tt(mb) == 0, -math.inf), 0) @ Tt(Cb)

    for m in range(tok.size):
        b = m // 2
        x = w["emb"][tok[m]]
        s1 = torch_gru(x, state[src[m]], w["W1"], w["U1"], w["b1"])
        c1 = att(Tt(s1) @ Tt(w["Wa"]), P[b], ctx[b], mask[b], w["va"])
        c2 = att(Tt(s1) @ Tt(w["Wa2"]), (Tt(ctx2[b]) @ Tt(w["Ua2"]) + Tt(w["ba2"])).numpy(), ctx2[b], mask2[b], w["va2"])
        c = torch.cat([c1, c2])
        s = torch_gru(c.numpy(), s1, w["W2"], w["U2"], w["b2"])
        t = torch.tanh(Tt(s) @ Tt(w["Wt_s"]) + Tt(x) @ Tt(w["Wt_y"]) + c @ Tt(w["Wt_c"]) + Tt(w["bt"]))
        lp = torch.log_softmax(t @ Tt(w["Wo"]) + Tt(w["bo"]), 0)
        assert np.max(np.abs(out["state"][m] - s)) <= 1e-6
        assert np.max(np.abs(out["logp"][m] - lp.numpy())) <= 1e-5


def test_deep_encoder_copying_transitions_equal_shallow_and_torch_per_block():
    """Transition blocks that copy their state (b_z = +40) leave the shallow encoder's
    context; general ones equal torch's GRU cell with a zero input applied per position
    after the input block (one direction, unpadded)."""
    E, H, Vs, B, S, T = 6, 5, 11, 2, 5, 3
    w = enc_weights(E, H, Vs, 76)
    rng = np.random.default_rng(77)
    tok = rng.integers(0, Vs, (B, S)).astype(np.int32)
    mask = np.ones((B, S), np.float32)
    mask[1, 3:] = 0
    copy_b = np.zeros((T, 3 * H), np.float32)
    copy_b[:, H:2 * H] = 40.0
    Ut = rnd(T, H, 3 * H, rng=rng)
    a = mtref.encode(tok, mask, *[w[k] for k in ("semb", "Wf", "Uf", "bf", "Wb", "Ub", "bb")],
                     transitions=(Ut, copy_b, Ut, copy_b))
    assert np.array_equal(a, enc(tok, mask, w))
    bt = rnd(T, 3 * H, s=0.3, rng=rng)
    got = mtref.encode(tok[:1], mask[:1], *[w[k] for k in ("semb", "Wf", "Uf", "bf", "Wb", "Ub", "bb")],
                       transitions=(Ut, bt, Ut, bt))
    h = np.zeros(H)
    for i in range(S):
        h = torch_gru(w["semb"][tok[0, i]], h, w["Wf"], w["Uf"], w["bf"])
        for j in range(T):
            h = torch_transition(h, Ut[j], bt[j])
        assert np.max(np.abs(got[0, i, :H] - h)) <= 1e-6


def enc_ln_params(H, T, seed, g=None):
    """(ga, ba, gu, bu) [2,3H] and, for T > 0, (gt, bt) [2,T,3H]; gains ~1 + N(0, 0.2) unless g."""
    rng = np.random.default_rng(seed)
    gain = (lambda *s: np.full(s, g, np.float32)) if g is not None else (lambda *s: 1 + rnd(*s, s=0.2, rng=rng))
    p = [gain(2, 3 * H), rnd(2, 3 * H, s=0.3, rng=rng), gain(2, 3 * H), rnd(2, 3 * H, s=0.3, rng=rng)]
    if T:
        p += [gain(2, T, 3 * H), rnd(2, T, 3 * H, s=0.3, rng=rng)]
    return tuple(p)


def enc_deep(tok, mask, w, trans=None, ln=None, eps=1e-5):
    return mtref.encode(tok, mask, *[w[k] for k in ("semb", "Wf", "Uf", "bf", "Wb", "Ub", "bb")],
                        transitions=trans, ln=ln, eps=eps)


def test_ln_encoder_zero_gains_give_closed_form():
    """With every layer-norm gain 0 each normalised path is its shift alone, so the gates are
    constants: r = s(ba_r + bu_r), z = s(ba_z + bu_z), n = tanh(ba_n + r bu_n) for the input
    block, and with the transition bias b_t added in place of ba for a transition block.  A
    block then maps h to (1 - z) n + z h; from the zero state the forward direction's state
    after the input block of position i (0-based, unpadded) follows that recursion."""
    E, H, Vs, S, T = 6, 5, 11, 5, 2
    w = enc_weights(E, H, Vs, 78)
    rng = np.random.default_rng(79)
    tok = rng.integers(0, Vs, (1, S)).astype(np.int32)
    Ut = rnd(T, H, 3 * H, rng=rng)
    btf, btb = rnd(T, 3 * H, s=0.3, rng=rng), rnd(T, 3 * H, s=0.3, rng=rng)
    ga, ba, gu, bu, gt, bt = enc_ln_params(H, T, 80, g=0.0)
    got = enc_deep(tok, np.ones((1, S), np.float32), w, (Ut, btf, Ut, btb), (ga, ba, gu, bu, gt, bt))
    sig = lambda v: 1 / (1 + np.exp(-v))

    def block(h, a, u):
        r = sig(a[:H] + u[:H])
        z = sig(a[H:2 * H] + u[H:2 * H])
        n = np.tanh(a[2 * H:] + r * u[2 * H:])
        return (1 - z) * n + z * h

    for d, order, bt_d in ((0, range(S), btf), (1, range(S - 1, -1, -1), btb)):
        h = np.zeros(H)
        for i in order:
            h = block(h, ba[d].astype(np.float64), bu[d].astype(np.float64))
            for j in range(T):
                h = block(h, bt_d[j].astype(np.float64), bt[d, j].astype(np.float64))
            assert np.max(np.abs(got[0, i, d * H:(d + 1) * H] - h)) <= 1e-6


def test_ln_encoder_scale_invariance_and_direction_reversal():
    """Layer norm on both paths of the input block and on the transition blocks' recurrent
    path: scaling Wf, bf, Wb, bb by 3 and Uf, Ub, Utf, Utb by 0.5 leaves the context
    unchanged (with a variance epsilon of 1e-12, which the scaling would otherwise see
    where a state is still small); reversing a sentence with every per-direction
    parameter swapped (layer-norm ones included) swaps the halves exactly."""
    E, H, Vs, S, T = 6, 5, 11, 6, 3
    w = enc_weights(E, H, Vs, 81)
    rng = np.random.default_rng(82)
    tok = rng.integers(0, Vs, (2, S)).astype(np.int32)
    one = np.ones((2, S), np.float32)
    Utf, Utb = rnd(T, H, 3 * H, rng=rng), rnd(T, H, 3 * H, rng=rng)
    btf, btb = rnd(T, 3 * H, s=0.3, rng=rng), rnd(T, 3 * H, s=0.3, rng=rng)
    ln = enc_ln_params(H, T, 83)
    a = enc_deep(tok, one, w, (Utf, btf, Utb, btb), ln, eps=1e-12)
    ws = dict(w, Wf=w["Wf"] * 3, bf=w["bf"] * 3, Wb=w["Wb"] * 3, bb=w["bb"] * 3, Uf=w["Uf"] * 0.5, Ub=w["Ub"] * 0.5)
    b = enc_deep(tok, one, ws, (Utf * 0.5, btf, Utb * 0.5, btb), ln, eps=1e-12)
    assert np.max(np.abs(a - b)) <= 1e-5
    # without layer norm the same scaling changes the context (the pin above has teeth)
    assert np.max(np.abs(enc_deep(tok, one, w, (Utf, btf, Utb, btb)) - enc_deep(tok, one, ws, (Utf * 0.5, btf,
                                                                                                 Utb * 0.5, btb)))) > 1e-2
    sw = dict(w, Wf=w["Wb"], Uf=w["Ub"], bf=w["bb"], Wb=w["Wf"], Ub=w["Uf"], bb=w["bf"])
    lsw = tuple(np.ascontiguousarray(x[::-1]) for x in ln)
    c = enc_deep(tok[:, ::-1].copy(), one, sw, (Utb, btb, Utf, btf), lsw, eps=1e-12)
    assert np.array_equal(a[:, :, :H], c[:, ::-1, H:]) and np.array_equal(a[:, :, H:], c[:, ::-1, :H])


def test_ln_deep_encoder_padding_leaves_valid_rows_unchanged():
    E, H, Vs, T = 6, 5, 11, 3
    w = enc_weights(E, H, Vs, 84)
    rng = np.random.default_rng(85)
    L, S = 3, 8
    tok = rng.integers(0, Vs, (1, S)).astype(np.int32)
    Ut, bt = rnd(T, H, 3 * H, rng=rng), rnd(T, 3 * H, s=0.3, rng=rng)
    ln = enc_ln_params(H, T, 86)
    a = enc_deep(tok, (np.arange(S) < L).astype(np.float32)[None], w, (Ut, bt, Ut, bt), ln)
    b = enc_deep(tok[:, :L], np.ones((1, L), np.float32), w, (Ut, bt, Ut, bt), ln)
    assert np.array_equal(a[:, :L], b)
    assert np.array_equal(a[0, L:, :H], np.repeat(b[0, L - 1:, :H], S - L, 0)) and np.all(a[0, L:, H:] == 0)
