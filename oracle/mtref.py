"""ctypes wrapper around the CPU oracle (mtref.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg.  Needs numpy only; it never imports the GPU
package, and the GPU package never imports it.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mtref.c")
LIB = os.path.join(HERE, "libmtref.so")

_f = C.POINTER(C.c_float)
_d = C.POINTER(C.c_double)
_i = C.POINTER(C.c_int32)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no fast-math, single-threaded)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fno-fast-math", "-shared", "-fPIC",
             "-o", tmp, SRC, "-lm"]
        )
        os.replace(tmp, LIB)
    return LIB


class _Dims(C.Structure):
    _fields_ = [("E", C.c_int32), ("H", C.c_int32), ("A", C.c_int32), ("V", C.c_int32),
                ("layer_norm", C.c_int32), ("tied_output", C.c_int32), ("ln_eps", C.c_double),
                ("transitions", C.c_int32)]


_WNAMES = ["emb", "W1", "U1", "b1", "Ua", "ba", "Wa", "va", "W2", "U2", "b2",
           "Wt_s", "Wt_y", "Wt_c", "bt", "Wo", "bo", "Wi", "bi",
           "g1a", "be1a", "g1u", "be1u", "g2a", "be2a", "g2u", "be2u", "gt", "bet",
           "Ut", "btr", "gtu", "betu", "Ua2", "ba2", "Wa2", "va2"]
_LN_NAMES = ("g1a", "be1a", "g1u", "be1u", "g2a", "be2a", "g2u", "be2u", "gt", "bet")


class _Weights(C.Structure):
    _fields_ = [(n, _f) for n in _WNAMES]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = C.CDLL(LIB)
        L.mtref_layer_norm.argtypes = [C.c_int, _d, _f, _f, C.c_double, _d]
        L.mtref_layer_norm.restype = None
        L.mtref_gru.argtypes = [C.c_int, C.c_int, _d, _d, _f, _f, _f, _f, _f, _f, _f, C.c_double, _d]
        L.mtref_gru.restype = None
        L.mtref_gru_transition.argtypes = [C.c_int, _d, _f, _f, _f, _f, C.c_double, _d]
        L.mtref_gru_transition.restype = None
        L.mtref_attention.argtypes = [C.c_int, C.c_int, C.c_int, _d, _f, _f, _f, _f, _d, _d]
        L.mtref_attention.restype = None
        L.mtref_log_softmax.argtypes = [C.c_int, _d, _d]
        L.mtref_log_softmax.restype = C.c_double
        L.mtref_precompute.argtypes = [C.POINTER(_Dims), C.POINTER(_Weights), C.c_int, C.c_int,
                                       _f, _f, _f, _f]
        L.mtref_precompute.restype = C.c_int
        L.mtref_step.argtypes = [C.POINTER(_Dims), C.POINTER(_Weights), C.c_int, C.c_int, C.c_int,
                                 _i, _i, C.c_int, _f, _f, _f, _f, _f, _f, _f, _f, _f, _f]
        L.mtref_step.restype = C.c_int
        L.mtref_keys2.argtypes = [C.POINTER(_Dims), C.POINTER(_Weights), C.c_int, C.c_int, _f, _f, _f]
        L.mtref_keys2.restype = C.c_int
        L.mtref_step_dual.argtypes = [C.POINTER(_Dims), C.POINTER(_Weights), C.c_int, C.c_int, C.c_int,
                                      _i, _i, C.c_int, _f, _f, _f, _f, C.c_int, _f, _f, _f, _f, _f, _f, _f, _f, _f]
        L.mtref_step_dual.restype = C.c_int
        L.mtref_encode.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, _i, _f, _f, _f, _f, _f, _f, _f, _f, _f]
        L.mtref_encode.restype = C.c_int
        L.mtref_encode_deep.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, _i, _f, _f, _f, _f, _f, _f,
                                        _f, _f, C.c_int, _f, _f, _f, _f, _f, _f, _f, _f, _f, _f,
                                        C.c_double, _f]
        L.mtref_encode_deep.restype = C.c_int
        L.mtref_topk.argtypes = [C.c_int, C.c_int, C.c_int, _f, _f, _i, _i, _f]
        L.mtref_topk.restype = C.c_int
        _lib = L
    return _lib


def _fp(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.dtype == np.float32 and a.flags.c_contiguous
    return a.ctypes.data_as(_f)


def _dp(a: np.ndarray):
    assert a.dtype == np.float64 and a.flags.c_contiguous
    return a.ctypes.data_as(_d)


def _ip(a: np.ndarray):
    assert a.dtype == np.int32 and a.flags.c_contiguous
    return a.ctypes.data_as(_i)


def f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


# ---- stage functions -----------------------------------------------------------


def layer_norm(x, gamma, beta, eps=1e-5) -> np.ndarray:
    x = f64(x)
    y = np.empty_like(x)
    lib().mtref_layer_norm(x.size, _dp(x), _fp(f32(gamma)), _fp(f32(beta)), eps, _dp(y))
    return y


def gru(x, h, W, U, b, ln=None, eps=1e-5) -> np.ndarray:
    """ln: None or (gamma_a, beta_a, gamma_u, beta_u), each [3H]."""
    x, h = f64(x), f64(h)
    W, U, b = f32(W), f32(U), f32(b)
    H = h.size
    assert W.shape == (x.size, 3 * H) and U.shape == (H, 3 * H) and b.shape == (3 * H,)
    out = np.empty(H, np.float64)
    lnp = [None] * 4 if ln is None else [f32(t) for t in ln]
    lib().mtref_gru(x.size, H, _dp(x), _dp(h), _fp(W), _fp(U), _fp(b),
                    *[_fp(t) for t in lnp], eps, _dp(out))
    return out


def gru_transition(h, U, b, ln=None, eps=1e-5) -> np.ndarray:
    """Transition block (no external input); ln: None or (gamma_u, beta_u), each [3H]."""
    h = f64(h)
    U, b = f32(U), f32(b)
    H = h.size
    assert U.shape == (H, 3 * H) and b.shape == (3 * H,)
    out = np.empty(H, np.float64)
    lnp = [None] * 2 if ln is None else [f32(t) for t in ln]
    lib().mtref_gru_transition(H, _dp(h), _fp(U), _fp(b), *[_fp(t) for t in lnp], eps, _dp(out))
    return out


def attention(q, P, Cx, mask, va):
    q, P, Cx, mask, va = f64(q), f32(P), f32(Cx), f32(mask), f32(va)
    S, A = P.shape
    Cd = Cx.shape[1]
    alpha = np.empty(S, np.float64)
    ctx = np.empty(Cd, np.float64)
    lib().mtref_attention(S, A, Cd, _dp(q), _fp(P), _fp(Cx), _fp(mask), _fp(va), _dp(alpha), _dp(ctx))
    return alpha, ctx


def log_softmax(l):
    l = f64(l)
    out = np.empty_like(l)
    lse = lib().mtref_log_softmax(l.size, _dp(l), _dp(out))
    return out, lse


# ---- model ----------------------------------------------------------------------


class Model:
    """Holds the fp32 weights (row-major logical [in x out]) and the dims."""

    def __init__(self, E: int, H: int, A: int, V: int, weights: Dict[str, np.ndarray],
                 layer_norm: bool = False, tied_output: bool = False, ln_eps: float = 1e-5,
                 transitions: int = 0, dual_source: bool = False):
        self.E, self.H, self.A, self.V = E, H, A, V
        self.C = 2 * H
        self.T = transitions
        self.dual = bool(dual_source)
        self.Cc = (2 if self.dual else 1) * 2 * H  # width of the context fed to GRU 2 and the readout
        self.dims = _Dims(E, H, A, V, int(layer_norm), int(tied_output), ln_eps, transitions)
        self._keep = {}
        shapes = {
            "emb": (V, E), "W1": (E, 3 * H), "U1": (H, 3 * H), "b1": (3 * H,),
            "Ua": (2 * H, A), "ba": (A,), "Wa": (H, A), "va": (A,),
            "W2": (2 * H, 3 * H), "U2": (H, 3 * H), "b2": (3 * H,),
            "Wt_s": (H, E), "Wt_y": (E, E), "Wt_c": (2 * H, E), "bt": (E,),
            "Wo": (E, V), "bo": (V,), "Wi": (2 * H, H), "bi": (H,),
        }
        for n in ("g1a", "be1a", "g1u", "be1u", "g2a", "be2a", "g2u", "be2u"):
            shapes[n] = (3 * H,)
        shapes["gt"] = (E,)
        shapes["bet"] = (E,)
        T = transitions
        shapes.update({"Ut": (T, H, 3 * H), "btr": (T, 3 * H), "gtu": (T, 3 * H), "betu": (T, 3 * H)})
        shapes.update({"Ua2": (2 * H, A), "ba2": (A,), "Wa2": (H, A), "va2": (A,)})
        shapes["W2"] = (self.Cc, 3 * H)
        shapes["Wt_c"] = (self.Cc, E)
        ptrs = {}
        for n in _WNAMES:
            a = weights.get(n)
            if n in ("Ut", "btr", "gtu", "betu") and T == 0:
                a = None  # a shallow model reads no transition weights
            if n in ("Ua2", "ba2", "Wa2", "va2") and not self.dual:
                a = None
            if a is None:
                if n in _LN_NAMES and not layer_norm:
                    ptrs[n] = None
                    continue
                if n in ("Ut", "btr", "gtu", "betu") and (T == 0 or (n in ("gtu", "betu") and not layer_norm)):
                    ptrs[n] = None
                    continue
                if n in ("Ua2", "ba2", "Wa2", "va2") and not self.dual:
                    ptrs[n] = None
                    continue
                if n == "Wo" and tied_output:
                    ptrs[n] = None
                    continue
                raise KeyError(n)
            a = f32(a)
            if a.shape != shapes[n]:
                raise ValueError(f"{n}: shape {a.shape} != {shapes[n]}")
            self._keep[n] = a
            ptrs[n] = _fp(a)
        self.w = _Weights(**{n: p for n, p in ptrs.items() if p is not None})

    def precompute(self, ctx, mask):
        ctx, mask = f32(ctx), f32(mask)
        B, S, Cd = ctx.shape
        assert Cd == self.C and mask.shape == (B, S)
        P = np.empty((B, S, self.A), np.float32)
        s0 = np.empty((B, self.H), np.float32)
        rc = lib().mtref_precompute(C.byref(self.dims), C.byref(self.w), B, S, _fp(ctx), _fp(mask),
                                    _fp(P), _fp(s0))
        if rc != 0:
            raise ValueError(f"mtref_precompute: {rc}")
        return P, s0

    def keys2(self, ctx2, mask2):
        ctx2, mask2 = f32(ctx2), f32(mask2)
        B, S, _ = ctx2.shape
        P2 = np.empty((B, S, self.A), np.float32)
        rc = lib().mtref_keys2(C.byref(self.dims), C.byref(self.w), B, S, _fp(ctx2), _fp(mask2), _fp(P2))
        if rc != 0:
            raise ValueError(f"mtref_keys2: {rc}")
        return P2

    def step(self, K, prev_tok, src_row, state_in, ctx, P, mask, want_logp=True,
             want_alpha=False, taps=False, src2=None):
        ctx, P, mask, state_in = f32(ctx), f32(P), f32(mask), f32(state_in)
        prev_tok = np.ascontiguousarray(prev_tok, np.int32)
        src_row = np.ascontiguousarray(src_row, np.int32)
        B, S, _ = ctx.shape
        M = B * K
        assert prev_tok.shape == (M,) and src_row.shape == (M,)
        out = {"state": np.empty((M, self.H), np.float32)}
        if want_logp:
            out["logp"] = np.empty((M, self.V), np.float32)
        if want_alpha:
            out["alpha"] = np.empty((M, S), np.float32)
        if taps:
            out["s1"] = np.empty((M, self.H), np.float32)
            out["c"] = np.empty((M, self.Cc), np.float32)
            out["t"] = np.empty((M, self.E), np.float32)
        tail = (_fp(out["state"]), _fp(out.get("logp")), _fp(out.get("alpha")), _fp(out.get("s1")),
                _fp(out.get("c")), _fp(out.get("t")))
        if self.dual:
            ctx2, P2, mask2 = (f32(a) for a in src2)
            rc = lib().mtref_step_dual(
                C.byref(self.dims), C.byref(self.w), B, K, S, _ip(prev_tok), _ip(src_row),
                state_in.shape[0], _fp(state_in), _fp(ctx), _fp(P), _fp(mask), ctx2.shape[1], _fp(ctx2), _fp(P2),
                _fp(mask2), *tail)
        else:
            rc = lib().mtref_step(
                C.byref(self.dims), C.byref(self.w), B, K, S, _ip(prev_tok), _ip(src_row),
                state_in.shape[0], _fp(state_in), _fp(ctx), _fp(P), _fp(mask), *tail)
        if rc != 0:
            raise ValueError(f"mtref_step: {rc}")
        return out


def ensemble_logp(logps, weights) -> np.ndarray:
    """Ensemble of models decoding the same beams (Section 2.3, ensembling as a meta-algorithm
    of batched beam search): the members' log-probabilities combined before one beam
    selection, out[m, v] = sum_i weights[i] * logp_i[m, v], summed in double in member order
    and stored in fp32.  The members' own states stay separate."""
    assert len(logps) == len(weights) and len(logps) >= 1
    acc = np.zeros(np.shape(logps[0]), np.float64)
    for lp, w in zip(logps, weights):
        acc += float(np.float32(w)) * f32(lp).astype(np.float64)
    return acc.astype(np.float32)


def encode(src_tok, mask, semb, Wf, Uf, bf, Wb, Ub, bb, transitions=None, ln=None, eps=1e-5) -> np.ndarray:
    """Bi-directional GRU encoder: ctx [B, S, 2H] fp32 (see mtref_encode); transitions:
    None or (Utf, btf, Utb, btb) stacked [T,H,3H] / [T,3H] (deep-transition cell); ln: None or
    (ga, ba, gu, bu) [2,3H] and, with transitions, (gt, bt) [2,T,3H] appended (see
    mtref_encode_deep)."""
    src_tok = np.ascontiguousarray(src_tok, np.int32)
    mask = f32(mask)
    semb, Wf, Uf, bf, Wb, Ub, bb = [f32(a) for a in (semb, Wf, Uf, bf, Wb, Ub, bb)]
    B, S = src_tok.shape
    Vs, E = semb.shape
    H = Uf.shape[0]
    out = np.empty((B, S, 2 * H), np.float32)
    if transitions is not None or ln is not None:
        if transitions is not None:
            Utf, btf, Utb, btb = [f32(a) for a in transitions]
            T = Utf.shape[0]
        else:
            Utf = btf = Utb = btb = None
            T = 0
        lnp = [None] * 6 if ln is None else [f32(a) for a in ln] + [None] * (6 - len(ln))
        assert ln is None or len(ln) == (6 if T else 4)
        rc = lib().mtref_encode_deep(E, H, Vs, B, S, _ip(src_tok), _fp(mask), _fp(semb), _fp(Wf), _fp(Uf), _fp(bf),
                                     _fp(Wb), _fp(Ub), _fp(bb), T, _fp(Utf), _fp(btf), _fp(Utb), _fp(btb),
                                     *[_fp(a) for a in lnp], eps, _fp(out))
        if rc != 0:
            raise ValueError(f"mtref_encode_deep: {rc}")
        return out
    rc = lib().mtref_encode(E, H, Vs, B, S, _ip(src_tok), _fp(mask), _fp(semb), _fp(Wf), _fp(Uf), _fp(bf),
                            _fp(Wb), _fp(Ub), _fp(bb), _fp(out))
    if rc != 0:
        raise ValueError(f"mtref_encode: {rc}")
    return out


def topk(K, prev_score, logp):
    prev_score, logp = f32(prev_score), f32(logp)
    M, V = logp.shape
    B = M // K
    tok = np.empty(M, np.int32)
    bp = np.empty(M, np.int32)
    sc = np.empty(M, np.float32)
    rc = lib().mtref_topk(B, K, V, _fp(prev_score), _fp(logp), _ip(tok), _ip(bp), _fp(sc))
    if rc != 0:
        raise ValueError(f"mtref_topk: {rc}")
    return tok, bp, sc


# ---- translation bookkeeping (finished hypotheses, beam shrink, n-best) ----------


def beam_finish(K, t, eos, alpha, tok, bp, row, score, beam, final=False):
    """One step of beam bookkeeping after the selection of step t (Section 2.3 batched beam
    search; Section 3.1.3 decodes to an n-best list of as many hypotheses as the beam).

    Per sentence b, `beam[b]` = K minus the hypotheses it has finished.  Of its ranked
    selection results (rank order, as the selection returns them) the first beam[b] with a
    finite score are its new hypotheses; those whose token is eos (every one if `final`)
    finish, with the normalised score score / (t + 1) ** alpha, and the beam shrinks by one
    for each.  The others move, in rank order, to the leading slots; the remaining slots are
    dead (score -inf, token eos, parent 0, state row b*K) and never extend.

    Returns (tok, bp, row, score, beam, finished) with finished a list of
    (b, score, normalised score, step, parent slot, token) in finishing order."""
    tok, bp, row = [np.array(a, np.int32) for a in (tok, bp, row)]
    score = np.array(score, np.float32)
    beam = np.array(beam, np.int32)
    B = beam.size
    fin = []
    o_tok, o_bp, o_row, o_score = tok.copy(), bp.copy(), row.copy(), score.copy()
    for b in range(B):
        keep = []
        nf = 0
        for r in range(int(beam[b])):
            m = b * K + r
            if not np.isfinite(score[m]):
                continue
            if final or tok[m] == eos:
                norm = float(score[m]) / float(t + 1) ** float(alpha)
                fin.append((b, float(score[m]), norm, t, int(bp[m]), int(tok[m])))
                nf += 1
            else:
                keep.append(m)
        for i in range(K):
            d = b * K + i
            if i < len(keep):
                s = keep[i]
                o_tok[d], o_bp[d], o_row[d], o_score[d] = tok[s], bp[s], row[s], score[s]
            else:
                o_tok[d], o_bp[d], o_row[d], o_score[d] = eos, 0, b * K, -np.inf
        beam[b] -= nf
    return o_tok, o_bp, o_row, o_score, beam, fin


def backtrack(K, hist_tok, hist_bp, b, step, parent, token):
    """Token sequence of a finished hypothesis: its own token at `step`, then its ancestors
    through the recorded (compacted) beams of the earlier steps."""
    seq = [int(token)]
    p = int(parent)
    for s in range(step - 1, -1, -1):
        seq.append(int(hist_tok[s][b * K + p]))
        p = int(hist_bp[s][b * K + p])
    return seq[::-1]


def translate(model, K, ctx, mask, tok0, score0, max_steps, eos, alpha):
    """Batched beam search to finished translations: the oracle's step and selection with
    the bookkeeping above; every hypothesis still alive at the last step finishes there.
    Returns per sentence the n-best list [(normalised score, score, tokens)] sorted by
    normalised score (descending; equal ones keep finishing order)."""
    ctx, mask = f32(ctx), f32(mask)
    B = ctx.shape[0]
    M = B * K
    P, s0 = model.precompute(ctx, mask)
    tok = np.ascontiguousarray(tok0, np.int32)
    score = np.ascontiguousarray(score0, np.float32)
    row = (np.arange(M) // K).astype(np.int32)
    state, nrows = s0, B
    beam = np.full(B, K, np.int32)
    hist_tok, hist_bp, fins = [], [], []
    for t in range(max_steps):
        out = model.step(K, tok, row, state, ctx, P, mask)
        ntok, nbp, nsc = topk(K, score, out["logp"])
        nrow = ((np.arange(M) // K) * K + nbp).astype(np.int32)
        tok, bp, row, score, beam, fin = beam_finish(K, t, eos, alpha, ntok, nbp, nrow, nsc, beam,
                                                     final=(t == max_steps - 1))
        hist_tok.append(tok.copy())
        hist_bp.append(bp.copy())
        fins += fin
        state, nrows = out["state"], M
        if not beam.any():
            break
    nbest = [[] for _ in range(B)]
    for (b, sc, norm, step, parent, token) in fins:
        nbest[b].append((norm, sc, backtrack(K, hist_tok, hist_bp, b, step, parent, token)))
    for b in range(B):
        nbest[b].sort(key=lambda e: -e[0])  # stable: equal scores keep finishing order
    return nbest
