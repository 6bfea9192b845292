"""Seeded synthetic inputs for the beam-search decoder step.

This module is the only code shared by the product path and the oracle.  It
draws numbers; it does none of the model's arithmetic (no GEMM, no gate, no
softmax, no search).  Every tensor comes from its own counter-free PCG64
stream keyed by (seed base + preset index, crc32(tensor name)), so adding a
tensor never shifts the values of another.

Presets are synthetic stand-ins for the paper's translation setting
(newstest-2017 with a shallow Nematus-style model, Section 3.1.4 / Table 2);
the dataset and trained weights are not available, so shapes, value
distributions and length mixes follow the model description instead:

* weights: Glorot-uniform per logical matrix (each gate block of a fused
  [in x 3H] matrix separately; va as an (A, 1) matrix);
* embeddings N(0, 0.1); encoder context N(0, 1); biases zero;
* layer-norm gains 1 + N(0, 0.05), shifts N(0, 0.05);
* source lengths uniform or lognormal (sigma_log = 0.5, mean as given),
  rounded and clamped to [1, max]; padded length S = longest in the batch;
* step-0 tokens: BOS for the tiny preset, otherwise a bounded Zipf(1.1) over
  ranks 1..V (token id = rank - 1).

For presets whose GEMMs run in bf16, every GEMM operand that is a model
input (weights, embeddings, encoder context) is drawn in fp32 and rounded to
the nearest bf16 value (ties to even), so both sides see identical inputs.
"""
from __future__ import annotations

import dataclasses
import math
import zlib
from typing import Dict, Optional

import numpy as np

SEED_BASE = 180400344
BOS = 1


@dataclasses.dataclass(frozen=True)
class Preset:
    name: str
    index: int
    E: int
    H: int
    A: int
    V: int
    B: int
    K: int
    len_dist: str          # "uniform" or "lognormal"
    len_a: float           # uniform: low; lognormal: mean
    len_b: float           # uniform: high; lognormal: max
    gemm: str              # "f32" or "bf16"
    layer_norm: bool
    steps: int
    start: str             # "bos" or "zipf"
    transitions: int = 0   # recurrent-only GRU blocks after GRU 2 (deep-transition cell)

    @property
    def C(self) -> int:
        return 2 * self.H

    @property
    def M(self) -> int:
        return self.B * self.K


PRESETS: Dict[str, Preset] = {
    p.name: p
    for p in [
        Preset("tiny_f32", 0, 32, 64, 64, 1000, 2, 4, "uniform", 5, 10, "f32", False, 20, "bos"),
        Preset("nematus_f32", 1, 512, 1024, 2048, 50000, 64, 12, "lognormal", 25, 80, "f32", False, 50, "zipf"),
        Preset("nematus_bf16_ln", 2, 512, 1024, 2048, 50000, 64, 12, "lognormal", 25, 80, "bf16", True, 50, "zipf"),
        Preset("vocab85k_bf16_ln", 3, 512, 1024, 2048, 85000, 128, 5, "lognormal", 30, 100, "bf16", True, 60, "zipf"),
        Preset("greedy_bf16_ln", 4, 512, 1024, 2048, 50000, 1024, 1, "lognormal", 25, 80, "bf16", True, 50, "zipf"),
        # tiny dimensions with layer norm and bf16 GEMMs at B=64, K=12: the
        # second reading of "same shapes as config 1" for the bf16+LN preset
        Preset("tiny_bf16_ln", 5, 32, 64, 64, 1000, 64, 12, "uniform", 5, 10, "bf16", True, 50, "zipf"),
        # deep-transition decoder cell (Section 3.1.1): eight GRU blocks per step, attention
        # between the first and the second, layer norm; Nematus sizes, and tiny ones
        Preset("deep_bf16_ln", 6, 512, 1024, 2048, 50000, 64, 12, "lognormal", 25, 80, "bf16", True, 50, "zipf", 6),
        Preset("deep_f32_ln", 7, 512, 1024, 2048, 50000, 64, 12, "lognormal", 25, 80, "f32", True, 50, "zipf", 6),
        Preset("tiny_deep_f32_ln", 8, 32, 64, 64, 1000, 8, 4, "uniform", 5, 10, "f32", True, 20, "zipf", 6),
    ]
}


def rng_for(preset: Preset, tensor: str, salt: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([SEED_BASE + preset.index, zlib.crc32(tensor.encode()), salt])
    return np.random.Generator(np.random.PCG64(ss))


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 value (ties to even), kept as fp32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32)
    # NaN stays NaN (quiet), inf stays inf
    nan = np.isnan(x)
    if nan.any():
        out = out.copy()
        out[nan] = np.float32("nan")
    return out.reshape(x.shape)


def glorot(rng: np.random.Generator, fan_in: int, fan_out: int, shape) -> np.ndarray:
    lim = math.sqrt(6.0 / (fan_in + fan_out))
    return rng.uniform(-lim, lim, size=shape).astype(np.float32)


def _gate_matrix(p: Preset, name: str, fan_in: int) -> np.ndarray:
    """[fan_in, 3H]; each H-wide gate block (r, z, h) drawn as its own matrix."""
    blocks = [glorot(rng_for(p, f"{name}.{g}"), fan_in, p.H, (fan_in, p.H)) for g in "rzh"]
    return np.concatenate(blocks, axis=1)


WEIGHT_NAMES = (
    "emb", "W1", "U1", "b1", "Ua", "ba", "Wa", "va", "W2", "U2", "b2",
    "Wt_s", "Wt_y", "Wt_c", "bt", "Wo", "bo", "Wi", "bi",
)
LN_NAMES = ("g1a", "be1a", "g1u", "be1u", "g2a", "be2a", "g2u", "be2u", "gt", "bet")
# tensors that are GEMM operands (rounded to bf16 for bf16 presets)
GEMM_OPERANDS = ("emb", "W1", "U1", "Ua", "Wa", "W2", "U2", "Wt_s", "Wt_y", "Wt_c", "Wo", "Wi", "Ut")
TRANSITION_NAMES = ("Ut", "btr", "gtu", "betu")  # stacked over the transition blocks


def make_weights(p: Preset, peaked_bias: bool = False, round_operands: bool = True) -> Dict[str, np.ndarray]:
    """All model parameters, fp32, row-major logical [in x out].  round_operands=False keeps
    a bf16 preset's matrices as drawn (fp32 masters), leaving the bf16 conversion to the
    consumer."""
    E, H, C, A, V = p.E, p.H, p.C, p.A, p.V
    w: Dict[str, np.ndarray] = {}
    w["emb"] = rng_for(p, "emb").normal(0.0, 0.1, size=(V, E)).astype(np.float32)
    w["W1"] = _gate_matrix(p, "W1", E)
    w["U1"] = _gate_matrix(p, "U1", H)
    w["b1"] = np.zeros(3 * H, np.float32)
    w["Ua"] = glorot(rng_for(p, "Ua"), C, A, (C, A))
    w["ba"] = np.zeros(A, np.float32)
    w["Wa"] = glorot(rng_for(p, "Wa"), H, A, (H, A))
    w["va"] = glorot(rng_for(p, "va"), A, 1, (A,))
    w["W2"] = _gate_matrix(p, "W2", C)
    w["U2"] = _gate_matrix(p, "U2", H)
    w["b2"] = np.zeros(3 * H, np.float32)
    w["Wt_s"] = glorot(rng_for(p, "Wt_s"), H, E, (H, E))
    w["Wt_y"] = glorot(rng_for(p, "Wt_y"), E, E, (E, E))
    w["Wt_c"] = glorot(rng_for(p, "Wt_c"), C, E, (C, E))
    w["bt"] = np.zeros(E, np.float32)
    w["Wo"] = glorot(rng_for(p, "Wo"), E, V, (E, V))
    if peaked_bias:
        # unigram log-prior of a bounded Zipf(1.1): spreads the log-probs so
        # that beam decisions are not all near-ties
        r = np.arange(1, V + 1, dtype=np.float64)
        pr = r ** -1.1
        w["bo"] = np.log(pr / pr.sum()).astype(np.float32)
    else:
        w["bo"] = np.zeros(V, np.float32)
    w["Wi"] = glorot(rng_for(p, "Wi"), C, H, (C, H))
    w["bi"] = np.zeros(H, np.float32)
    if p.layer_norm:
        for path in ("1a", "1u", "2a", "2u"):
            w["g" + path] = (1.0 + rng_for(p, "g" + path).normal(0, 0.05, 3 * H)).astype(np.float32)
            w["be" + path] = rng_for(p, "be" + path).normal(0, 0.05, 3 * H).astype(np.float32)
        w["gt"] = (1.0 + rng_for(p, "gt").normal(0, 0.05, E)).astype(np.float32)
        w["bet"] = rng_for(p, "bet").normal(0, 0.05, E).astype(np.float32)
    if p.transitions:
        T = p.transitions
        w["Ut"] = np.stack([_gate_matrix(p, f"Ut{j}", H) for j in range(T)])
        w["btr"] = np.zeros((T, 3 * H), np.float32)
        if p.layer_norm:
            w["gtu"] = np.stack([(1.0 + rng_for(p, f"gtu{j}").normal(0, 0.05, 3 * H)).astype(np.float32)
                                 for j in range(T)])
            w["betu"] = np.stack([rng_for(p, f"betu{j}").normal(0, 0.05, 3 * H).astype(np.float32)
                                  for j in range(T)])
    if p.gemm == "bf16" and round_operands:
        for k in GEMM_OPERANDS:
            if k in w:
                w[k] = round_bf16(w[k])
    return w


def source_lengths(p: Preset, B: Optional[int] = None) -> np.ndarray:
    B = p.B if B is None else B
    rng = rng_for(p, "src_len")
    if p.len_dist == "uniform":
        L = rng.integers(int(p.len_a), int(p.len_b) + 1, size=B)
    else:
        sig = 0.5
        mu = math.log(p.len_a) - sig * sig / 2.0
        L = np.rint(rng.lognormal(mu, sig, size=B))
        L = np.clip(L, 1, int(p.len_b))
    return L.astype(np.int32)


def make_source(p: Preset, nan_padding: bool = False, round_operands: bool = True):
    """Encoder output stand-in: (ctx [B,S,C] fp32, mask [B,S] fp32 0/1, lens [B]);
    round_operands=False keeps a bf16 preset's context as drawn."""
    lens = source_lengths(p)
    S = int(p.len_b) if p.len_dist == "uniform" else int(lens.max())
    S = max(S, int(lens.max()))
    ctx = rng_for(p, "ctx").normal(0.0, 1.0, size=(p.B, S, p.C)).astype(np.float32)
    mask = (np.arange(S)[None, :] < lens[:, None]).astype(np.float32)
    if p.gemm == "bf16" and round_operands:
        ctx = round_bf16(ctx)
    if nan_padding:
        ctx = ctx.copy()
        ctx[mask == 0] = np.float32("nan")
    return ctx, mask, lens


def bounded_zipf(rng: np.random.Generator, V: int, n: int, s: float = 1.1) -> np.ndarray:
    """Token ids (rank - 1) from P(rank) proportional to rank^-s over 1..V (inverse CDF)."""
    r = np.arange(1, V + 1, dtype=np.float64)
    cdf = np.cumsum(r ** -s)
    cdf /= cdf[-1]
    u = rng.random(n)
    return np.minimum(np.searchsorted(cdf, u, side="right"), V - 1).astype(np.int32)


def start_beam(p: Preset):
    """Step-0 decoder inputs: (prev_tok [M], src_row [M] into s0 rows, prev_score [M])."""
    M = p.M
    src_row = (np.arange(M) // p.K).astype(np.int32)
    if p.start == "bos":
        tok = np.full(M, BOS, np.int32)
        score = np.full((p.B, p.K), -np.inf, np.float32)
        score[:, 0] = 0.0
        score = score.reshape(M)
    else:
        tok = bounded_zipf(rng_for(p, "tok0"), p.V, M)
        score = np.zeros(M, np.float32)
    return tok, src_row, score


def mid_decode_inputs(p: Preset, salt: int = 0):
    """A synthetic mid-decode step: (prev_tok, src_row, state_in [M,H], prev_score).

    States are tanh of N(0,1) draws (GRU states lie in (-1, 1)); every row's
    source state comes from a hypothesis of its own sentence; scores are
    per-sentence descending partial log-probabilities.
    """
    M, K = p.M, p.K
    rng = rng_for(p, "mid", salt)
    tok = bounded_zipf(rng, p.V, M)
    src_row = ((np.arange(M) // K) * K + rng.integers(0, K, size=M)).astype(np.int32)
    state = np.tanh(rng.normal(0.0, 1.0, size=(M, p.H))).astype(np.float32)
    score = -np.sort(rng.uniform(0.0, 20.0, size=(p.B, K)), axis=1)
    return tok, src_row, state, score.reshape(M).astype(np.float32)


DUAL_NAMES = ("Ua2", "ba2", "Wa2", "va2")


def make_dual_weights(p: Preset) -> Dict[str, np.ndarray]:
    """A second source's attention (Ua2, ba2, Wa2, va2) and the 2C-row W2 and Wt_c that take
    the two contexts side by side; Glorot-uniform like the single-source ones."""
    H, C, A, E = p.H, p.C, p.A, p.E
    w = {"Ua2": glorot(rng_for(p, "Ua2"), C, A, (C, A)), "ba2": np.zeros(A, np.float32),
         "Wa2": glorot(rng_for(p, "Wa2"), H, A, (H, A)), "va2": glorot(rng_for(p, "va2"), A, 1, (A,)),
         "W2": _gate_matrix(p, "W2dual", 2 * C), "Wt_c": glorot(rng_for(p, "Wt_cdual"), 2 * C, E, (2 * C, E))}
    if p.gemm == "bf16":
        for k in ("Ua2", "Wa2", "W2", "Wt_c"):
            w[k] = round_bf16(w[k])
    return w


def make_source2(p: Preset):
    """A second source's encoder output stand-in (ctx2 [B,S2,C], mask2, lens2): lengths and
    values drawn like the first source's, from their own streams."""
    q = dataclasses.replace(p, index=p.index + 1000)
    return make_source(q)


ENCODER_NAMES = ("semb", "Wef", "Uef", "bef", "Web", "Ueb", "beb")
ENCODER_TRANSITION_NAMES = ("Utef", "btef", "Uteb", "bteb")  # stacked over the transition blocks
ENCODER_LN_NAMES = ("gea", "bea", "geu", "beu", "gteu", "beteu")  # forward, backward stacked


def make_encoder_weights(p: Preset, src_V: int, transitions: int = 0, layer_norm: bool = False
                         ) -> Dict[str, np.ndarray]:
    """Bi-directional GRU encoder over a source vocabulary of src_V: embeddings N(0, 0.1),
    gate matrices Glorot-uniform per gate block, zero biases (bf16 presets round the product
    operands to bf16); with transitions = T > 0 also T recurrent-only blocks per direction
    (Glorot-uniform gate matrices, biases N(0, 0.1)); with layer_norm gains 1 + N(0, 0.1) and
    shifts N(0, 0.1) for the input blocks' two paths [2,3H] and the transition blocks'
    recurrent path [2,T,3H]."""
    E, H = p.E, p.H
    w = {"semb": rng_for(p, "semb").normal(0.0, 0.1, size=(src_V, E)).astype(np.float32),
         "Wef": _gate_matrix(p, "Wef", E), "Uef": _gate_matrix(p, "Uef", H), "bef": np.zeros(3 * H, np.float32),
         "Web": _gate_matrix(p, "Web", E), "Ueb": _gate_matrix(p, "Ueb", H), "beb": np.zeros(3 * H, np.float32)}
    if transitions:
        T = transitions
        w["Utef"] = np.stack([_gate_matrix(p, f"Utef{j}", H) for j in range(T)])
        w["Uteb"] = np.stack([_gate_matrix(p, f"Uteb{j}", H) for j in range(T)])
        w["btef"] = rng_for(p, "btef").normal(0.0, 0.1, size=(T, 3 * H)).astype(np.float32)
        w["bteb"] = rng_for(p, "bteb").normal(0.0, 0.1, size=(T, 3 * H)).astype(np.float32)
    if layer_norm:
        r = rng_for(p, "enc_ln")
        T = transitions
        for g, b, shape in (("gea", "bea", (2, 3 * H)), ("geu", "beu", (2, 3 * H)), ("gteu", "beteu", (2, T, 3 * H))):
            if shape[1] == 0:
                continue
            w[g] = (1.0 + r.normal(0.0, 0.1, size=shape)).astype(np.float32)
            w[b] = r.normal(0.0, 0.1, size=shape).astype(np.float32)
    if p.gemm == "bf16":
        for k in ("semb", "Wef", "Uef", "Web", "Ueb", "Utef", "Uteb"):
            if k in w:
                w[k] = round_bf16(w[k])
    return w


def source_tokens(p: Preset, src_V: int, lens: np.ndarray, S: int) -> np.ndarray:
    """Source token ids [B, S]: Zipf(1.1) over src_V at valid positions, 0 at padding."""
    rng = rng_for(p, "src_tok")
    r = np.arange(1, src_V + 1, dtype=np.float64)
    cdf = np.cumsum(r ** -1.1)
    cdf /= cdf[-1]
    tok = np.searchsorted(cdf, rng.random((len(lens), S))).astype(np.int32)
    tok[np.arange(S)[None, :] >= np.asarray(lens)[:, None]] = 0
    return np.minimum(tok, src_V - 1).astype(np.int32)


def with_sizes(p: Preset, **kw) -> Preset:
    return dataclasses.replace(p, **kw)
