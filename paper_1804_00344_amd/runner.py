"""Device-buffer harness around the libmtstep calls (allocation and call order only).

Holds a loaded model, one batch's device inputs (context, mask, attention keys,
start state), a workspace and ping-pong state/beam buffers, and issues
mt_precompute_ctx / mt_decoder_step / mt_beam_topk in decode order.  torch
provides device memory and the stream; all arithmetic runs in libmtstep.
"""
from __future__ import annotations

import contextlib
from typing import Dict, Optional

import numpy as np
import torch

from . import mtstep as mt


class Decoder:
    def __init__(self, E: int, H: int, A: int, V: int, weights: Dict[str, np.ndarray], *, gemm: str = "f32",
                 layer_norm: bool = False, tied_output: bool = False, k_max: int = 16, ln_eps: float = 1e-5,
                 transitions: int = 0, src_V: int = 0, dual_source: bool = False, enc_transitions: int = 0,
                 enc_layer_norm: bool = False, device: str = "cuda:0"):
        self.E, self.H, self.A, self.V, self.C = E, H, A, V, 2 * H
        self.gemm = gemm
        self.device = torch.device(device)
        self.cfg = mt.make_config(E, H, A, V, layer_norm=layer_norm, tied_output=tied_output, k_max=k_max,
                                  gemm=gemm, ln_eps=ln_eps, transitions=transitions, src_V=src_V,
                                  dual_source=dual_source, enc_transitions=enc_transitions,
                                  enc_layer_norm=enc_layer_norm)
        self.dual = bool(dual_source)
        self.S2 = 0
        with torch.cuda.device(self.device):
            self.model = mt.mt_load_weights(self.cfg, weights)
        self.io_dtype = torch.bfloat16 if gemm == "bf16" else torch.float32
        self.reuse_state = True  # the decode loop's steps reuse the previous step's bf16 state copy

    @classmethod
    def from_preset(cls, p, weights, **kw):
        return cls(p.E, p.H, p.A, p.V, weights, gemm=p.gemm, layer_norm=p.layer_norm, k_max=max(p.K, 1),
                   transitions=p.transitions, **kw)

    # ---- batch ------------------------------------------------------------------------
    def set_batch(self, ctx: np.ndarray, mask: np.ndarray, K: int):
        B, S, Cd = ctx.shape
        assert Cd == self.C and mask.shape == (B, S)
        d = self.device
        self.B, self.S, self.K, self.M = B, S, K, B * K
        self.ctx = torch.from_numpy(np.ascontiguousarray(ctx, np.float32)).to(d).to(self.io_dtype).contiguous()
        self.mask = torch.from_numpy(np.ascontiguousarray(mask, np.float32)).to(d)
        self.pctx = torch.empty((B, S, self.A), dtype=self.io_dtype, device=d)
        self.s0 = torch.empty((B, self.H), dtype=torch.float32, device=d)
        nbytes = mt.mt_workspace_bytes(self.model, B, K, S)
        assert nbytes > 0
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=d)
        M = self.M
        self.state = [torch.empty((M, self.H), dtype=torch.float32, device=d) for _ in range(2)]
        self.tok = torch.empty(M, dtype=torch.int32, device=d)
        self.row = torch.empty(M, dtype=torch.int32, device=d)
        self.bp = torch.empty(M, dtype=torch.int32, device=d)
        self.score = torch.empty(M, dtype=torch.float32, device=d)
        self.cur = 0

    def set_source(self, src_tok: np.ndarray, mask: np.ndarray, K: int, stream=None):
        """Batch from source tokens: the context comes from the model's encoder (mt_encode)."""
        B, S = src_tok.shape
        self.set_batch(np.zeros((1, 1, self.C), np.float32), np.ones((1, 1), np.float32), K)  # buffers of the right kind
        d = self.device
        self.B, self.S, self.K, self.M = B, S, K, B * K
        self.src_tok = torch.from_numpy(np.ascontiguousarray(src_tok, np.int32)).to(d)
        self.mask = torch.from_numpy(np.ascontiguousarray(mask, np.float32)).to(d)
        self.ctx = torch.empty((B, S, self.C), dtype=self.io_dtype, device=d)
        self.pctx = torch.empty((B, S, self.A), dtype=self.io_dtype, device=d)
        self.s0 = torch.empty((B, self.H), dtype=torch.float32, device=d)
        nbytes = mt.mt_workspace_bytes(self.model, B, K, S)
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=d)
        self.ews = torch.empty(mt.mt_encode_workspace_bytes(self.model, B, S), dtype=torch.uint8, device=d)
        M = self.M
        self.state = [torch.empty((M, self.H), dtype=torch.float32, device=d) for _ in range(2)]
        self.tok = torch.empty(M, dtype=torch.int32, device=d)
        self.row = torch.empty(M, dtype=torch.int32, device=d)
        self.bp = torch.empty(M, dtype=torch.int32, device=d)
        self.score = torch.empty(M, dtype=torch.float32, device=d)
        self.cur = 0
        self.encode(stream=stream)

    def encode(self, stream=None):
        mt.mt_encode(self.model, self.B, self.S, self.src_tok, self.mask, self.ctx, self.ews, stream=stream)

    def set_second_source(self, ctx2: np.ndarray, mask2: np.ndarray):
        """The second source of a dual-source model (after set_batch / set_source)."""
        B, S2, Cd = ctx2.shape
        assert self.dual and B == self.B and Cd == self.C and mask2.shape == (B, S2)
        d = self.device
        self.S2 = S2
        self.ctx2 = torch.from_numpy(np.ascontiguousarray(ctx2, np.float32)).to(d).to(self.io_dtype).contiguous()
        self.mask2 = torch.from_numpy(np.ascontiguousarray(mask2, np.float32)).to(d)
        self.pctx2 = torch.empty((B, S2, self.A), dtype=self.io_dtype, device=d)
        need = mt.mt_workspace_bytes(self.model, B, self.K, S2)
        if need > self.ws.numel():
            self.ws = torch.empty(need, dtype=torch.uint8, device=d)

    def precompute(self, stream=None):
        mt.mt_precompute_ctx(self.model, self.B, self.S, self.ctx, self.mask, self.pctx, self.s0, self.ws,
                             stream=stream)
        if self.dual:
            mt.mt_precompute_keys2(self.model, self.B, self.S2, self.ctx2, self.mask2, self.pctx2, self.ws,
                                   stream=stream)

    def step(self, prev_tok, src_row, state_in, n_state_rows: int, state_out, *, logp=None, attn=None,
             taps=None, stream=None):
        if self.dual:
            mt.mt_decoder_step_dual(self.model, self.B, self.K, self.S, prev_tok, src_row, n_state_rows, state_in,
                                    self.ctx, self.pctx, self.mask, self.S2, self.ctx2, self.pctx2, self.mask2,
                                    state_out, logp_out=logp, attn_out=attn, taps=taps, ws=self.ws, stream=stream)
            return
        mt.mt_decoder_step(self.model, self.B, self.K, self.S, prev_tok, src_row, n_state_rows, state_in, self.ctx,
                           self.pctx, self.mask, state_out, logp_out=logp, attn_out=attn, taps=taps, ws=self.ws,
                           stream=stream)

    def topk(self, prev_score, logp=None, *, score_out=None, tok_out=None, bp_out=None, row_out=None,
             stream=None):
        score_out = self.score if score_out is None else score_out
        tok_out = self.tok if tok_out is None else tok_out
        bp_out = self.bp if bp_out is None else bp_out
        row_out = self.row if row_out is None else row_out
        mt.mt_beam_topk(self.model, self.B, self.K, prev_score, logp, score_out, tok_out, bp_out, row_out,
                        ws=self.ws, stream=stream)
        return score_out, tok_out, bp_out, row_out

    # ---- decode loop ------------------------------------------------------------------
    def start(self, tok0: np.ndarray, score0: np.ndarray):
        """Beam start: every row reads its sentence's start state (src_row = m // K).

        The start beam is staged on the device once per (tok0, score0) pair; later starts
        are device-to-device copies on the stream, so a new decode does not synchronise."""
        d = self.device
        tok0 = np.ascontiguousarray(tok0, np.int32)
        score0 = np.ascontiguousarray(score0, np.float32)
        key = (self.M, tok0.tobytes(), score0.tobytes())
        if getattr(self, "_start_key", None) != key:
            self._start_tok = torch.from_numpy(tok0).to(d)
            self._start_score = torch.from_numpy(score0).to(d)
            self._start_row = torch.arange(self.M, dtype=torch.int32, device=d) // self.K
            self._start_key = key
        self.tok.copy_(self._start_tok)
        self.row.copy_(self._start_row)
        self.score.copy_(self._start_score)
        self.first = True

    @contextlib.contextmanager
    def _reuse(self):
        """Within the decode loop the state a step reads is the previous step's output, which
        nothing else writes: a bf16 model's step may take the copy of it the previous step
        left in the workspace (mt_set_state_reuse), for that call only."""
        on = self.reuse_state and self.gemm == "bf16" and not self.first
        if on:
            mt.mt_set_state_reuse(self.model, True)
        try:
            yield
        finally:
            if on:
                mt.mt_set_state_reuse(self.model, False)

    def advance(self, *, logp=None, attn=None, stream=None):
        """One beam-search step: decoder step on the current beam, then top-K in place."""
        if self.first:
            state_in, nrows = self.s0, self.B
        else:
            state_in, nrows = self.state[self.cur], self.M
        out = self.state[1 - self.cur] if not self.first else self.state[self.cur]
        with self._reuse():
            self.step(self.tok, self.row, state_in, nrows, out, logp=logp, attn=attn, stream=stream)
        self.topk(self.score, None, stream=stream)
        if not self.first:
            self.cur = 1 - self.cur
        self.first = False
        return self.state[self.cur]


def translate(dec: "Decoder", tok0, score0, max_steps: int, eos: int, alpha: float, check_every: int = 4,
              stream=None):
    """Batched beam search to finished translations: steps, selections and the device-side
    bookkeeping (mt_beam_finish) until every sentence has finished its K hypotheses or
    max_steps is reached (the last step finishes every live one).  The host looks at the
    beams every `check_every` steps (one synchronisation) to stop early.  Returns
    (n-best lists per sentence [(normalised score, score, tokens)], steps run)."""
    d, B, K, M = dec.device, dec.B, dec.K, dec.M
    dec.precompute(stream=stream)
    dec.start(tok0, score0)
    beam = torch.full((B,), K, dtype=torch.int32, device=d)
    fcount = torch.zeros(B, dtype=torch.int32, device=d)
    hist_tok = torch.empty((max_steps, M), dtype=torch.int32, device=d)
    hist_bp = torch.empty((max_steps, M), dtype=torch.int32, device=d)
    fs = torch.empty(M, dtype=torch.float32, device=d)
    fn = torch.empty(M, dtype=torch.float32, device=d)
    fst, fpa, fto = [torch.empty(M, dtype=torch.int32, device=d) for _ in range(3)]
    steps = 0
    for t in range(max_steps):
        dec.advance(stream=stream)
        mt.mt_beam_finish(dec.model, B, K, t, eos, alpha, t == max_steps - 1, dec.tok, dec.bp, dec.row, dec.score,
                          beam, fcount, hist_tok[t], hist_bp[t], fs, fn, fst, fpa, fto, stream=stream)
        steps = t + 1
        if (t + 1) % check_every == 0 and int(beam.sum().item()) == 0:
            break
    # the n-best lists ranked and backtracked on the device (mt_beam_nbest); the host only
    # unpacks them
    order = torch.empty(M, dtype=torch.int32, device=d)
    seq = torch.empty((M, max(steps, 1)), dtype=torch.int32, device=d)
    mt.mt_beam_nbest(dec.model, B, K, steps, hist_tok, hist_bp, fcount, fn, fst, fpa, fto, order, seq, stream=stream)
    fc, od, sq = fcount.cpu().numpy(), order.cpu().numpy(), seq.cpu().numpy()
    fs, fn, fst = fs.cpu().numpy(), fn.cpu().numpy(), fst.cpu().numpy()
    nbest = []
    for b in range(B):
        lst = []
        for r in range(min(int(fc[b]), K)):
            f = b * K + int(od[b * K + r])
            lst.append((float(fn[f]), float(fs[f]), sq[b * K + r, :int(fst[f]) + 1].tolist()))
        nbest.append(lst)
    return nbest, steps


class Ensemble:
    """Members decoding one beam (ensembling, a meta-algorithm of batched beam search), each
    with its own states.  Fused (the default): every member's step adds its weighted logits
    into one buffer (mt_ensemble_step) and one selection subtracts the per-row constant
    sum_i w_i LSE_i (mt_ensemble_topk), selecting from the beam candidates the last member
    collected on the combined values; where the library supports it (joint) the members' steps
    stop after the readout and one vocabulary pass serves them all.  Materialised (fused=False): every member writes its
    log-probabilities, mt_ensemble_logp combines them and mt_beam_topk selects.  Either way the
    first member's beam buffers hold the beam that all members read next."""

    def __init__(self, members, weights, fused=True, joint=None, concurrent=True):
        assert len(members) == len(weights) >= 1
        self.members, self.weights = list(members), [float(x) for x in weights]
        self.lead = self.members[0]
        self.fused = fused
        # fused: one vocabulary pass for all members where the library supports it (no combined
        # buffer), else each member adds its weighted logits into the combined buffer
        ok = fused and mt.mt_ensemble_joint_ok([d.model for d in self.members])
        self.joint = ok if joint is None else bool(joint)
        if self.joint and not ok:
            raise ValueError("the joint vocabulary pass does not support these members")
        # Members whose steps are independent (the joint pass, or materialised log-probabilities)
        # run on streams of their own, so that one member's latency-bound kernels overlap the
        # other's; the per-member fused pass adds into one buffer in member order and stays on
        # the caller's stream.  The streams keep the default priority.
        self.concurrent = concurrent and len(self.members) > 1 and (self.joint or not self.fused)
        dev = self.lead.device
        self.streams = [torch.cuda.Stream(device=dev) for _ in self.members] if self.concurrent else None
        self._ev = [torch.cuda.Event() for _ in range(len(self.members) + 1)] if self.concurrent else None

    def set_batch(self, ctx: np.ndarray, mask: np.ndarray, K: int):
        if self.concurrent:  # the members' old buffers may still be in use on their streams
            torch.cuda.synchronize(self.lead.device)
        for d in self.members:
            d.set_batch(ctx, mask, K)
        self._alloc_logp()

    def _alloc_logp(self):
        lead = self.lead
        if self.concurrent:  # no member stream may still use buffers that are about to be replaced
            torch.cuda.synchronize(lead.device)
        # the fused path needs only the combined buffer, the joint pass not even that
        self.logp = [None if self.fused else torch.empty((lead.M, lead.V), dtype=torch.float32, device=lead.device)
                     for _ in self.members]
        self.comb = None if self.joint else torch.empty((lead.M, lead.V), dtype=torch.float32, device=lead.device)

    def set_source(self, src_tok: np.ndarray, mask: np.ndarray, K: int, stream=None):
        """Batch from source tokens: every member encodes them with its own encoder (mt_encode)
        into its own context, as each member of an ensemble has its own encoder."""
        if self.concurrent:
            torch.cuda.synchronize(self.lead.device)
        for d in self.members:
            d.set_source(src_tok, mask, K, stream=stream)
        self._alloc_logp()

    def encode(self, stream=None):
        for d in self.members:
            d.encode(stream=stream)

    def precompute(self, stream=None):
        for d in self.members:
            d.precompute(stream=stream)

    def start(self, tok0: np.ndarray, score0: np.ndarray):
        for d in self.members:
            d.start(tok0, score0)

    def advance(self, stream=None, row_const=None):
        lead = self.lead
        base = stream if stream is not None else torch.cuda.current_stream(lead.device)
        if self.concurrent:  # the members' streams start after what the caller queued
            self._ev[-1].record(base)
        for i, (d, lp) in enumerate(zip(self.members, self.logp)):
            if d.first:
                state_in, nrows = d.s0, d.B
            else:
                state_in, nrows = d.state[d.cur], d.M
            out = d.state[1 - d.cur] if not d.first else d.state[d.cur]
            st = base
            if self.concurrent:
                st = self.streams[i]
                st.wait_event(self._ev[-1])
            with d._reuse():
                if self.fused:
                    mt.mt_ensemble_step(d.model, i, len(self.members), self.weights[i], d.B, d.K, d.S, lead.tok,
                                        lead.row, nrows, state_in, d.ctx, d.pctx, d.mask, out, self.comb, d.ws,
                                        stream=st)
                else:
                    d.step(lead.tok, lead.row, state_in, nrows, out, logp=lp, stream=st)
            if self.concurrent:
                self._ev[i].record(st)
        if self.concurrent:  # the selection waits for every member
            for i in range(len(self.members)):
                base.wait_event(self._ev[i])
        stream = base
        if self.fused:
            mt.mt_ensemble_topk([d.model for d in self.members], self.weights, [d.ws for d in self.members], lead.B,
                                lead.K, lead.score, self.comb, lead.score, lead.tok, lead.bp, lead.row,
                                row_const_out=row_const, stream=stream)
        else:
            mt.mt_ensemble_logp(lead.model, self.logp, self.weights, lead.M, self.comb, stream=stream)
            lead.topk(lead.score, self.comb, stream=stream)
        for d in self.members:
            if not d.first:
                d.cur = 1 - d.cur
            d.first = False
        return [d.state[d.cur] for d in self.members]
