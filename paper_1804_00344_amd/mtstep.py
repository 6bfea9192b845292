"""ctypes binding of libmtstep (declarations in include/mtstep.h).

Argument marshalling only: every step of the decoder runs in the library's HIP
kernels.  Device buffers are passed as torch tensors (or raw integer device
addresses); streams as torch streams (default: torch's current stream).  The
binding raises if the built library is missing — there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmtstep.so")

MT_OK, MT_ERR_ARG, MT_ERR_SHAPE, MT_ERR_DTYPE, MT_ERR_HIP, MT_ERR_OOM, MT_ERR_STATE, MT_ERR_WORKSPACE = (
    0, -1, -2, -3, -4, -5, -6, -7)
MT_F32, MT_BF16 = 0, 1
KERNELS = ["GEMM_GRU1", "GRU_CELL", "GEMM_S1", "ATTENTION", "GEMM_CTX", "GEMM_READOUT", "READOUT",
           "VOCAB_GEMM", "LSE", "TOPK", "PRECOMPUTE", "VOCAB_THRESHOLD", "GEMM_TRANSITION", "ENSEMBLE",
           "BEAM_FINISH", "ENCODE"]
KERNEL_ID = {n: i for i, n in enumerate(KERNELS)}


class MtError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libmtstep status {status}: {msg}")
        self.status = status


class mt_config(C.Structure):
    _fields_ = [("E", C.c_int32), ("H", C.c_int32), ("A", C.c_int32), ("V", C.c_int32),
                ("layer_norm", C.c_int32), ("tied_output", C.c_int32), ("k_max", C.c_int32),
                ("gemm_dtype", C.c_int32), ("ln_eps", C.c_float), ("dec_transitions", C.c_int32),
                ("src_V", C.c_int32), ("dual_source", C.c_int32), ("enc_transitions", C.c_int32),
                ("enc_layer_norm", C.c_int32)]


WEIGHT_FIELDS = ["emb", "W1", "U1", "b1", "Ua", "ba", "Wa", "va", "W2", "U2", "b2", "Wt_s", "Wt_y",
                 "Wt_c", "bt", "Wo", "bo", "Wi", "bi", "g1a", "be1a", "g1u", "be1u", "g2a", "be2a",
                 "g2u", "be2u", "gt", "bet", "Ut", "btr", "gtu", "betu",
                 "semb", "Wef", "Uef", "bef", "Web", "Ueb", "beb", "Ua2", "ba2", "Wa2", "va2",
                 "Utef", "btef", "Uteb", "bteb", "gea", "bea", "geu", "beu", "gteu", "beteu"]

_fp = C.POINTER(C.c_float)


class mt_weights(C.Structure):
    _fields_ = [(n, _fp) for n in WEIGHT_FIELDS]


class mt_taps(C.Structure):
    _fields_ = [("s1", C.c_void_p), ("c", C.c_void_p), ("t", C.c_void_p)]


_lib = None
_vp = C.c_void_p


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        # The library must run on torch's HIP runtime: its device pointers and streams are
        # torch's.  torch's runtime carries the soname libamdhip64.so.7 but torch names it
        # libamdhip64.so, so loading libmtstep first would bring in a second runtime (the one
        # libmtstep was linked against), which then fails to initialise beside torch's.  With
        # torch loaded first, libmtstep's dependency resolves to the runtime already there.
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                               "(python -m paper_1804_00344_amd.build)")
        L = C.CDLL(LIB_PATH)
        L.mt_last_error.restype = C.c_char_p
        L.mt_last_error.argtypes = []
        L.mt_load_weights.argtypes = [C.POINTER(mt_config), C.POINTER(mt_weights), C.POINTER(_vp)]
        L.mt_free.argtypes = [_vp]
        L.mt_workspace_bytes.argtypes = [_vp, C.c_int, C.c_int, C.c_int]
        L.mt_workspace_bytes.restype = C.c_size_t
        L.mt_precompute_ctx.argtypes = [_vp, C.c_int, C.c_int, _vp, _vp, _vp, _vp, _vp, C.c_size_t, _vp]
        L.mt_precompute_ctx_noalloc.argtypes = [_vp, C.c_int, C.c_int, _vp, _vp, _vp, _vp, _vp]
        L.mt_precompute_ctx_noalloc.restype = C.c_int
        L.mt_decoder_step.argtypes = [_vp, C.c_int, C.c_int, C.c_int, _vp, _vp, C.c_int, _vp, _vp, _vp,
                                      _vp, _vp, _vp, _vp, C.POINTER(mt_taps), _vp, C.c_size_t, _vp]
        L.mt_beam_topk.argtypes = [_vp, C.c_int, C.c_int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, C.c_size_t, _vp]
        L.mt_device_errors.argtypes = [_vp, C.POINTER(C.c_int32)]
        L.mt_ensemble_logp.argtypes = [_vp, C.c_int, C.POINTER(_vp), C.POINTER(C.c_float), C.c_int, _vp, _vp]
        L.mt_precompute_keys2.argtypes = [_vp, C.c_int, C.c_int, _vp, _vp, _vp, _vp, C.c_size_t, _vp]
        L.mt_decoder_step_dual.argtypes = [_vp, C.c_int, C.c_int, C.c_int, _vp, _vp, C.c_int, _vp, _vp, _vp, _vp,
                                           C.c_int, _vp, _vp, _vp, _vp, _vp, _vp, C.POINTER(mt_taps), _vp,
                                           C.c_size_t, _vp]
        L.mt_encode_workspace_bytes.argtypes = [_vp, C.c_int, C.c_int]
        L.mt_encode_workspace_bytes.restype = C.c_size_t
        L.mt_encode.argtypes = [_vp, C.c_int, C.c_int, _vp, _vp, _vp, _vp, C.c_size_t, _vp]
        L.mt_beam_finish.argtypes = [_vp, C.c_int, C.c_int, C.c_int, C.c_int32, C.c_float, C.c_int] + [_vp] * 14
        L.mt_profile_enable.argtypes = [_vp, C.c_uint32]
        L.mt_profile_reset.argtypes = [_vp]
        L.mt_profile_sample.argtypes = [_vp, C.c_uint32]
        L.mt_profile_sample.restype = C.c_int
        L.mt_profile_query.argtypes = [_vp, C.c_int, C.POINTER(C.c_double), C.POINTER(C.c_int64)]
        L.mt_ensemble_step.argtypes = [_vp, C.c_int, C.c_int, C.c_float, C.c_int, C.c_int, C.c_int, _vp, _vp, C.c_int, _vp,
                                       _vp, _vp, _vp, _vp, _vp, _vp, C.c_size_t, _vp]
        L.mt_ensemble_step.restype = C.c_int
        L.mt_ensemble_topk.argtypes = [C.c_int, C.POINTER(_vp), C.POINTER(C.c_float), C.POINTER(_vp),
                                       C.POINTER(C.c_size_t), C.c_int, C.c_int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
        L.mt_ensemble_topk.restype = C.c_int
        L.mt_beam_nbest.argtypes = [_vp, C.c_int, C.c_int, C.c_int] + [_vp] * 9 + [C.c_int, _vp]
        L.mt_beam_nbest.restype = C.c_int
        L.mt_set_state_reuse.argtypes = [_vp, C.c_int]
        L.mt_set_state_reuse.restype = C.c_int
        L.mt_ensemble_joint_ok.argtypes = [C.c_int, C.POINTER(_vp)]
        L.mt_ensemble_joint_ok.restype = C.c_int
        L.mt_recomputed_rows.argtypes = [_vp, C.POINTER(C.c_int64)]
        L.mt_recomputed_rows.restype = C.c_int
        L.mt_round_bf16.argtypes = [_vp, _vp, C.c_size_t]
        L.mt_round_bf16.restype = None
        for f in ("mt_load_weights", "mt_free", "mt_precompute_ctx", "mt_decoder_step", "mt_beam_topk",
                  "mt_ensemble_logp", "mt_beam_finish", "mt_encode", "mt_precompute_keys2", "mt_decoder_step_dual",
                  "mt_device_errors", "mt_profile_enable", "mt_profile_reset", "mt_profile_query"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


def mt_round_bf16(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) of fp32 values, as mt_load_weights converts a bf16 model's
    matrices (host memory, no device)."""
    src = np.ascontiguousarray(x, np.float32)
    dst = np.empty(src.shape, np.uint16)
    lib().mt_round_bf16(src.ctypes.data, dst.ctypes.data, src.size)
    return dst


def _check(rc: int):
    if rc != MT_OK:
        raise MtError(rc, lib().mt_last_error().decode())


def _ptr(x) -> Optional[int]:
    """Device address of a torch tensor (contiguous), an int, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not x.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_config(E, H, A, V, *, layer_norm=False, tied_output=False, k_max=16, gemm="f32", ln_eps=1e-5,
                transitions=0, src_V=0, dual_source=False, enc_transitions=0, enc_layer_norm=False):
    return mt_config(E, H, A, V, int(layer_norm), int(tied_output), k_max,
                     MT_BF16 if gemm == "bf16" else MT_F32, ln_eps, transitions, src_V, int(dual_source),
                     enc_transitions, int(enc_layer_norm))


class Model:
    """Owns an mt_model handle (freed with mt_free)."""

    def __init__(self, handle: int, cfg: mt_config):
        self.handle = handle
        self.cfg = cfg

    def __del__(self):
        if getattr(self, "handle", None):
            try:
                lib().mt_free(self.handle)
            except Exception:
                pass
            self.handle = None


def mt_load_weights(cfg: mt_config, weights: Dict[str, np.ndarray]) -> Model:
    """weights: host fp32 arrays by field name (see mt_weights)."""
    keep = {}
    w = mt_weights()
    for n in WEIGHT_FIELDS:
        a = weights.get(n)
        if a is None:
            continue
        a = np.ascontiguousarray(a, dtype=np.float32)
        keep[n] = a
        setattr(w, n, a.ctypes.data_as(_fp))
    h = _vp()
    _check(lib().mt_load_weights(C.byref(cfg), C.byref(w), C.byref(h)))
    return Model(h.value, cfg)


def mt_ensemble_logp(model: Model, logps, weights, M: int, out, stream=None):
    """out = sum_i weights[i] * logps[i] over [M, V] (device tensors; out may be one of them)."""
    n = len(logps)
    ptrs = (_vp * n)(*[_ptr(x) for x in logps])
    w = (C.c_float * n)(*[float(x) for x in weights])
    _check(lib().mt_ensemble_logp(model.handle, n, ptrs, w, M, _ptr(out), _stream(stream)))


def mt_beam_finish(model: Model, B, K, step, eos, alpha, final, tok, bp, row, score, beam, fin_count, hist_tok,
                   hist_bp, fin_score, fin_norm, fin_step, fin_parent, fin_tok, stream=None):
    _check(lib().mt_beam_finish(model.handle, B, K, step, eos, alpha, int(bool(final)),
                                *[_ptr(x) for x in (tok, bp, row, score, beam, fin_count, hist_tok, hist_bp,
                                                    fin_score, fin_norm, fin_step, fin_parent, fin_tok)],
                                _stream(stream)))


def mt_encode_workspace_bytes(model: Model, B: int, S: int) -> int:
    return int(lib().mt_encode_workspace_bytes(model.handle, B, S))


def mt_encode(model: Model, B, S, src_tok, mask, ctx_out, ws, ws_bytes=None, stream=None):
    ws_bytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().mt_encode(model.handle, B, S, _ptr(src_tok), _ptr(mask), _ptr(ctx_out), _ptr(ws), ws_bytes,
                           _stream(stream)))


def mt_free(model: Model):
    if model.handle:
        _check(lib().mt_free(model.handle))
        model.handle = None


def mt_workspace_bytes(model: Model, B: int, K: int, S: int) -> int:
    return int(lib().mt_workspace_bytes(model.handle, B, K, S))


def mt_precompute_ctx(model: Model, B, S, ctx, mask, pctx_out, s0_out, ws, ws_bytes=None, stream=None):
    ws_bytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().mt_precompute_ctx(model.handle, B, S, _ptr(ctx), _ptr(mask), _ptr(pctx_out), _ptr(s0_out),
                                   _ptr(ws), ws_bytes, _stream(stream)))


def mt_precompute_ctx_noalloc(model: Model, B, S, ctx, mask, pctx_out, s0_out, stream=None):
    _check(lib().mt_precompute_ctx_noalloc(model.handle, B, S, _ptr(ctx), _ptr(mask), _ptr(pctx_out), _ptr(s0_out),
                                           _stream(stream)))


def mt_decoder_step(model: Model, B, K, S, prev_tok, src_row, n_state_rows, state_in, ctx, pctx, mask,
                    state_out, logp_out=None, attn_out=None, taps=None, ws=None, ws_bytes=None, stream=None):
    ws_bytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    tp = None
    if taps:
        tp = mt_taps(_ptr(taps.get("s1")), _ptr(taps.get("c")), _ptr(taps.get("t")))
    _check(lib().mt_decoder_step(model.handle, B, K, S, _ptr(prev_tok), _ptr(src_row), n_state_rows,
                                 _ptr(state_in), _ptr(ctx), _ptr(pctx), _ptr(mask), _ptr(state_out),
                                 _ptr(logp_out), _ptr(attn_out), C.byref(tp) if tp is not None else None,
                                 _ptr(ws), ws_bytes, _stream(stream)))


def mt_decoder_step_dual(model: Model, B, K, S, prev_tok, src_row, n_state_rows, state_in, ctx, pctx, mask, S2,
                         ctx2, pctx2, mask2, state_out, logp_out=None, attn_out=None, taps=None, ws=None,
                         ws_bytes=None, stream=None):
    ws_bytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    tp = None
    if taps:
        tp = mt_taps(_ptr(taps.get("s1")), _ptr(taps.get("c")), _ptr(taps.get("t")))
    _check(lib().mt_decoder_step_dual(model.handle, B, K, S, _ptr(prev_tok), _ptr(src_row), n_state_rows,
                                      _ptr(state_in), _ptr(ctx), _ptr(pctx), _ptr(mask), S2, _ptr(ctx2), _ptr(pctx2),
                                      _ptr(mask2), _ptr(state_out), _ptr(logp_out), _ptr(attn_out),
                                      C.byref(tp) if tp is not None else None, _ptr(ws), ws_bytes, _stream(stream)))


def mt_precompute_keys2(model: Model, B, S2, ctx2, mask2, pctx2_out, ws, ws_bytes=None, stream=None):
    ws_bytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().mt_precompute_keys2(model.handle, B, S2, _ptr(ctx2), _ptr(mask2), _ptr(pctx2_out), _ptr(ws),
                                     ws_bytes, _stream(stream)))


def mt_beam_topk(model: Model, B, K, prev_score, logp, score_out, tok_out, bp_out, row_out=None, ws=None,
                 ws_bytes=None, stream=None):
    ws_bytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().mt_beam_topk(model.handle, B, K, _ptr(prev_score), _ptr(logp), _ptr(score_out), _ptr(tok_out),
                              _ptr(bp_out), _ptr(row_out), _ptr(ws), ws_bytes, _stream(stream)))


def mt_device_errors(model: Model) -> int:
    f = C.c_int32(0)
    _check(lib().mt_device_errors(model.handle, C.byref(f)))
    return int(f.value)


def mt_ensemble_step(model: Model, member, n_members, weight, B, K, S, prev_tok, src_row, n_state_rows, state_in, ctx,
                     pctx, mask, state_out, comb_logits, ws, ws_bytes=None, stream=None):
    ws_bytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    _check(lib().mt_ensemble_step(model.handle, member, n_members, float(weight), B, K, S, _ptr(prev_tok), _ptr(src_row),
                                  n_state_rows, _ptr(state_in), _ptr(ctx), _ptr(pctx), _ptr(mask), _ptr(state_out),
                                  _ptr(comb_logits), _ptr(ws), ws_bytes, _stream(stream)))


def mt_beam_nbest(model: Model, B, K, steps, hist_tok, hist_bp, fin_count, fin_norm, fin_step, fin_parent, fin_tok,
                  order, seq, stream=None):
    ld_seq = seq.shape[1]
    _check(lib().mt_beam_nbest(model.handle, B, K, steps, _ptr(hist_tok), _ptr(hist_bp), _ptr(fin_count),
                               _ptr(fin_norm), _ptr(fin_step), _ptr(fin_parent), _ptr(fin_tok), _ptr(order), _ptr(seq),
                               ld_seq, _stream(stream)))


def mt_set_state_reuse(model: Model, on: bool):
    _check(lib().mt_set_state_reuse(model.handle, 1 if on else 0))


def mt_ensemble_joint_ok(models) -> bool:
    n = len(models)
    hs = (_vp * n)(*[m.handle for m in models])
    return bool(lib().mt_ensemble_joint_ok(n, hs))


def mt_ensemble_topk(models, weights, wss, B, K, prev_score, comb_logits, score_out, tok_out, bp_out, row_out=None,
                     row_const_out=None, stream=None):
    n = len(models)
    hs = (_vp * n)(*[m.handle for m in models])
    ws_ = (C.c_float * n)(*[float(x) for x in weights])
    wp = (_vp * n)(*[_ptr(w) for w in wss])
    wb = (C.c_size_t * n)(*[w.numel() * w.element_size() for w in wss])
    _check(lib().mt_ensemble_topk(n, hs, ws_, wp, wb, B, K, _ptr(prev_score), _ptr(comb_logits), _ptr(score_out),
                                  _ptr(tok_out), _ptr(bp_out), _ptr(row_out), _ptr(row_const_out), _stream(stream)))


def mt_recomputed_rows(model: Model) -> int:
    n = C.c_int64(0)
    _check(lib().mt_recomputed_rows(model.handle, C.byref(n)))
    return int(n.value)


def mt_profile_enable(model: Model, kernels=("VOCAB_GEMM",)):
    """Times the given kernel classes (names or ids) with HIP events; () turns timing off."""
    mask = 0
    for k in kernels:
        mask |= 1 << (KERNEL_ID[k] if isinstance(k, str) else int(k))
    _check(lib().mt_profile_enable(model.handle, mask))


def mt_profile_sample(model: Model, every: int):
    """Times one launch in `every` of each selected class."""
    _check(lib().mt_profile_sample(model.handle, int(every)))


def mt_profile_reset(model: Model):
    _check(lib().mt_profile_reset(model.handle))


def mt_profile_query(model: Model, kernel) -> tuple:
    k = KERNEL_ID[kernel] if isinstance(kernel, str) else int(kernel)
    ms, n = C.c_double(0), C.c_int64(0)
    _check(lib().mt_profile_query(model.handle, k, C.byref(ms), C.byref(n)))
    return float(ms.value), int(n.value)
