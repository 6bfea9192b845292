"""C-ABI checks that need no GPU: the library loads, exports every declared entry
point, and rejects bad arguments on the host before touching the device."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_1804_00344_amd import mtstep as mt
from paper_1804_00344_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mtstep.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mt_[a-z_]+)\s*\(", src)))


def test_header_declares_the_four_calls():
    names = declared_functions()
    for n in ("mt_load_weights", "mt_precompute_ctx", "mt_decoder_step", "mt_beam_topk"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = mt.lib()
    for n in declared_functions():
        assert hasattr(L, n), n


def _cfg(**kw):
    base = dict(E=32, H=64, A=64, V=1000, layer_norm=False, tied_output=False, k_max=4, gemm="f32")
    base.update(kw)
    gemm = base.pop("gemm")
    E, H, A, V = base.pop("E"), base.pop("H"), base.pop("A"), base.pop("V")
    return mt.make_config(E, H, A, V, gemm=gemm, **base)


def _load_status(cfg, weights):
    w = mt.mt_weights()
    keep = []
    for n, a in weights.items():
        a = np.ascontiguousarray(a, np.float32)
        keep.append(a)
        setattr(w, n, a.ctypes.data_as(C.POINTER(C.c_float)))
    h = C.c_void_p()
    return mt.lib().mt_load_weights(C.byref(cfg), C.byref(w), C.byref(h)), h


@pytest.mark.parametrize("kw,status", [
    (dict(E=24), mt.MT_ERR_SHAPE),
    (dict(H=0), mt.MT_ERR_SHAPE),
    (dict(A=8192), mt.MT_ERR_SHAPE),
    (dict(V=1), mt.MT_ERR_SHAPE),
    (dict(k_max=17), mt.MT_ERR_SHAPE),
    (dict(k_max=0), mt.MT_ERR_SHAPE),
    (dict(V=8, k_max=9), mt.MT_ERR_SHAPE),
    (dict(transitions=-1), mt.MT_ERR_SHAPE),
    (dict(transitions=17), mt.MT_ERR_SHAPE),
    (dict(src_V=100, enc_transitions=-1), mt.MT_ERR_SHAPE),
    (dict(src_V=100, enc_transitions=17), mt.MT_ERR_SHAPE),
    (dict(enc_transitions=3), mt.MT_ERR_ARG),  # encoder transition blocks without an encoder
    (dict(enc_layer_norm=True), mt.MT_ERR_ARG),  # encoder layer norm without an encoder
])
def test_load_weights_rejects_bad_config(kw, status):
    p = synth.PRESETS["tiny_f32"]
    rc, h = _load_status(_cfg(**kw), synth.make_weights(p))
    assert rc == status and not h.value
    assert mt.lib().mt_last_error().decode()


def test_load_weights_rejects_bad_dtype_and_flags():
    w = synth.make_weights(synth.PRESETS["tiny_f32"])
    cfg = _cfg()
    cfg.gemm_dtype = 7
    assert _load_status(cfg, w)[0] == mt.MT_ERR_DTYPE
    cfg = _cfg()
    cfg.layer_norm = 2
    assert _load_status(cfg, w)[0] == mt.MT_ERR_ARG


def test_load_weights_rejects_missing_tensors():
    w = synth.make_weights(synth.PRESETS["tiny_f32"])
    for name in ("emb", "U2", "bo", "Wo"):
        w2 = dict(w)
        del w2[name]
        rc, _ = _load_status(_cfg(), w2)
        assert rc == mt.MT_ERR_ARG
        assert name in mt.lib().mt_last_error().decode()
    # layer norm on but its parameters absent
    rc, _ = _load_status(_cfg(layer_norm=True), w)
    assert rc == mt.MT_ERR_ARG
    # transition blocks requested but their weights absent (or, with layer norm, their gains)
    rc, _ = _load_status(_cfg(transitions=2), w)
    assert rc == mt.MT_ERR_ARG and "Ut" in mt.lib().mt_last_error().decode()
    wd = synth.make_weights(synth.PRESETS["tiny_deep_f32_ln"])
    del wd["gtu"]
    rc, _ = _load_status(_cfg(layer_norm=True, transitions=6), wd)
    assert rc == mt.MT_ERR_ARG and "gtu" in mt.lib().mt_last_error().decode()
    # encoder transition blocks requested but their weights absent
    p = synth.PRESETS["tiny_f32"]
    we = {**w, **synth.make_encoder_weights(p, 100, transitions=3)}
    del we["bteb"]
    rc, _ = _load_status(_cfg(src_V=100, enc_transitions=3), we)
    assert rc == mt.MT_ERR_ARG and "bteb" in mt.lib().mt_last_error().decode()
    we = {**w, **synth.make_encoder_weights(p, 100, transitions=3, layer_norm=True)}
    del we["beteu"]
    rc, _ = _load_status(_cfg(src_V=100, enc_transitions=3, enc_layer_norm=True), we)
    assert rc == mt.MT_ERR_ARG and "beteu" in mt.lib().mt_last_error().decode()
    del we["geu"]
    rc, _ = _load_status(_cfg(src_V=100, enc_layer_norm=True), we)
    assert rc == mt.MT_ERR_ARG and "geu" in mt.lib().mt_last_error().decode()
    # NULL config / weights / out
    L = mt.lib()
    h = C.c_void_p()
    assert L.mt_load_weights(None, None, C.byref(h)) == mt.MT_ERR_ARG
    assert L.mt_load_weights(C.byref(_cfg()), None, None) == mt.MT_ERR_ARG


def test_calls_reject_invalid_handles():
    L = mt.lib()
    assert L.mt_workspace_bytes(None, 1, 1, 1) == 0
    assert L.mt_free(None) == mt.MT_ERR_ARG
    assert L.mt_precompute_ctx(None, 1, 1, None, None, None, None, None, 0, None) == mt.MT_ERR_ARG
    assert L.mt_decoder_step(None, 1, 1, 1, None, None, 1, None, None, None, None, None, None, None, None, None,
                             0, None) == mt.MT_ERR_ARG
    assert L.mt_beam_topk(None, 1, 1, None, None, None, None, None, None, None, 0, None) == mt.MT_ERR_ARG
    assert L.mt_device_errors(None, None) == mt.MT_ERR_ARG
    assert L.mt_ensemble_logp(None, 2, None, None, 1, None, None) == mt.MT_ERR_ARG
    assert L.mt_profile_enable(None, 1) == mt.MT_ERR_ARG
    # a pointer to garbage that is not a handle is rejected by its magic word
    junk = (C.c_uint32 * 64)()
    assert L.mt_profile_enable(C.cast(junk, C.c_void_p), 1) == mt.MT_ERR_ARG
    assert "invalid model handle" in L.mt_last_error().decode()
