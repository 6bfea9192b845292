"""C-ABI checks that need no GPU: the library loads, exports every declared entry
point, and rejects bad arguments on the host before touching the device."""
import ctypes as C
import math
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
    return sorted(set(re.findall(r"\b(mt_[a-z0-9_]+)\s*\(", src)))


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


# ------------------------------------------------------------------------------------------
# the fp32 -> bf16 conversion that mt_load_weights applies to a bf16 model's matrices
# ------------------------------------------------------------------------------------------

def _nearest_bf16_exact(x: float):
    """Nearest bf16 value to a finite fp32 value by exact rational arithmetic over the two
    bf16 neighbours (ties to the one with an even significand); None if it overflows."""
    from fractions import Fraction
    if x == 0.0:
        return math.copysign(0.0, x)
    sign = -1 if x < 0 else 1
    a = Fraction(abs(x))
    e = math.frexp(abs(x))[1] - 1          # 2^e <= |x| < 2^(e+1)
    e = max(e, -126)                        # subnormal range shares the smallest exponent
    ulp = Fraction(2) ** (e - 7)            # 8 significand bits (7 stored)
    lo = (a // ulp) * ulp
    hi = lo + ulp
    if a - lo < hi - a:
        r = lo
    elif hi - a < a - lo:
        r = hi
    else:                                   # exact tie: the even multiple of ulp
        r = lo if (lo / ulp) % 2 == 0 else hi
    if r > Fraction(2) ** 127 * (2 - Fraction(2) ** -7):
        return None
    return sign * float(r)


def _bf16_value(bits: int) -> float:
    return float(np.array([bits << 16], np.uint32).view(np.float32)[0])


def test_bf16_conversion_round_to_nearest_even():
    one = 1.0
    cases = [
        one + 2.0 ** -8,                    # halfway between 1 and 1 + 2^-7: ties to even -> 1
        one + 3 * 2.0 ** -8,                # halfway, odd neighbour below -> rounds up to 1 + 2^-6
        one + 2.0 ** -8 + 2.0 ** -20,       # just above the tie -> up
        -(one + 2.0 ** -8),                 # the sign does not change the rule
        3.140625, 1e-40, -1e-42, 2.0 ** -133,  # exact, subnormals
        float(np.float32(3.3895313892515355e38)),  # the largest finite bf16
        0.0, -0.0, 65504.0, 1.0e-3, 123456.7,
    ]
    x = np.array(cases, np.float32)
    got = mt.mt_round_bf16(x)
    for xi, gi in zip(x.tolist(), got.tolist()):
        want = _nearest_bf16_exact(float(np.float32(xi)))
        assert want is not None
        g = _bf16_value(gi)
        assert g == want and math.copysign(1.0, g) == math.copysign(1.0, want), (xi, hex(gi), g, want)
    rng = np.random.default_rng(12)
    r = (rng.standard_normal(2000) * np.exp(rng.uniform(-30, 30, 2000))).astype(np.float32)
    for xi, gi in zip(r.tolist(), mt.mt_round_bf16(r).tolist()):
        assert _bf16_value(gi) == _nearest_bf16_exact(xi), xi


def test_bf16_conversion_special_values():
    bits = np.array([0x7F800000, 0xFF800000, 0x7FC00000, 0x7F800001, 0xFF800123, 0x7F7FFFFF, 0xFF7FFFFF],
                    np.uint32)
    got = mt.mt_round_bf16(bits.view(np.float32)).tolist()
    assert got[0] == 0x7F80 and got[1] == 0xFF80            # +-inf stay infinite
    for g in got[2:5]:                                      # NaNs stay NaN (quiet), never inf
        assert (g & 0x7F80) == 0x7F80 and (g & 0x7F) != 0 and (g & 0x40)
    assert got[4] & 0x8000                                  # a negative NaN keeps its sign
    assert got[5] == 0x7F80 and got[6] == 0xFF80            # the largest floats round past bf16 -> inf
