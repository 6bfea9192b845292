"""mt_precompute_ctx_noalloc (the precompute with its workspace in the library's static
scratch, for callers that cannot allocate) against mt_precompute_ctx through the C ABI."""
import dataclasses

import numpy as np
import pytest

from paper_1804_00344_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU-only machines
    pytestmark = [pytest.mark.gpu, pytest.mark.skip(reason="no GPU")]
else:
    from paper_1804_00344_amd import mtstep as mt
    from paper_1804_00344_amd.runner import Decoder

DEV = "cuda:0"


def _both(dec, B, S, ctx, mask):
    """(P, s0) of the existing entry point and of the no-alloc one on the same inputs."""
    c = torch.from_numpy(np.ascontiguousarray(ctx, np.float32)).to(DEV).to(dec.io_dtype).contiguous()
    m = torch.from_numpy(np.ascontiguousarray(mask, np.float32)).to(DEV)
    outs = []
    for noalloc in (False, True):
        P = torch.full((B, S, dec.A), 7.0, dtype=dec.io_dtype, device=DEV)  # masked rows are left as they were
        s0 = torch.empty((B, dec.H), dtype=torch.float32, device=DEV)
        if noalloc:
            mt.mt_precompute_ctx_noalloc(dec.model, B, S, c, m, P, s0)
        else:
            ws = torch.empty(mt.mt_workspace_bytes(dec.model, B, 1, S), dtype=torch.uint8, device=DEV)
            mt.mt_precompute_ctx(dec.model, B, S, c, m, P, s0, ws)
        torch.cuda.synchronize()
        outs.append((P.float().cpu().numpy(), s0.cpu().numpy()))
    return outs


@pytest.mark.parametrize("name", ["nematus_f32", "nematus_bf16_ln"])
def test_noalloc_precompute_matches_workspace_entry_point(name):
    p = synth.PRESETS[name]
    w = synth.make_weights(p)
    dec = Decoder.from_preset(p, w)
    ctx, mask, lens = synth.make_source(p)
    B, S = mask.shape
    # two calls in a row, the second on a smaller batch with shorter sources: the scratch holds
    # the first call's contents when the second starts
    q = dataclasses.replace(p, B=13, len_b=37, index=p.index + 500)
    ctx2, mask2, _ = synth.make_source(q)
    for (c, m) in ((ctx, mask), (ctx2, mask2)):
        b_, s_ = m.shape
        (Pw, sw), (Pn, sn) = _both(dec, b_, s_, c, m)
        assert np.array_equal(sw, sn)
        valid = m != 0
        assert np.array_equal(Pw[valid], Pn[valid])
        assert np.all(Pn[~valid] == 7.0)  # rows at masked positions are not written
        print(f"[noalloc] {name} B={b_} S={s_}: P and s0 identical to the workspace entry point", flush=True)


def test_noalloc_precompute_rejects_oversize_and_reports():
    p = synth.PRESETS["tiny_f32"]
    dec = Decoder.from_preset(p, synth.make_weights(p))
    B, S = 4096, 1024   # 4096*128*4 + 4096*1024*4 bytes: more than the 16 MiB scratch
    dummy = torch.empty(16, device=DEV)
    with pytest.raises(mt.MtError) as e:
        mt.mt_precompute_ctx_noalloc(dec.model, B, S, dummy, dummy, dummy, dummy)
    assert e.value.status == mt.MT_ERR_WORKSPACE
