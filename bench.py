#!/usr/bin/env python3
"""Throughput of the batched beam-search decoder step on one MI355X.

A bench step is one pass of the whole hot path over the batch: mt_decoder_step
(cGRU 1, attention, cGRU 2, readout, vocabulary GEMM with fused log-sum-exp and
per-tile top-K) followed by mt_beam_topk.  A new decode (mt_precompute_ctx: the
attention keys and the start state, then the start beam) begins whenever the
running step index, warmup steps included, reaches a multiple of preset.steps;
the timed region contains such a restart only if it spans that index (the JSON
line says how many it contained).  Inputs are synthetic and already resident in
HBM when timing starts.

    python bench.py [--steps K] [--warmup W] [--preset nematus_f32]

Prints one JSON line (see README of the driver contract): steps/s for the whole
batch, the dominant kernel's roofline fraction (timed with HIP events on its
launch stream) and the CPU oracle's rate on a bounded sample.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "beam decoder steps/s (B×K hyp-rows/s) + % of HBM BW / bf16 MFMA peak"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}
HBM_GBS = 8000.0
# transcendental issue rate (exp2, rcp): a quarter of the 16 lanes per SIMD per clock, 4 SIMDs
# per CU, 256 CUs at 2.4 GHz
TRANS_TOPS = 256 * 4 * 4 * 2.4e9 / 1e12
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def source_hash(path):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def kernel_work(p, lens, S, nsrc=1):
    """Algorithmic work of each kernel class in one step (summed over its launches): flops of
    the matrix products, HBM bytes of the streaming kernels (every operand read once, every
    result written once; weights of the products are not counted as bytes here), and the
    transcendental operations of the attention (2 per tanh: exp2 and rcp).  Returns
    {class: (bound, amount, unit)}."""
    M, E, H, A, V, C, K = p.M, p.E, p.H, p.A, p.V, p.C, p.K
    es = 4 if p.gemm == "f32" else 2                # operand bytes
    bf_copy = 0 if p.gemm == "f32" else H * 2        # bf16 copy of a new state / s1
    T = p.transitions
    slen = float(sum(int(x) for x in lens))
    w = {}
    w["GEMM_GRU1"] = ("mfma", 2.0 * M * H * 3 * H)
    cell = M * (3 * H * 4 + 3 * H * 4 + H * 4 + H * 4 + bf_copy)   # a, u, h read; state (+bf16) written
    cell_t = M * (3 * H * 4 + H * 4 + H * 4 + bf_copy)            # transition block: u, h, state
    w["GRU_CELL"] = ("hbm", 2.0 * cell + T * cell_t)
    w["GEMM_S1"] = ("mfma", 2.0 * M * H * (nsrc * A + 3 * H))
    attn_bytes = nsrc * slen * (A + C) * es + M * nsrc * A * 4 + M * nsrc * C * es
    w["ATTENTION"] = ("hbm", attn_bytes)
    w["ATTENTION_tanh"] = ("trans", 2.0 * K * slen * A * nsrc)
    w["GEMM_CTX"] = ("mfma", 2.0 * M * nsrc * C * (3 * H + E))
    w["GEMM_READOUT"] = ("mfma", 2.0 * M * H * E)
    w["READOUT"] = ("hbm", M * (E * 4 * 3 + E * es))
    w["VOCAB_GEMM"] = ("mfma", 2.0 * M * E * V)
    w["VOCAB_THRESHOLD"] = ("mfma", 2.0 * M * E * min(V, 2048))
    if T:
        w["GEMM_TRANSITION"] = ("mfma", T * 2.0 * M * H * 3 * H)
    return w


def roof_of(bound, amount, us, gemm):
    if not us:
        return None
    t = us * 1e-6
    if bound == "mfma":
        a = amount / t / 1e12
        return {"bound": "mfma", "achieved": round(a, 2), "peak": PEAK_TFLOPS[gemm], "unit": "TFLOP/s",
                "frac": round(a / PEAK_TFLOPS[gemm], 4)}
    if bound == "hbm":
        a = amount / t / 1e9
        return {"bound": "hbm", "achieved": round(a, 1), "peak": HBM_GBS, "unit": "GB/s", "frac": round(a / HBM_GBS, 4)}
    a = amount / t / 1e12
    return {"bound": "alu", "achieved": round(a, 3), "peak": round(TRANS_TOPS, 3), "unit": "Ttrans/s",
            "frac": round(a / TRANS_TOPS, 4)}


def host_cpu():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count()
    return {"nproc": avail, "cpu_count": os.cpu_count(), "cpu_model": model}


def cpu_baseline(members, ctx, mask, budget_s=15.0, src2=None):
    """The oracle (single-threaded C, double accumulation) on whole sentences of the same
    workload: one precompute + decoder step per member, their combination (ensembles) and
    one top-K per sentence, scaled to full-batch steps/s with the precompute amortised over
    preset.steps steps.  members: [(preset, weights)], the first one's shapes."""
    import numpy as np
    from oracle import mtref
    from paper_1804_00344_amd import synth

    p = members[0][0]
    oms = [mtref.Model(q.E, q.H, q.A, q.V, wq, layer_norm=q.layer_norm, transitions=q.transitions,
                       dual_source=src2 is not None) for q, wq in members]
    ew = [1.0 / len(oms)] * len(oms)
    tok, src, state, score = synth.mid_decode_inputs(p, salt=11)
    t_pre = t_step = 0.0
    n = 0
    t_start = time.perf_counter()
    while n < p.B and (time.perf_counter() - t_start) < budget_s:
        b = n
        rows = slice(b * p.K, (b + 1) * p.K)
        t0 = time.perf_counter()
        Ps = [om.precompute(ctx[b:b + 1], mask[b:b + 1])[0] for om in oms]
        s2 = None
        if src2 is not None:
            c2, m2 = src2[0][b:b + 1], src2[1][b:b + 1]
            s2 = (c2, oms[0].keys2(c2, m2), m2)
        t1 = time.perf_counter()
        lps = [om.step(p.K, tok[rows], (src[rows] - b * p.K).astype(np.int32), state[rows], ctx[b:b + 1], P,
                       mask[b:b + 1], want_alpha=False, src2=s2)["logp"] for om, P in zip(oms, Ps)]
        lp = lps[0] if len(lps) == 1 else mtref.ensemble_logp(lps, ew)
        mtref.topk(p.K, score[rows], lp)
        t2 = time.perf_counter()
        t_pre += t1 - t0
        t_step += t2 - t1
        n += 1
    per_sentence = t_step / n + t_pre / n / p.steps
    steps_per_s = 1.0 / (per_sentence * p.B)
    return {
        "value": steps_per_s,
        "unit": "steps/s",
        "cores": 1,
        "kind": "oracle",
        "host": host_cpu(),
        "sample": f"{n} of {p.B} sentences ({n * p.K} hyp rows), one step each + their start-state precompute "
                  f"amortised over {p.steps} steps; {t_pre + t_step:.1f} s of CPU; scaled linearly to the batch",
        "hyp_rows_per_s": steps_per_s * p.M,
    }


PROF_EVERY = 10  # vocabulary launches per event-timed one in the timed region


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--preset", default="nematus_f32")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--ensemble", type=int, default=1,
                    help="members decoding one beam (seeded weights per member, equal weights)")
    ap.add_argument("--dual", action="store_true",
                    help="dual-source model: a second source (seeded like the first) with its own attention")
    ap.add_argument("--encode", type=int, default=0,
                    help="also time the encoder (mt_encode) over the batch with a source vocabulary of this size")
    ap.add_argument("--enc-transitions", type=int, default=0,
                    help="with --encode: recurrent-only GRU blocks after each direction's input block "
                         "(the deep model's four-block encoder cell: 3)")
    ap.add_argument("--enc-layer-norm", action="store_true",
                    help="with --encode: layer norm inside the encoder's GRU blocks")
    ap.add_argument("--translate", type=int, default=0,
                    help="time whole translations of the batch to n-best lists (this many steps at most; "
                         "EOS = token 0, length normalisation alpha 0.6) instead of a fixed step count")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="also run one device copy of this size (counter calibration under rocprofv3)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(decoding would shard by sentence, with no exchange between GPUs)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1804_00344_amd import mtstep as mt
    from paper_1804_00344_amd import synth
    from paper_1804_00344_amd.runner import Decoder

    p = synth.PRESETS[args.preset]
    cell = (f"deep-transition cGRU ({2 + p.transitions} GRU blocks)" if p.transitions else "shallow cGRU")
    log(f"[bench] preset {p.name}: B={p.B} K={p.K} E={p.E} H={p.H} A={p.A} V={p.V} gemm={p.gemm} ln={p.layer_norm}")
    w = synth.make_weights(p)
    ctx, mask, lens = synth.make_source(p)
    if args.dual:
        w = {**w, **synth.make_dual_weights(p)}
        dec = Decoder(p.E, p.H, p.A, p.V, w, gemm=p.gemm, layer_norm=p.layer_norm, k_max=max(p.K, 1),
                      transitions=p.transitions, dual_source=True)
        dec.set_batch(ctx, mask, p.K)
        ctx2, mask2, lens2 = synth.make_source2(p)
        dec.set_second_source(ctx2, mask2)
        cell = f"dual-source {cell}"
    else:
        dec = Decoder.from_preset(p, w)
        dec.set_batch(ctx, mask, p.K)
    tok0, src0, score0 = synth.start_beam(p)
    stream = torch.cuda.current_stream()
    NE = args.ensemble
    drive = dec
    members = [(p, w)]
    if NE > 1:
        from paper_1804_00344_amd.runner import Ensemble
        decs = [dec]
        for i in range(1, NE):
            pi = dataclasses.replace(p, name=f"{p.name}_m{i}", index=p.index + 100 * i)
            wi = synth.make_weights(pi)
            members.append((pi, wi))
            decs.append(Decoder.from_preset(pi, wi))
        drive = Ensemble(decs, [1.0 / NE] * NE)
        drive.set_batch(ctx, mask, p.K)
        cell = f"ensemble of {NE} {cell}"

    tr = {"translations": 0, "steps": 0, "restarts": 0}

    def run(n, first_index):
        """n steps (or, translating, whole translations until at least n steps); returns the steps run"""
        if args.translate:
            from paper_1804_00344_amd.runner import translate
            done = 0
            while done < n:
                _, ran = translate(dec, tok0, score0, args.translate, 0, 0.6)
                done += ran
                tr["translations"] += 1
                tr["steps"] += ran
            return done
        for i in range(first_index, first_index + n):
            if i % p.steps == 0:
                drive.precompute()
                drive.start(tok0, score0)
                tr["restarts"] += 1
            drive.advance()
        return n

    log("[bench] warmup")
    run(args.warmup, 0)
    torch.cuda.synchronize()
    # the vocabulary launches are timed with HIP events on their stream; an event record makes
    # the stream wait for the work queued before it (a few microseconds on each side of a
    # timed launch), so one launch in PROF_EVERY is timed and the step time stays the step's
    mt.mt_profile_enable(dec.model, ("VOCAB_GEMM",))
    mt.mt_profile_sample(dec.model, PROF_EVERY)
    mt.mt_profile_reset(dec.model)
    log(f"[bench] timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    tr.update(translations=0, steps=0, restarts=0)
    timed_steps = run(args.steps, args.warmup)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    restarts_timed = tr["restarts"]
    vocab_ms, vocab_n = mt.mt_profile_query(dec.model, "VOCAB_GEMM")
    mt.mt_profile_enable(dec.model, ())
    mt.mt_profile_sample(dec.model, 1)
    assert mt.mt_device_errors(dec.model) == 0

    # per-kernel breakdown (separate pass, every class timed)
    mt.mt_profile_enable(dec.model, mt.KERNELS)
    mt.mt_profile_reset(dec.model)
    bsteps = run(min(args.steps, 50), args.warmup + args.steps)
    torch.cuda.synchronize()
    breakdown = {}
    work = kernel_work(p, lens, dec.S, nsrc=2 if args.dual else 1)
    for k in mt.KERNELS:
        ms, n = mt.mt_profile_query(dec.model, k)
        if n:
            us = 1e3 * ms / bsteps
            ent = {"us_per_step": round(us, 2), "launches": n}
            if k in work and NE == 1 and not args.translate:
                r = roof_of(*work[k], us, p.gemm)
                if r:
                    ent["roof"] = r
                if k == "ATTENTION":
                    ent["roof_tanh"] = roof_of(*work["ATTENTION_tanh"], us, p.gemm)
            breakdown[k.lower()] = ent
    mt.mt_profile_enable(dec.model, ())

    # HBM traffic per launch from the counter passes (profiles/traffic.json), for the classes
    # whose kernels the counters were taken on (the source file's hash still matches)
    if os.path.exists(TRAFFIC_FILE):
        tf = json.load(open(TRAFFIC_FILE)).get(p.name, {})
        cls_of = {"GRU_CELL": "gru_cell", "ATTENTION": "attention", "READOUT": "readout", "VOCAB_GEMM": "vocab_gemm",
                  "TOPK": "topk_row_select", "VOCAB_THRESHOLD": "vocab_threshold", "LSE": "lse"}
        for k, cls in cls_of.items():
            ent = breakdown.get(k.lower())
            hits = [e for key, e in tf.items() if key.startswith(cls + "@")]
            if not ent or not hits:
                continue
            e = hits[0]
            src = os.path.join(ROOT, "paper_1804_00344_amd", "csrc", e["source"])
            if os.path.exists(src) and source_hash(src) == e["source_hash"]:
                ent["counter_MB_per_launch"] = round(e["bytes_per_launch"] / 1e6, 3)

    # the materialised selection: mt_beam_topk reading a [M, V] fp32 log-probability matrix
    # (ensembles, or callers that want the log-probabilities), an HBM-bound first level
    topk_mat = None
    if NE == 1 and not args.translate:
        g = torch.Generator(device="cuda").manual_seed(5)
        lp = torch.randn((p.M, p.V), device="cuda", generator=g) - math.log(p.V)
        sc = torch.zeros(p.M, device="cuda")
        so, to, bo_, ro = (torch.empty_like(dec.score), torch.empty_like(dec.tok), torch.empty_like(dec.bp),
                           torch.empty_like(dec.row))
        for _ in range(3):
            dec.topk(sc, lp, score_out=so, tok_out=to, bp_out=bo_, row_out=ro)
        torch.cuda.synchronize()
        mt.mt_profile_enable(dec.model, ("TOPK",))
        mt.mt_profile_reset(dec.model)
        nrep = 20
        for _ in range(nrep):
            dec.topk(sc, lp, score_out=so, tok_out=to, bp_out=bo_, row_out=ro)
        torch.cuda.synchronize()
        ms, n = mt.mt_profile_query(dec.model, "TOPK")
        mt.mt_profile_enable(dec.model, ())
        us = 1e3 * ms / nrep
        topk_mat = {"what": "mt_beam_topk on a materialised [M, V] fp32 log-probability matrix (both levels)",
                    "us_per_call": round(us, 2), "bytes": p.M * p.V * 4,
                    "roof": roof_of("hbm", p.M * p.V * 4, us, p.gemm)}
        del lp

    if args.copy_calib_mib:
        # a plain elementwise kernel of known traffic: reads N MiB, writes N MiB
        src = torch.ones((args.copy_calib_mib << 20) // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()

    steps_per_s = timed_steps / elapsed
    avg_vocab_s = vocab_ms / 1e3 / max(vocab_n, 1)
    # a joint ensemble pass computes every member's logits in one launch
    vocab_members = NE if NE > 1 and getattr(drive, "joint", False) else 1
    flops = 2.0 * p.M * p.E * p.V * vocab_members
    achieved = flops / avg_vocab_s / 1e12
    peak = PEAK_TFLOPS[p.gemm]
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        # HBM bytes per launch from the FETCH_SIZE / WRITE_SIZE passes, valid only while the
        # vocabulary kernel's source is the one the counters were taken on
        tf = json.load(open(TRAFFIC_FILE))
        if vocab_members == 1:
            ent = tf.get(p.name, {}).get("vocab_gemm")
            src_h = source_hash(os.path.join(ROOT, "paper_1804_00344_amd", "csrc", "mt_vocab.hip"))
        else:
            ent = tf.get(f"{p.name}_ens{NE}", {}).get("vocab_joint")
            src_h = source_hash(os.path.join(ROOT, "paper_1804_00344_amd", "csrc", "mt_vocab_joint.hip"))
        if ent and ent.get("source_hash") == src_h:
            traffic = ent["bytes_per_launch"]
    roofline = {
        "kernel": ("vocab_joint (every member's t Wo + bo in one pass, per-member log-sum-exp partials + "
                   "candidates of the combined value)" if vocab_members > 1 else
                   "vocab_gemm (t Wo + bo, fused log-sum-exp partials + per-tile top-K)"),
        "bound": "mfma",
        "achieved": round(achieved, 2),
        "peak": peak,
        "unit": "TFLOP/s",
        "frac": round(achieved / peak, 4),
        "traffic": traffic,
        "avg_launch_us": round(avg_vocab_s * 1e6, 2),
        "flops_per_launch": flops,
        "launches_timed": vocab_n,
        "timed_one_launch_in": PROF_EVERY,
    }
    rec = {
        "metric": METRIC,
        "value": round(steps_per_s, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": timed_steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / timed_steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if p.gemm == "f32" else "bf16",
        "data": "synthetic (seeded; shapes and distributions of the preset)",
        "config": {
            "workload": f"{p.name}: {cell} attention decoder step + beam top-K, B={p.B} sentences, beam K={p.K}, "
                        f"E={p.E}, H={p.H}, C={p.C}, A={p.A}, V={p.V}, padded S={dec.S} (mean len {lens.mean():.1f}), "
                        f"{p.gemm} GEMMs, layer_norm={p.layer_norm}, precompute every {p.steps} steps",
            "B": p.B, "K": p.K, "S": dec.S, "V": p.V, "members": NE, "parallelism": "single GPU",
        },
        "hyp_rows_per_s": round(steps_per_s * p.M, 1),
        "target_tok_per_s": round(steps_per_s * p.B, 1),
        "roofline": roofline,
        "kernels": breakdown,
        "restarts_in_timed_region": restarts_timed,
    }
    if topk_mat:
        rec["topk_materialised"] = topk_mat
    if args.encode:
        # encoder of the same shapes over Zipf source tokens with the batch's lengths
        ew = synth.make_encoder_weights(p, args.encode, transitions=args.enc_transitions,
                                        layer_norm=args.enc_layer_norm)
        encd = Decoder(p.E, p.H, p.A, p.V, {**w, **ew}, gemm=p.gemm, layer_norm=p.layer_norm, k_max=max(p.K, 1),
                       src_V=args.encode, enc_transitions=args.enc_transitions,
                       enc_layer_norm=args.enc_layer_norm)
        src = synth.source_tokens(p, args.encode, lens, dec.S)
        encd.set_source(src, mask, p.K)
        for _ in range(3):
            encd.encode()
        torch.cuda.synchronize()
        reps = 20
        t0 = time.perf_counter()
        for _ in range(reps):
            encd.encode()
        torch.cuda.synchronize()
        e_s = (time.perf_counter() - t0) / reps
        rec["encode"] = {
            "what": "mt_encode of the batch: bi-directional GRU over the padded source (one input product, then "
                    "per position the recurrent products of both directions and two cells, then per "
                    "transition block one more product and two more cells)",
            "src_V": args.encode, "enc_transitions": args.enc_transitions, "enc_layer_norm": args.enc_layer_norm, "padded_S": int(dec.S), "ms_per_batch": round(1e3 * e_s, 3),
            "src_tokens_per_s": round(float(lens.sum()) / e_s, 1),
            "per_decoder_step_us_at_precompute_interval": round(1e6 * e_s / p.steps, 2),
        }
    if args.translate:
        rec["translate"] = {
            "what": "whole translations of the batch to n-best lists of K (steps, selections, bookkeeping, "
                    "an early-exit check every 4 steps, host backtracking), EOS = token 0, alpha = 0.6",
            "max_steps": args.translate, "translations": tr["translations"],
            "mean_steps": round(tr["steps"] / max(tr["translations"], 1), 2),
            "sentences_per_s": round(tr["translations"] * p.B / elapsed, 1),
        }
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        rec["cpu_baseline"] = cpu_baseline(members, ctx, mask, args.cpu_budget,
                                           src2=(ctx2, mask2) if args.dual else None)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
