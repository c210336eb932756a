#!/usr/bin/env python3
"""Benchmark: accepted output tokens/s of greedy self-speculative decoding on one MI355X.

A step is one whole decode job of the FlanT5-xl-shaped workload (24 layers, d 2048, 32 heads,
d_ff 5120, vocab 32128, bf16, batch 1): prefill of 8 prompt tokens with 32 visual tokens as the
cross-attention memory, then rounds of gamma=5 draft steps (layers 1..6 + imitation network + LM
head), one verify pass over all 24 layers and greedy acceptance, until 128 tokens are emitted.
Inputs are seeded synthetic tensors already resident in HBM when the timed region starts.

Prints one JSON line.  Besides the headline value it reports the same build's full-depth greedy
decode (the speedup denominator), the acceptance rate, the draft-step time against the HBM
roofline of the bytes a draft step must read, the dominant kernel's roofline (live HIP-event
timing of every launch of the one-row weight-streaming GEMV) and the CPU oracle's throughput on
a bounded sample of the same workload.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c3-flant5-xl]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published


def cross_folded(shape, max_batch: int) -> bool:
    """Whether the library folds the T5 cross-attention of a context into two float32 matrices
    per layer (one-sequence contexts with a supported number of visual keys)."""
    nv = shape.n_visual
    return (shape.arch == "t5" and max_batch == 1 and nv in (8, 16, 32, 64)
            and nv <= shape.d_head and shape.n_heads * nv <= 6144
            and shape.d_model <= 6144)


def draft_step_bytes(shape, k: int, ctx: int, kv_bytes: int = 4, folded: bool = False) -> float:
    """Algorithmic bytes of one batch-1 draft step at context length ctx (weights read once,
    KV of layers 1..k read, one position's K/V written; kv_bytes per cached element).  With the
    cross-attention folded, its two float32 matrices replace the cross query / output weights and
    the visual K/V."""
    we = 2 if shape.dtype == "bf16" else 4
    d, hd, f, V, h = shape.d_model, shape.hd, shape.d_ff, shape.vocab, shape.in_width
    layer = (4 * d * hd + 3 * d * f) * we + 3 * d * 4  # QKVO + FFN + norm gains
    kv = 2 * ctx * hd * kv_bytes + 2 * hd * kv_bytes
    if shape.arch == "t5" and folded:
        layer += 2 * shape.n_heads * shape.n_visual * d * 4 + d * 4
    elif shape.arch == "t5":
        layer += 2 * d * hd * we + d * 4
        kv += 2 * shape.n_visual * hd * kv_bytes
    imit = 2 * d * h * we + (h + 3 * d) * 4
    head = V * d * we + d * 4
    return k * (layer + kv) + imit + head


def verify_bytes(shape, B: int, gamma: int, ctx: int, kv_bytes: int = 4) -> float:
    """Algorithmic bytes of one verify pass (all L layers and the LM head read once; KV of every
    layer read for B sequences at context ctx; gamma+1 positions of K/V written per sequence)."""
    we = 2 if shape.dtype == "bf16" else 4
    d, hd, f, V = shape.d_model, shape.hd, shape.d_ff, shape.vocab
    layer = (4 * d * hd + 3 * d * f) * we + 3 * d * 4
    kv = B * (2 * ctx * hd + 2 * (gamma + 1) * hd) * kv_bytes
    if shape.arch == "t5":
        layer += 2 * d * hd * we + d * 4
        kv += B * 2 * shape.n_visual * hd * kv_bytes
    return shape.n_layers * (layer + kv) + V * d * we + d * 4


MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16 matrix peak, published


def prefill_flops(shape, B: int, P: int) -> float:
    """Algorithmic flops of one prefill: every projection at 2 flops per weight and context row,
    causal self-attention (QK and PV over the lower triangle), T5 cross K/V of the visual rows and
    cross-attention of the prompt rows, the LM head for the last row."""
    d, hd, f, V = shape.d_model, shape.hd, shape.d_ff, shape.vocab
    rows = P + (shape.n_visual if shape.arch == "llama" else 0)
    per_layer = 2.0 * (4 * d * hd + 3 * d * f) * rows + 2.0 * rows * rows * hd
    if shape.arch == "t5":
        nv = shape.n_visual
        per_layer += 2.0 * 2 * d * hd * nv + 2.0 * 2 * d * hd * rows + 4.0 * rows * nv * hd
    return B * (shape.n_layers * per_layer + 2.0 * V * d)


def verify_flops(shape, B: int, gamma: int, ctx: int) -> float:
    """Algorithmic flops of one verify pass: 2 per weight and row for every projection of all L
    layers and the LM head over M = B (gamma + 1) rows, plus attention (QK and PV) over the
    context, and T5 cross-attention over the visual keys."""
    d, hd, f, V = shape.d_model, shape.hd, shape.d_ff, shape.vocab
    M = B * (gamma + 1)
    per_layer = 2.0 * (4 * d * hd + 3 * d * f) * M + 4.0 * M * (ctx + gamma) * hd
    if shape.arch == "t5":
        per_layer += 2.0 * 2 * d * hd * M + 4.0 * M * shape.n_visual * hd
    return shape.n_layers * per_layer + 2.0 * V * d * M


def prefill_timing(dd, pt, vt, reps: int = 3) -> float:
    """Median seconds of one prefill call (HIP events on the decoder's stream)."""
    import numpy as np
    import torch
    from paper_2510_22641_amd import ssd as abi
    B, P = pt.shape
    pending = dd.buf("pending", (B,))
    s = dd.stream
    ts = []
    for _ in range(reps + 1):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        s.wait_stream(torch.cuda.current_stream())
        ev[0].record(s)
        abi.ssd_prefill(dd.ctx, B, P, pt, vt, pending, None)
        ev[1].record(s)
        torch.cuda.synchronize()
        ts.append(ev[0].elapsed_time(ev[1]) * 1e-3)
    return float(np.median(ts[1:]))


def dominant_kernel_name(sh) -> str:
    """rocprof name of the one-row GEMV instantiation that streams the RMS-normalised d_model-wide
    matrices (the kernel the library times while profiling)."""
    d = sh.d_model
    if sh.dtype == "bf16" and 2048 <= d <= 6144 and d % 8 == 0:
        return "gemv1k_kernel<unsigned short, %d, 1>" % ((d + 2047) // 2048)
    pieces = (d + 511) // 512
    kp = 2 if pieces <= 2 else 4 if pieces <= 4 else (12 if 8 < pieces <= 12 else 8)
    return "gemv1_kernel<%s, %d, 1>" % ("unsigned short" if sh.dtype == "bf16" else "float", kp)


# the sources that define the one-row GEMV kernels (their hash ties a counter summary to them)
GEMV_SOURCES = ("device.h", "gemv_common.h", "kernels.h", "linear.hip")


def kernel_sources_sha256() -> str:
    """sha256 over the GEMV kernel sources, concatenated in GEMV_SOURCES order."""
    import hashlib
    h = hashlib.sha256()
    for name in GEMV_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2510_22641_amd", "csrc", name), "rb").read())
    return h.hexdigest()


def counted_traffic(kernel: str):
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3 counter summary
    (FETCH_SIZE and WRITE_SIZE runs scaled by a copy-kernel reading), or None when the summary is
    missing or the kernel sources have changed since the counters were taken."""
    import re
    path = os.path.join(ROOT, "profiles", "gemv1k_c3_flant5_xl_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    if f"`{kernel}`" not in text:
        return None
    fields = dict(re.findall(r"^([a-z_0-9]+): (\S+)$", text, re.M))
    if fields.get("kernel_sources_sha256") != kernel_sources_sha256():
        return None
    return {"bytes": int(fields["traffic_bytes_per_launch"]),
            "algorithmic_bytes": int(fields["algorithmic_bytes_per_launch"]),
            "launches": int(fields["launches"]), "source": os.path.relpath(path, ROOT)}


def step_timings(dd, pt, vt, B: int, g: int, rounds: int = 8):
    """Median per-step draft time and per-pass verify time over a few rounds after prefill (HIP
    events on the decoder's stream around the captured draft and verify graphs)."""
    import numpy as np
    import torch
    from paper_2510_22641_amd import ssd as abi
    pending, _ = dd.prefill(pt, vt)
    s = dd.stream
    dts, vts, ctxs = [], [], []
    for _ in range(rounds):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ctxs.append(int(dd.seq_len[:B].float().mean().item()))
        s.wait_stream(torch.cuda.current_stream())
        d = dd.buf("draft", (B, g))
        ev[0].record(s)
        abi.ssd_draft(dd.ctx, B, g, pending, d, None)
        ev[1].record(s)
        t = dd.buf("target", (B, g + 1))
        abi.ssd_verify(dd.ctx, B, g, pending, d, 1, t, None)
        ev[2].record(s)
        dd.accept(d, t, pending, g)
        torch.cuda.synchronize()
        dts.append(ev[0].elapsed_time(ev[1]) * 1e-3 / g)
        vts.append(ev[1].elapsed_time(ev[2]) * 1e-3)
    return float(np.median(dts)), float(np.median(vts)), int(np.median(ctxs))


def sweep_c4(args):
    """The FlanT5-xl sweep: batch {1, 8} x draft depth {4, 8, 12} x gamma {2, 4, 8} over one
    decoder (deep layers scaled from layer 7 on); one JSON line per point."""
    import torch
    import synth
    from paper_2510_22641_amd import runtime
    pts = synth.c4_points()
    weights = synth.workload_weights(pts[0], args.seed)
    # one context per (draft depth, batch): a one-sequence context folds the cross-attention
    for k, mb in sorted({(p.draft_layers, p.batch) for p in pts}):
        group = [p for p in pts if p.draft_layers == k and p.batch == mb]
        gm = max(p.gamma for p in group)
        dd = runtime.from_workload(group[0], args.seed, weights=weights, max_batch=mb,
                                   max_gamma=gm)
        for wl in group:
            sh, B, T, g = wl.shape, wl.batch, wl.new_tokens, wl.gamma
            prompts = synth.make_prompts(sh, args.seed, B, wl.prompt_len)
            visual = synth.make_visual(sh, args.seed, B)
            pt, vt = dd.upload_inputs(prompts, visual)

            def timed(spec):
                for _ in range(args.warmup):
                    dd.generate(pt, vt, T, g, speculative=spec, reuse=True)
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                for _ in range(args.steps):
                    toks, st = dd.generate(pt, vt, T, g, speculative=spec, reuse=True)
                torch.cuda.synchronize()
                return time.perf_counter() - t0, st, toks

            dt, st, toks = timed(True)
            dtg, _, gtoks = timed(False)
            d_s, v_s, ctx = step_timings(dd, pt, vt, B, g)
            db = draft_step_bytes(sh, k, ctx, dd.k_pool.element_size(), cross_folded(sh, mb))
            db += (B - 1) * 2 * k * (ctx + (sh.n_visual if sh.arch == "t5" else 0)) * sh.hd * \
                dd.k_pool.element_size()
            vb = verify_bytes(sh, B, g, ctx, dd.k_pool.element_size())
            rec = {"workload": wl.name, "batch": B, "draft_layers": k, "gamma": g, "new_tokens": T,
                   "tokens_per_s": round(B * T * args.steps / dt, 2),
                   "greedy_tokens_per_s": round(B * T * args.steps / dtg, 2),
                   "speedup_vs_greedy": round(dtg / dt, 3),
                   "acceptance_rate": round(st["accepted"] / max(1, st["drafted"]), 4),
                   "ssd_equals_greedy_tokens": bool(torch.equal(toks, gtoks)),
                   "draft_step": {"us": round(d_s * 1e6, 2), "bytes": int(db),
                                  "frac": round(db / d_s / 1e9 / HBM_PEAK_GBS, 4)},
                   "verify": {"us": round(v_s * 1e6, 2), "bytes": int(vb),
                              "frac": round(vb / v_s / 1e9 / HBM_PEAK_GBS, 4)}}
            print(json.dumps(rec), flush=True)
        dd.close()
        del dd
        torch.cuda.empty_cache()


def sampled_decode(dd, pt, vt, T: int, gamma: int, tau: float, uniforms):
    """One sequence decoded with speculative sampling (gamma > 0) or plain sampling from the full
    model (gamma = 0: a one-row verify and the rule's extra sample), uniforms [rounds, 2 gamma + 1];
    a host read of the accepted count per round.  Returns (seconds, tokens, accepted, drafted)."""
    import numpy as np
    import torch
    ud = dd.buf("u_draft", (1, max(gamma, 1)), torch.float32)
    ua = dd.buf("u_accept", (1, gamma + 1), torch.float32)
    u_dev = torch.from_numpy(np.ascontiguousarray(uniforms, dtype=np.float32)).to(ud.device)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    pending, _ = dd.prefill(pt, vt)
    emitted, r, acc, drafted = 1, 0, 0, 0
    while emitted < T:
        if gamma > 0:
            ud.copy_(u_dev[r:r + 1, :gamma])
        ua.copy_(u_dev[r:r + 1, gamma:])
        if gamma > 0:
            d, dl = dd.draft_sample(pending, gamma, ud, tau)
        else:
            d, dl = dd.buf("no_draft", (1, 1)), None
        t, tl = dd.verify(pending, d, gamma, reuse=gamma > 0, logits=True)
        _, alen = dd.accept_sample(d, dl, tl, ua, tau, pending, gamma)
        a = int(alen.cpu()[0])
        emitted += a + 1
        acc += a
        drafted += gamma
        r += 1
    torch.cuda.synchronize()
    return time.perf_counter() - t0, min(emitted, T), acc, drafted


def cpu_baseline(wl, weights, prompt, visual, budget_s: float):
    """The float64 oracle on the host over a bounded sample of the workload: one prefill, as many
    rounds of Algorithm 1 as fit about 60% of the budget and as many greedy steps as fit the rest
    (each run restarts from the prefill, whose time is subtracted).  Decode-phase rates are
    emitted tokens over decode time; end-to-end rates are T over the prefill plus T - 1 tokens at
    the decode rate."""
    import numpy as np
    from oracle import decode
    from oracle.model import Decoder
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        threads = max([i.get("num_threads", 1) for i in info] or [1])
        vendor = ",".join(sorted({str(i.get("internal_api")) for i in info})) or "unknown"
    except Exception:
        threads, vendor = 1, "unknown"
    dec = Decoder(wl.shape, weights, wl.draft_layers)
    T, g = wl.new_tokens, wl.gamma
    t0 = time.perf_counter()
    decode.prefill(dec, prompt, visual, wl.max_seq())
    t_prefill = time.perf_counter() - t0
    t0 = time.perf_counter()
    one = decode.ssd(dec, prompt, visual, T, g, max_rounds=1)
    per_round = max(time.perf_counter() - t0 - t_prefill, 1e-3)
    rounds = int(max(1, min(T, (0.6 * budget_s - t_prefill) / per_round)))
    t0 = time.perf_counter()
    run = decode.ssd(dec, prompt, visual, T, g, max_rounds=rounds)
    t_ssd = max(time.perf_counter() - t0 - t_prefill, 1e-6)
    n_ssd = len(run.tokens) - 1
    drafted = sum(len(r.drafts) for r in run.rounds)
    alpha = sum(r.accepted for r in run.rounds) / max(1, drafted)
    per_step = per_round / (g + 1 + g * wl.draft_layers / wl.shape.n_layers)
    steps = int(max(1, min(T - 1, (0.4 * budget_s - t_prefill) / max(per_step, 1e-4))))
    t0 = time.perf_counter()
    gr = decode.greedy(dec, prompt, visual, steps + 1)
    t_gr = max(time.perf_counter() - t0 - t_prefill, 1e-6)
    ssd_dec = n_ssd / t_ssd
    gr_dec = steps / t_gr
    e2e = lambda rate: T / (t_prefill + (T - 1) / rate)
    del one, gr
    return {"value": round(e2e(ssd_dec), 4), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"{wl.name} seed 0: float64 oracle ({vendor} BLAS), one prefill "
                       f"({t_prefill:.2f} s), {len(run.rounds)} rounds of Algorithm 1 (gamma {g}, "
                       f"{n_ssd} tokens in {t_ssd:.1f} s) and {steps} greedy steps "
                       f"({t_gr:.1f} s); end-to-end rates extrapolate the decode rate to the "
                       f"{T}-token job; host affinity {len(os.sched_getaffinity(0))} cpus"),
            "ssd": {"decode_tokens_per_s": round(ssd_dec, 4),
                    "end_to_end_tokens_per_s": round(e2e(ssd_dec), 4),
                    "acceptance_rate": round(alpha, 4), "rounds": len(run.rounds)},
            "greedy": {"decode_tokens_per_s": round(gr_dec, 4),
                       "end_to_end_tokens_per_s": round(e2e(gr_dec), 4), "steps": steps},
            "prefill_s": round(t_prefill, 3), "blas": vendor}


def read_ceiling(nbytes: int = 2 << 30) -> dict:
    """The measured HBM read ceiling: a read-only stream kernel of the library over nbytes."""
    import torch
    from paper_2510_22641_amd import ssd as abi
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    out = torch.empty(4096, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream()
    gbps = abi.ssd_read_bandwidth(buf, nbytes, out, 5, s.cuda_stream)
    del buf, out
    return {"GBps": round(gbps, 1), "frac_of_nominal": round(gbps / HBM_PEAK_GBS, 4),
            "bytes": nbytes, "kernel": "read_probe_kernel (one 16 KB chunk per block, 16-byte loads)"}


def confidence_sweep(dd, pt, vt, wl, steps: int, greedy_toks, greedy_s: float):
    """Confidence-stopped drafting at c3: the device's own draft confidences of one job at
    threshold 0 give thresholds at their 5/10/20/30/50% quantiles; each threshold is timed with
    ssd_generate_confident (threshold 0 too: no stop, no per-step read-back)."""
    import numpy as np
    import torch
    B, T, g = wl.batch, wl.new_tokens, wl.gamma
    pending, _ = dd.prefill(pt, vt)
    confs, emitted = [], 1
    while emitted < T:
        d, nd, cf, _, st = dd.draft_confident(pending, g, 0.0)
        t, _ = dd.verify(pending, d, st, reuse=True)
        _, alen = dd.accept_counts(d, nd, t, pending, st)
        confs.append(cf.cpu().numpy()[0, :st].copy())
        emitted += int(alen.cpu()[0]) + 1
    confs = np.concatenate(confs)
    qs = [0.05, 0.1, 0.2, 0.3, 0.5]
    out = {"confidence_quantiles": {str(q): float(np.quantile(confs, q)) for q in qs},
           "confidence_range": [float(confs.min()), float(confs.max())], "points": []}
    for q, tau in [(0.0, 0.0)] + [(q, float(np.quantile(confs, q))) for q in qs]:
        dd.generate_confident(pt, vt, T, g, tau)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            toks, st = dd.generate_confident(pt, vt, T, g, tau)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        out["points"].append({
            "quantile": q, "threshold": tau, "tokens_per_s": round(B * T * steps / dt, 2),
            "speedup_vs_greedy": round(greedy_s / (dt / steps), 3),
            "acceptance_rate": round(st["accepted"] / max(1, st["drafted"]), 4),
            "drafts_per_round": round(st["drafted"] / max(1, st["rounds"]), 3),
            "rounds": st["rounds"], "equals_greedy_tokens": bool(torch.equal(toks, greedy_toks))})
        print(f"[bench] confidence stop q={q} tau={tau:.3g}: {out['points'][-1]}", file=sys.stderr,
              flush=True)
    return out


def per_config(seed: int, steps: int) -> dict:
    """One whole job of each other single-GPU workload (c1, c2, c5): speculative and greedy
    decode through ssd_generate, their tokens, acceptance, and the draft-step / verify times
    against their byte rooflines."""
    import torch
    import synth
    from paper_2510_22641_amd import runtime
    res = {}
    for wl in (synth.C1, synth.C2, synth.C5):
        t_setup = time.time()
        sh = wl.shape
        dd = runtime.from_workload(wl, seed)
        prompts = synth.make_prompts(sh, seed, wl.batch, wl.prompt_len)
        visual = synth.make_visual(sh, seed, wl.batch)
        pt, vt = dd.upload_inputs(prompts, visual)
        B, T, g = wl.batch, wl.new_tokens, wl.gamma

        def timed(spec):
            dd.generate(pt, vt, T, g, speculative=spec, reuse=True)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                toks, st = dd.generate(pt, vt, T, g, speculative=spec, reuse=True)
            torch.cuda.synchronize()
            return (time.perf_counter() - t0) / steps, st, toks

        ds, st, toks = timed(True)
        dg, _, gtoks = timed(False)
        d_s, v_s, ctx = step_timings(dd, pt, vt, B, g)
        db = draft_step_bytes(sh, wl.draft_layers, ctx, dd.k_pool.element_size(),
                              cross_folded(sh, dd.cap.max_batch))
        vb = verify_bytes(sh, B, g, ctx, dd.k_pool.element_size())
        pf = prefill_timing(dd, pt, vt)
        res[wl.name] = {
            "tokens_per_s": round(B * T / ds, 2), "greedy_tokens_per_s": round(B * T / dg, 2),
            "speedup_vs_greedy": round(dg / ds, 3),
            "acceptance_rate": round(st["accepted"] / max(1, st["drafted"]), 4),
            "rounds": st["rounds"], "ssd_equals_greedy_tokens": bool(torch.equal(toks, gtoks)),
            "prefill_ms": round(pf * 1e3, 3),
            "draft_step": {"us": round(d_s * 1e6, 2), "bytes": int(db),
                           "frac": round(db / d_s / 1e9 / HBM_PEAK_GBS, 4)},
            "verify": {"us": round(v_s * 1e6, 2), "bytes": int(vb),
                       "frac": round(vb / v_s / 1e9 / HBM_PEAK_GBS, 4)},
            "jobs": steps, "setup_s": round(time.time() - t_setup, 1)}
        print(f"[bench] {wl.name}: {res[wl.name]}", file=sys.stderr, flush=True)
        dd.close()
        del dd
        torch.cuda.empty_cache()
    return res


def counter_pass(args):
    """A short uncaptured pass for rocprofv3 --pmc: the workload's prefill and, for 'verify', three
    speculative rounds (draft, verify reusing the layer-k states, accept), or, for 'generate', one
    whole speculative job through ssd_generate (prefill included)."""
    import torch
    import synth
    from paper_2510_22641_amd import runtime
    wl = synth.ALL[args.workload]
    dd = runtime.from_workload(wl, args.seed)
    dd.set_graphs(False)
    pr = synth.make_prompts(wl.shape, args.seed, wl.batch, wl.prompt_len)
    z = synth.make_visual(wl.shape, args.seed, wl.batch)
    pt, vt = dd.upload_inputs(pr, z)
    torch.cuda.synchronize()
    print(f"[counter pass] {wl.name} set up", file=sys.stderr, flush=True)
    if args.counter_pass == "generate":
        toks, st = dd.generate(pt, vt, wl.new_tokens, wl.gamma, speculative=True, reuse=True)
        torch.cuda.synchronize()
        status = dd.sync_status()
        print(json.dumps({"counter_pass": "generate", "workload": wl.name, "rounds": st["rounds"],
                          "status": list(status)}), flush=True)
        if tuple(status) != (0, 0):
            raise RuntimeError(f"device status {status}")
        return
    pending, _ = dd.prefill(pt, vt)
    torch.cuda.synchronize()
    print(f"[counter pass] {wl.name} prefill done", file=sys.stderr, flush=True)
    rounds = 3 if args.counter_pass == "verify" else 0
    for _ in range(rounds):
        d, _ = dd.draft(pending, wl.gamma)
        t, _ = dd.verify(pending, d, wl.gamma, reuse=True)
        dd.accept(d, t, pending, wl.gamma)
    torch.cuda.synchronize()
    status = dd.sync_status()
    print(json.dumps({"counter_pass": args.counter_pass, "workload": wl.name, "rounds": rounds,
                      "status": list(status)}), flush=True)
    if tuple(status) != (0, 0):
        raise RuntimeError(f"device status {status}")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="c3-flant5-xl")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--fit-prompts", type=int, default=32,
                    help="sequences (seeds 1000..) whose states fit the imitation network's second "
                         "layer before a second measurement (0: skip)")
    ap.add_argument("--sample-temps", default="1.0,0.1",
                    help="temperatures of the speculative-sampling measurement (empty: skip)")
    ap.add_argument("--per-config", type=int, default=1,
                    help="also time one whole job of c1, c2 and c5 (0: skip)")
    ap.add_argument("--confidence", type=int, default=1,
                    help="also sweep confidence-stopped drafting over thresholds (0: skip)")
    ap.add_argument("--sweep", choices=["c4"], default=None,
                    help="run the FlanT5-xl sweep instead (one JSON line per point)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only copy this many bytes device to device three times (the reference "
                         "reading for the HBM byte counters) and exit")
    ap.add_argument("--counter-pass", choices=["verify", "prefill", "generate"], default=None,
                    help="only run a short pass of --workload for hardware counters and exit, "
                         "graphs off so that every kernel is its own dispatch: 'verify' = prefill "
                         "and three speculative rounds, 'prefill' = one prefill, 'generate' = one "
                         "whole speculative job through ssd_generate")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the decode loop is not sharded (asked for {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    if args.sweep:
        sweep_c4(args)
        return
    if args.copy_bytes:
        import torch
        src = torch.ones(args.copy_bytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel() * 4, "copies": 3}))
        return

    import numpy as np
    import torch
    import synth
    from paper_2510_22641_amd import runtime
    from paper_2510_22641_amd import ssd as abi

    if args.counter_pass:
        counter_pass(args)
        return

    wl = synth.ALL[args.workload]
    sh = wl.shape
    t_setup = time.time()
    weights = synth.workload_weights(wl, args.seed)
    prompts = synth.make_prompts(sh, args.seed, wl.batch, wl.prompt_len)
    visual = synth.make_visual(sh, args.seed, wl.batch)
    # capacity for the dynamic draft length too (up to gamma + 9 drafts a round)
    dd = runtime.from_workload(wl, args.seed, weights=weights, max_gamma=wl.gamma + 9)
    pt, vt = dd.upload_inputs(prompts, visual)
    torch.cuda.synchronize()
    print(f"[bench] setup {time.time() - t_setup:.1f}s", file=sys.stderr, flush=True)

    B, T, g = wl.batch, wl.new_tokens, wl.gamma

    def timed(speculative: bool, steps: int, warmup: int, dynamic: bool = False):
        for _ in range(warmup):
            dd.generate(pt, vt, T, g, speculative=speculative, reuse=True, dynamic=dynamic)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        stats = None
        for _ in range(steps):
            toks, stats = dd.generate(pt, vt, T, g, speculative=speculative, reuse=True,
                                      dynamic=dynamic)
        torch.cuda.synchronize()
        return time.perf_counter() - t0, stats, toks

    # Algorithm 1 (the timed steps)
    dt, st, toks_ssd = timed(True, args.steps, args.warmup)
    ssd_tps = B * T * args.steps / dt
    alpha = st["accepted"] / max(1, st["drafted"])
    print(f"[bench] ssd {ssd_tps:.1f} tok/s alpha {alpha:.3f}", file=sys.stderr, flush=True)
    dtg, _, toks_greedy = timed(False, args.steps, 1)
    greedy_tps = B * T * args.steps / dtg
    same = bool(torch.equal(toks_ssd, toks_greedy))
    print(f"[bench] greedy {greedy_tps:.1f} tok/s", file=sys.stderr, flush=True)
    # the context-length draft schedule d(t) (d(0) = gamma), same decoder and inputs
    dtd, std, toks_dyn = timed(True, args.steps, 1, dynamic=True)
    dyn = {"tokens_per_s": round(B * T * args.steps / dtd, 2),
           "speedup_vs_greedy": round(dtg / dtd, 3),
           "acceptance_rate": round(std["accepted"] / max(1, std["drafted"]), 4),
           "rounds": std["rounds"], "drafted": std["drafted"],
           "equals_greedy_tokens": bool(torch.equal(toks_dyn, toks_greedy)),
           "schedule": f"d(t) = {g} + floor(10 sigmoid(0.01 (t - {dd.cap.max_seq}/2)))"}
    print(f"[bench] dynamic d(t) {dyn['tokens_per_s']:.1f} tok/s", file=sys.stderr, flush=True)

    conf = None
    if args.confidence and B == 1:
        conf = confidence_sweep(dd, pt, vt, wl, max(1, args.steps // 2), toks_greedy,
                                dtg / args.steps)

    # prefill alone (its projections on MFMA tiles once the context exceeds the skinny chunk)
    pf_s = prefill_timing(dd, pt, vt)
    pf_flops = prefill_flops(sh, B, wl.prompt_len)
    prefill = {"ms": round(pf_s * 1e3, 3), "tflop": round(pf_flops / 1e12, 4),
               "tflops_per_s": round(pf_flops / pf_s / 1e12, 1),
               "frac_of_bf16_mfma_peak": round(pf_flops / pf_s / 1e12 / MFMA_BF16_PEAK_TFS, 4)}
    print(f"[bench] prefill {prefill}", file=sys.stderr, flush=True)

    # draft-step time: events around the gamma-step draft call (captured graph) on its stream
    step_s, verify_s, ctx = step_timings(dd, pt, vt, B, g)
    step_bytes = draft_step_bytes(sh, wl.draft_layers, ctx, dd.k_pool.element_size(),
                                  cross_folded(sh, dd.cap.max_batch))
    draft = {"us": round(step_s * 1e6, 2), "bytes": int(step_bytes),
             "GBps": round(step_bytes / step_s / 1e9, 1),
             "frac": round(step_bytes / step_s / 1e9 / HBM_PEAK_GBS, 4)}
    vbytes = verify_bytes(sh, B, g, ctx, dd.k_pool.element_size())
    verify = {"us": round(verify_s * 1e6, 2), "bytes": int(vbytes),
              "GBps": round(vbytes / verify_s / 1e9, 1),
              "frac": round(vbytes / verify_s / 1e9 / HBM_PEAK_GBS, 4)}
    # MFMA utilisation of the verify pass: its flops over its time against the bf16 peak; the HBM
    # roofline caps it at M / 312.5 for M rows (M flops per weight byte at 8 TB/s)
    vfl = verify_flops(sh, B, g, ctx)
    Mv = B * (g + 1)
    verify["mfma"] = {"tflops_per_s": round(vfl / verify_s / 1e12, 2),
                      "frac_of_bf16_peak": round(vfl / verify_s / 1e12 / MFMA_BF16_PEAK_TFS, 5),
                      "hbm_bound_frac": round(Mv / 312.5, 5),
                      "frac_of_bound": round(vfl / verify_s / 1e12 / MFMA_BF16_PEAK_TFS /
                                             (Mv / 312.5), 4)}

    # dominant kernel: every launch of the one-row weight-streaming GEMV that streams the
    # RMS-normalised d_model-wide matrices, timed by events bound to its own dispatch
    abi.ssd_profile_enable(dd.ctx, True)
    abi.ssd_profile_read(dd.ctx)
    for _ in range(max(1, args.steps // 2)):
        dd.generate(pt, vt, T, g, speculative=True, reuse=True)
    n_launch, secs, nbytes = abi.ssd_profile_read(dd.ctx)
    abi.ssd_profile_enable(dd.ctx, False)
    if n_launch == 0 or secs <= 0:
        raise RuntimeError("no launch of the profiled GEMV was timed")
    per_launch_bytes = nbytes / n_launch
    avg_s = secs / n_launch
    achieved = per_launch_bytes / avg_s / 1e9
    kname = dominant_kernel_name(sh)
    counted = counted_traffic(kname) if wl.name == "c3-flant5-xl" else None
    roofline = {"bound": "hbm", "kernel": kname + " (one-row weight-streaming GEMV, RMSNorm folded)",
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": counted["bytes"] if counted else None,
                "traffic_algorithmic": counted["algorithmic_bytes"] if counted else None,
                "traffic_source": counted["source"] if counted else None,
                "bytes_per_launch": int(per_launch_bytes), "avg_launch_us": round(avg_s * 1e6, 3),
                "launches": n_launch}

    # speculative sampling against plain sampling from the full model, same build and uniforms
    sampling = []
    temps = [] if args.sample_temps.strip() in ("", "=", "none") else \
        [float(x) for x in args.sample_temps.split(",") if x.strip()]
    for tau in temps:
        u_ssd = synth.make_uniforms(args.seed, 1, T, 2 * g + 1)[0]
        u_full = synth.make_uniforms(args.seed + 1, 1, T, 1)[0]
        sampled_decode(dd, pt[:1], vt[:1], T, g, tau, u_ssd)  # warm-up (graph capture)
        sampled_decode(dd, pt[:1], vt[:1], T, 0, tau, u_full)
        ts, ns, acc, dr = 0.0, 0, 0, 0
        tf, nf = 0.0, 0
        for _ in range(args.steps):
            t1, n1, a1, d1 = sampled_decode(dd, pt[:1], vt[:1], T, g, tau, u_ssd)
            t2, n2, _, _ = sampled_decode(dd, pt[:1], vt[:1], T, 0, tau, u_full)
            ts, ns, acc, dr, tf, nf = ts + t1, ns + n1, acc + a1, dr + d1, tf + t2, nf + n2
        sampling.append({"temperature": tau, "tokens_per_s": round(ns / ts, 2),
                         "acceptance_rate": round(acc / max(1, dr), 4),
                         "full_model_sampling_tokens_per_s": round(nf / tf, 2),
                         "speedup_vs_full_model_sampling": round((ns / ts) / (nf / tf), 3),
                         "loop": "host-driven rounds (one accepted-count read per round)"})
        print(f"[bench] sampling tau {tau}: {sampling[-1]}", file=sys.stderr, flush=True)

    # the imitation network's second layer fitted on the decoder's own states (other sequences),
    # then the same job measured again; the headline keeps the configured network
    fit = None
    if args.fit_prompts > 0:
        from paper_2510_22641_amd import imitation
        t_fit = time.time()
        rows = [[], [], []]
        for s in range(1000, 1000 + args.fit_prompts):
            zf = synth.make_visual(sh, s, B)
            pf = synth.make_prompts(sh, s, B, wl.prompt_len)
            ptf, vtf = dd.upload_inputs(pf, zf)
            for r, a in zip(rows, imitation.collect(dd, ptf[:1], vtf[:1], T, g)):
                r.append(a)
        phi, xk, xl = (np.concatenate(r) for r in rows)
        w2, b2, info = imitation.fit_validated(phi, xk, xl, weights["in_w2"], weights["in_b2"],
                                               residual=dd.in_residual)
        fit = {"fit_sequences": args.fit_prompts, "fit_rows": info["rows"],
               "ridge": info["ridge"], "val_mse": info["val_mse"],
               "val_mse_configured": info["val_mse_configured"], "installed": w2 is not None,
               "method": "ridge least squares of x_k + W2 phi + b2 against x_L on the decoder's "
                         "own states (W1, b1, LayerNorm kept; ridge chosen on 20% held-out rows)"}
        if w2 is not None:
            imitation.install(dd, w2, b2)
            dtf, stf, toks_fit = timed(True, args.steps, 1)
            fit.update({"tokens_per_s": round(B * T * args.steps / dtf, 2),
                        "speedup_vs_greedy": round(dtg / dtf, 3),
                        "acceptance_rate": round(stf["accepted"] / max(1, stf["drafted"]), 4),
                        "equals_greedy_tokens": bool(torch.equal(toks_fit, toks_greedy))})
        fit["seconds"] = round(time.time() - t_fit, 1)
        print(f"[bench] fitted imitation network: {fit}", file=sys.stderr, flush=True)

    rc, status = dd.sync_status()
    if rc != 0:
        print(f"[bench] device status {status}", file=sys.stderr)
        sys.exit(1)
    dd.close()
    del dd
    torch.cuda.empty_cache()

    ceiling = read_ceiling()
    print(f"[bench] read ceiling {ceiling}", file=sys.stderr, flush=True)
    for part in (draft, verify):
        part["frac_of_read_ceiling"] = round(part["GBps"] / ceiling["GBps"], 4)
    others = per_config(args.seed, 3) if args.per_config and wl.name == "c3-flant5-xl" else None

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, weights, prompts[0], visual[0], args.cpu_seconds)

    out = {
        "metric": "accepted output tokens/s @ batch 1 (FlanT5-xl-shaped); draft-step HBM GB/s vs peak",
        "value": round(ssd_tps, 2), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(dt / args.steps * 1e3, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init decoder, N(0,1) visual tokens, uniform prompt ids)",
        "config": {"workload": wl.name, "decoder": f"{'T5' if sh.arch == 't5' else 'LLaMA'}-style "
                   f"L{sh.n_layers} d{sh.d_model} "
                   f"H{sh.n_heads}x{sh.d_head} ff{sh.d_ff} V{sh.vocab}", "batch": B,
                   "prompt": wl.prompt_len, "visual_tokens": sh.n_visual,
                   "draft_layers": wl.draft_layers, "gamma": g, "new_tokens": T,
                   "deep_scale": wl.deep_scale, "parallelism": "none (1 GPU)"},
        "acceptance_rate": round(alpha, 4),
        "rounds": st["rounds"],
        "greedy_tokens_per_s": round(greedy_tps, 2),
        "speedup_vs_greedy": round(ssd_tps / greedy_tps, 3),
        "ssd_equals_greedy_tokens": same,
        "dynamic_gamma": dyn,
        "confidence_stop": conf,
        "speculative_sampling": sampling or None,
        "fitted_imitation": fit,
        "prefill": prefill,
        "draft_step": draft,
        "verify": verify,
        "roofline": roofline,
        "read_ceiling": ceiling,
        "per_config": others,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
