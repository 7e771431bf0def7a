"""Benchmark: STaR-Quant W4A4 SGAT linear layer set per denoising step on one MI355X.

Workload (default): the LLaDA-8B-shaped layer set, one sequence of 1024 tokens
(512 unmasked prompt tokens, 512 generation tokens with 8 of 16 32-token blocks
masked): QKV 4096->12288, O 4096->4096 with TAC (g = 16) ahead of it,
gate+up 4096->24576, down 12288->4096, all W4A4 SGAT, fp16 in and out.

One step = the whole per-step hot path for every linear of the set:
    [TAC] -> x P G_s (dense fp32 transform, Eq. 11) -> per-token int4 -> W4A4 GEMM
with the weights prepared offline (Eq. 12, outside the timed region) and every
input resident in HBM.  A second measurement runs the deployment form in which P
is folded into the weights and the upstream activations, so the step is
[TAC] -> gate -> int4 -> GEMM; it is reported next to the main figure.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]

Prints one JSON line.  Synthetic, seeded inputs (no datasets, no trained weights).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_INT8_TOPS = 5000.0           # dense int8 MFMA, TOP/s
PEAK_FP16_TFLOPS = 2500.0         # dense fp16 MFMA, TFLOP/s
PEAK_FP6_TFLOPS = 10100.0         # dense FP6 / FP4 MFMA, TFLOP/s
# fp32 FMA on the VALU without packed-fp32 instructions (the library is built
# without them): 256 CU x 4 SIMD x 16 lanes x 2 flop x 2.4 GHz
PEAK_FP32_VALU_TFLOPS = 78.6


def recorded_traffic(kernel: str, field: str = "traffic_bytes_per_launch"):
    """HBM bytes per launch of `kernel` from the committed counter record, or None
    when the kernel's sources have changed since the counters were taken."""
    import hashlib
    try:
        with open(os.path.join(ROOT, "profiles", "counters.json")) as f:
            rec = json.load(f)[kernel]
    except (OSError, KeyError, ValueError):
        return None
    for name, h in rec["sources_sha256_16"].items():
        path = os.path.join(ROOT, "paper_2606_04945_amd", "csrc", name)
        with open(path, "rb") as f:
            if hashlib.sha256(f.read()).hexdigest()[:16] != h:
                return None
    return rec.get(field)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=384, help="tokens in the oracle timing sample")
    ap.add_argument("--only", choices=["dense", "folded", "both"], default="both")
    ap.add_argument("--no-w8", action="store_true", help="skip the W8A8 (App. D) folded-basis measurement")
    ap.add_argument("--no-large", action="store_true",
                    help="skip the 16384-token Dream-shaped layer set (large-token GEMM figures)")
    ap.add_argument("--no-small", action="store_true",
                    help="skip the 16/32/64-token denoising-step layer sets (small-token HBM figures)")
    ap.add_argument("--no-calib", action="store_true", help="skip the TAC calibration timing")
    ap.add_argument("--no-fast", action="store_true", help="skip the dense step with the matrix-core transform")
    ap.add_argument("--no-sweep", action="store_true", help="skip the GEMM token-count sweep")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (reference for HBM byte counters)")
    return ap.parse_args()


class Timer:
    """HIP event pairs on the launching stream, summed per label."""

    def __init__(self, torch):
        self.torch = torch
        self.pairs = {}

    def wrap(self, label, fn):
        s = self.torch.cuda.Event(enable_timing=True)
        e = self.torch.cuda.Event(enable_timing=True)
        s.record()
        fn()
        e.record()
        self.pairs.setdefault(label, []).append((s, e))

    def ms(self, label):
        ps = self.pairs.get(label, [])
        return sum(s.elapsed_time(e) for s, e in ps), len(ps)

    def reset(self):
        self.pairs = {}


LLC_DEFEAT_BYTES = 800 << 20     # weight copies cycled per timing: over 3x the 256 MB last-level cache


def rotating_copies(Wq, s_w, floor=4):
    """(Wq, s_w) followed by enough clones that one pass over them streams at
    least LLC_DEFEAT_BYTES, so that no call finds its weights in the last-level
    cache."""
    n = max(floor, -(-LLC_DEFEAT_BYTES // (Wq.numel() * Wq.element_size() + s_w.numel() * 4)))
    return [(Wq, s_w)] + [(Wq.clone(), s_w.clone()) for _ in range(n - 1)]


def graph_ms(torch, fn, calls, replays=5):
    """Median milliseconds per call of fn(i), i = 0 .. calls - 1, captured back to
    back in one HIP graph, so that no host work sits between the launches."""
    fn(0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(calls):
                fn(i)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    ts = []
    for _ in range(replays):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) / calls)
    ts.sort()
    return ts[len(ts) // 2], g


def large_token_block(torch, sq, synth, dev, steps, warmup):
    """Dream-shaped layer set, 8 x 2048 tokens, folded P: per linear the gate +
    int4 quantiser (TAC ahead of O) and the W4A4 GEMM.  Event pairs per call; the
    kernels are long enough that the host keeps the queue full."""
    cfg = synth.CONFIGS[synth.DREAM]
    st_np = synth.config_state(synth.DREAM)
    M = len(st_np)
    state = torch.from_numpy(st_np).to(dev)
    sites = []
    for si, site in enumerate(cfg.sites):
        t = synth.site_tensors(synth.DREAM, si, st_np, with_P=False)
        W = torch.from_numpy(t.W).to(dev)
        Wq, s_w = sq.sgat_prepare_weights(W, None)
        del W
        d = dict(name=site.name, K=site.K, N=site.N, dm=t.dm, du=t.du, X=torch.from_numpy(t.X).to(dev),
                 Wq=Wq, Wf=sq.weights_to_frag(Wq), s_w=s_w,
                 Aq=torch.empty((M, site.K // 2), dtype=torch.uint8, device=dev),
                 s_a=torch.empty((M,), dtype=torch.float32, device=dev),
                 Y=torch.empty((M, site.N), dtype=torch.float16, device=dev))
        if site.tac:
            d.update(tac_M=torch.from_numpy(t.tac_M).to(dev), tac_d=torch.from_numpy(t.tac_d).to(dev), g=t.g)
        d["qws"] = torch.empty(max(sq.quant_act_workspace_bytes(M, site.K, False, site.tac), 1), dtype=torch.uint8,
                               device=dev)
        d["gws"] = torch.empty(max(sq.gemm_workspace_bytes(M, site.N, site.K), 1), dtype=torch.uint8, device=dev)
        sites.append(d)
        del t
    timer = Timer(torch)

    def step(tm):
        for d in sites:
            tm.wrap("q/" + d["name"], lambda: sq.sgat_quant_act(d["X"], state, None, d["dm"], d["du"], d.get("tac_M"),
                                                                 d.get("tac_d"), d.get("g", 0), Aq=d["Aq"],
                                                                 s_a=d["s_a"], ws=d["qws"]))
            tm.wrap("g/" + d["name"], lambda: sq.w4a4_gemm_frag(d["Aq"], d["s_a"], d["Wf"], d["s_w"], Y=d["Y"],
                                                                 ws=d["gws"]))
    for _ in range(warmup):
        step(Timer(torch))
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step(timer)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    per = {}
    tot_ops = tot_ms = 0.0
    for d in sites:
        gms = timer.ms("g/" + d["name"])[0] / steps
        ops = 2.0 * M * d["N"] * d["K"]
        per[d["name"]] = {"M": M, "N": d["N"], "K": d["K"], "gemm_us": gms * 1e3, "tops": ops / gms / 1e9,
                          "frac_int8_peak": ops / gms / 1e9 / PEAK_INT8_TOPS,
                          "quant_act_us": timer.ms("q/" + d["name"])[0] / steps * 1e3}
        tot_ops += ops
        tot_ms += gms
    dom = max(per, key=lambda n: per[n]["gemm_us"])
    fp6 = fp6_variant(torch, sq, sites, state, M, steps, warmup)
    for d in sites:      # context: the vendor library's int8 GEMM (torch._int_mm) at the same shape
        per[d["name"]]["vendor_int8_gemm_us"] = vendor_int8_us(torch, M, d["N"], d["K"], d["X"].device)
    out = {"workload": "Dream-7B-shaped SGAT layer set (QKV 3584->4608, O+TAC 3584->3584, gate+up 3584->37888, "
                       "down 18944->3584), 8 x 2048 tokens, folded P",
           "tokens": M, "ms_per_step": ms, "tokens_per_s": M / (ms / 1e3),
           "gemm_tops": tot_ops / tot_ms / 1e9, "gemm_frac_int8_peak": tot_ops / tot_ms / 1e9 / PEAK_INT8_TOPS,
           "per_site": per,
           "roofline": {"bound": "mfma", "achieved": per[dom]["tops"], "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                        "frac": per[dom]["frac_int8_peak"],
                        "traffic": recorded_traffic("gemm_large") if dom == "gate_up" else None,
                        "kernel": f"w4a4 gemm ({dom})"},
           "fp6": fp6}
    del sites
    torch.cuda.empty_cache()
    return out


def vendor_int8_us(torch, M, N, K, dev, reps=5):
    """Microseconds per call of the vendor library's int8 GEMM (torch._int_mm,
    int32 out) on int8 operands of the same shape: a reference point only."""
    g = torch.Generator(device="cpu").manual_seed(M + N + K)
    A = torch.randint(-8, 8, (M, K), dtype=torch.int8, generator=g).to(dev)
    B = torch.randint(-8, 8, (N, K), dtype=torch.int8, generator=g).to(dev)
    try:
        torch._int_mm(A, B.t())
    except (RuntimeError, AttributeError):
        return None
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        torch._int_mm(A, B.t())
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    del A, B
    return us


def fp6_variant(torch, sq, sites, state, M, steps, warmup):
    """The same layer set with the codes carried as e3m2 on the FP6 matrix cores:
    per linear the gate + int4 quantiser, the conversion of the activation codes
    to the FP6 operand layout, and the GEMM on FP6 operands (weights converted
    once, offline).  Its outputs are checked equal to the int4 path's."""
    ref = {d["name"]: d["Y"].clone() for d in sites}
    for d in sites:
        d["W6"] = sq.codes_to_fp6(d["Wq"])
        d["A6"] = torch.empty((M, sq.fp6_row_bytes(d["K"])), dtype=torch.uint8, device=d["Aq"].device)
        d["Y6"] = torch.empty_like(d["Y"])
    timer = Timer(torch)

    def step(tm):
        for d in sites:
            tm.wrap("q/" + d["name"], lambda: sq.sgat_quant_act(d["X"], state, None, d["dm"], d["du"], d.get("tac_M"),
                                                                 d.get("tac_d"), d.get("g", 0), Aq=d["Aq"],
                                                                 s_a=d["s_a"], ws=d["qws"]))
            tm.wrap("c/" + d["name"], lambda: sq.codes_to_fp6(d["Aq"], out=d["A6"]))
            tm.wrap("g/" + d["name"], lambda: sq.w4a4_gemm_fp6(d["A6"], d["s_a"], d["W6"], d["s_w"], d["K"],
                                                                Y=d["Y6"]))
    for _ in range(warmup):
        step(Timer(torch))
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step(timer)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    per, tot_ops, tot_ms = {}, 0.0, 0.0
    for d in sites:
        gms = timer.ms("g/" + d["name"])[0] / steps
        ops = 2.0 * M * d["N"] * d["K"]
        per[d["name"]] = {"gemm_us": gms * 1e3, "tops": ops / gms / 1e9,
                          "frac_fp6_peak": ops / gms / 1e9 / PEAK_FP6_TFLOPS,
                          "frac_int8_peak": ops / gms / 1e9 / PEAK_INT8_TOPS,
                          "convert_us": timer.ms("c/" + d["name"])[0] / steps * 1e3}
        tot_ops += ops
        tot_ms += gms
    same = all(torch.equal(ref[d["name"]], d["Y6"]) for d in sites)
    dom = max(per, key=lambda n: per[n]["gemm_us"])
    for d in sites:
        del d["W6"], d["A6"], d["Y6"]
    return {"ms_per_step": ms, "tokens_per_s": M / (ms / 1e3), "gemm_tops": tot_ops / tot_ms / 1e9,
            "per_site": per, "outputs_equal_int4_path": same,
            "roofline": {"bound": "mfma", "achieved": per[dom]["tops"], "peak": PEAK_FP6_TFLOPS, "unit": "TFLOP/s",
                         "frac": per[dom]["frac_fp6_peak"], "traffic": None,
                         "kernel": f"w4a4 gemm on FP6 operands ({dom})"}}


def small_token_block(torch, sq, synth, dev, token_counts=(16, 32, 64), copies=8):
    """Denoising-step layer sets at small token counts (LLaDA shapes, step 32 of
    64, folded P), captured in a HIP graph.  `copies` rotating sets of prepared
    weights (8 x 108 MB) keep the 256 MB last-level cache from serving them; each
    GEMM timed on its own cycles through at least 800 MB of its weights.
    Bytes are the algorithmic HBM traffic: fp16 activations read once, codes
    written and read once, the packed weights and scales, the fp16 outputs."""
    cfg = synth.CONFIGS[synth.LLADA_SWEEP]
    st64 = synth.config_state(synth.LLADA_SWEEP, M=max(token_counts), t=32)
    wsets = [[] for _ in range(copies)]
    meta = []
    for si, site in enumerate(cfg.sites):
        t = synth.site_tensors(synth.LLADA_SWEEP, si, st64, with_P=False)
        W = torch.from_numpy(t.W).to(dev)
        Wq, s_w = sq.sgat_prepare_weights(W, None)
        Wf = sq.weights_to_frag(Wq)
        del W, Wq
        for c in range(copies):
            wsets[c].append((Wf.clone(), s_w.clone()))
        meta.append(site)
        del t, Wf, s_w
    out = {}
    dom_rec = None
    for M in token_counts:
        st_np = synth.config_state(synth.LLADA_SWEEP, M=M, t=32)
        state = torch.from_numpy(st_np).to(dev)
        sites = []
        byts = 0
        for si, site in enumerate(meta):
            t = synth.site_tensors(synth.LLADA_SWEEP, si, st_np, with_W=False, with_P=False)
            K, N = site.K, site.N
            d = dict(name=site.name, K=K, N=N, dm=t.dm, du=t.du, X=torch.from_numpy(t.X).to(dev),
                     Aq=torch.empty((M, K // 2), dtype=torch.uint8, device=dev),
                     s_a=torch.empty((M,), dtype=torch.float32, device=dev),
                     Y=torch.empty((M, N), dtype=torch.float16, device=dev))
            tb = 0
            if site.tac:
                d.update(tac_M=torch.from_numpy(t.tac_M).to(dev), tac_d=torch.from_numpy(t.tac_d).to(dev), g=t.g)
                tb = t.tac_M.nbytes + t.tac_d.nbytes
            d["qws"] = torch.empty(max(sq.quant_act_workspace_bytes(M, K, False, site.tac), 1), dtype=torch.uint8,
                                   device=dev)
            d["gws"] = torch.empty(max(sq.gemm_workspace_bytes(M, N, K), 1), dtype=torch.uint8, device=dev)
            d["gemm_bytes"] = N * K // 2 + N * 4 + M * K // 2 + M * 4 + M * N * 2
            byts += M * K * 2 + tb + M * K // 2 + M * 4 + d["gemm_bytes"]
            sites.append(d)

        def qa(d):
            sq.sgat_quant_act(d["X"], state, None, d["dm"], d["du"], d.get("tac_M"), d.get("tac_d"),
                              d.get("g", 0), Aq=d["Aq"], s_a=d["s_a"], ws=d["qws"])

        def step(i):
            for d, (Wf, s_w) in zip(sites, wsets[i % copies]):
                qa(d)
                sq.w4a4_gemm_frag(d["Aq"], d["s_a"], Wf, s_w, Y=d["Y"], ws=d["gws"])

        step(0)
        torch.cuda.synchronize()
        eager = [d["Y"].clone() for d in sites]
        ms, g = graph_ms(torch, step, copies)
        g.replay()
        torch.cuda.synchronize()
        same = all(torch.equal(a, d["Y"]) for a, d in zip(eager, sites))
        del g
        rec = {"ms_per_step": ms, "tokens_per_s": M / (ms / 1e3), "hbm_bytes_per_step": byts,
               "hbm_gbs": byts / ms / 1e6, "frac_hbm_peak": byts / ms / 1e6 / PEAK_HBM_GBS,
               "graph_matches_eager": same, "gemm": {}}
        for si, d in enumerate(sites):
            qa(d)
            rot = rotating_copies(*wsets[0][si])
            gms, g = graph_ms(torch, lambda i, d=d, rot=rot: sq.w4a4_gemm_frag(d["Aq"], d["s_a"],
                                                                               rot[i % len(rot)][0],
                                                                               rot[i % len(rot)][1], Y=d["Y"],
                                                                               ws=d["gws"]), 2 * len(rot))
            del g, rot
            rec["gemm"][d["name"]] = {"us": gms * 1e3, "gbs": d["gemm_bytes"] / gms / 1e6,
                                      "frac_hbm_peak": d["gemm_bytes"] / gms / 1e6 / PEAK_HBM_GBS}
        out[str(M)] = rec
        if M == min(token_counts):
            dn = max(rec["gemm"], key=lambda n: rec["gemm"][n]["us"])
            dom_rec = (dn, rec["gemm"][dn])
        del sites
    res = {"workload": "LLaDA-8B-shaped layer set at 16, 32 and 64 tokens (denoising step 32 of 64), folded P, "
                       "HIP-graph replay, 8 rotating weight sets (per-GEMM timings: >= 800 MB of rotating weights)",
           "per_tokens": out}
    if dom_rec:
        dn, r = dom_rec
        res["roofline"] = {"bound": "hbm", "achieved": r["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                           "frac": r["frac_hbm_peak"],
                           "traffic": recorded_traffic("gemm_small") if dn == "gate_up" else None,
                           "kernel": f"w4a4 gemm ({dn}, {min(token_counts)} tokens)"}
    del wsets
    torch.cuda.empty_cache()
    return res


def sweep_block(torch, sq, synth, dev, token_counts=(16, 64, 256, 1024, 4096, 16384), copies=1):
    """Denoising-step sweep over token counts (LLaDA shapes, step 32 of 64, folded P):
    the W4A4 GEMM of every linear, graph-replayed with rotating weights, as
    achieved TOP/s and algorithmic GB/s, from memory-bound to compute-bound."""
    cfg = synth.CONFIGS[synth.LLADA_SWEEP]
    st_max = synth.config_state(synth.LLADA_SWEEP, M=max(token_counts), t=32)
    wsets, meta = [[] for _ in range(copies)], []
    for si, site in enumerate(cfg.sites):
        t = synth.site_tensors(synth.LLADA_SWEEP, si, st_max[:16], with_P=False)
        W = torch.from_numpy(t.W).to(dev)
        Wq, s_w = sq.sgat_prepare_weights(W, None)
        Wf = sq.weights_to_frag(Wq)
        del W, Wq
        for c in range(copies):
            wsets[c].append((Wf.clone(), s_w.clone()))
        meta.append(site)
        del t, Wf, s_w
    rots = [rotating_copies(*wsets[0][si]) for si in range(len(meta))]
    out = {}
    for M in token_counts:
        rec = {}
        for si, site in enumerate(meta):
            K, N = site.K, site.N
            g = torch.Generator(device="cpu").manual_seed(M * 10 + si)
            Aq = torch.randint(0, 256, (M, K // 2), dtype=torch.uint8, generator=g).to(dev)
            s_a = (torch.rand(M, generator=g) + 0.5).to(dev)
            Y = torch.empty((M, N), dtype=torch.float16, device=dev)
            gws = torch.empty(max(sq.gemm_workspace_bytes(M, N, K), 1), dtype=torch.uint8, device=dev)
            rot = rots[si]
            calls = 2 * len(rot) if M <= 1024 else len(rot)
            ms, gr = graph_ms(torch, lambda i: sq.w4a4_gemm_frag(Aq, s_a, rot[i % len(rot)][0],
                                                                 rot[i % len(rot)][1], Y=Y, ws=gws), calls)
            del gr
            ops = 2.0 * M * N * K
            byts = N * K // 2 + N * 4 + M * K // 2 + M * 4 + M * N * 2
            rec[site.name] = {"us": ms * 1e3, "tops": ops / ms / 1e9, "frac_int8_peak": ops / ms / 1e9 / PEAK_INT8_TOPS,
                              "gbs": byts / ms / 1e6, "frac_hbm_peak": byts / ms / 1e6 / PEAK_HBM_GBS}
            del Aq, s_a, Y, gws
        out[str(M)] = rec
    del wsets, rots
    torch.cuda.empty_cache()
    return {"workload": "W4A4 GEMMs of the LLaDA-shaped layer set, token counts 16 ... 16384, graph-replayed, "
                        ">= 800 MB of rotating weights per GEMM", "per_tokens": out}


def tac_oproj_block(torch, sq, synth, dev, steps=5):
    """TAC (32 blocks of 128) on 8 x 2048 attention outputs of width 4096, then the
    gate + int4 quantiser and the 4096 -> 4096 W4A4 GEMM (folded P).  TAC at
    g = 128 runs as its own kernel (the fused form covers g <= 16)."""
    st_np = synth.config_state(synth.TAC_OPROJ)
    M = len(st_np)
    state = torch.from_numpy(st_np).to(dev)
    t = synth.site_tensors(synth.TAC_OPROJ, 0, st_np, with_P=False)
    K, N, g = t.site.K, t.site.N, t.g
    W = torch.from_numpy(t.W).to(dev)
    Wq, s_w = sq.sgat_prepare_weights(W, None)
    Wf = sq.weights_to_frag(Wq)
    del W, Wq
    X = torch.from_numpy(t.X).to(dev)
    tM, td = torch.from_numpy(t.tac_M).to(dev), torch.from_numpy(t.tac_d).to(dev)
    Z = torch.empty_like(X)
    Aq = torch.empty((M, K // 2), dtype=torch.uint8, device=dev)
    s_a = torch.empty((M,), dtype=torch.float32, device=dev)
    Y = torch.empty((M, N), dtype=torch.float16, device=dev)
    gws = torch.empty(max(sq.gemm_workspace_bytes(M, N, K), 1), dtype=torch.uint8, device=dev)
    timer = Timer(torch)

    def step(tm):
        tm.wrap("tac", lambda: sq.tac_apply(X, tM, td, g, out=Z))
        tm.wrap("q", lambda: sq.sgat_quant_act(Z, state, None, t.dm, t.du, Aq=Aq, s_a=s_a))
        tm.wrap("g", lambda: sq.w4a4_gemm_frag(Aq, s_a, Wf, s_w, Y=Y, ws=gws))
    step(Timer(torch))
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step(timer)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    tac_ms = timer.ms("tac")[0] / steps
    g_ms = timer.ms("g")[0] / steps
    tac_flop = 2.0 * M * K * g
    return {"workload": f"TAC g = {g} + O projection {K}->{N}, 8 x 2048 tokens, folded P",
            "tokens": M, "ms_per_step": ms, "tokens_per_s": M / (ms / 1e3),
            "tac_ms": tac_ms, "quant_ms": timer.ms("q")[0] / steps, "gemm_ms": g_ms,
            "gemm_frac_int8_peak": 2.0 * M * N * K / g_ms / 1e9 / PEAK_INT8_TOPS,
            "roofline": {"bound": "alu", "achieved": tac_flop / tac_ms / 1e9, "peak": PEAK_FP32_VALU_TFLOPS,
                         "unit": "TFLOP/s", "frac": tac_flop / tac_ms / 1e9 / PEAK_FP32_VALU_TFLOPS,
                         "traffic": recorded_traffic("tac_g128") if g == 128 else None,
                         "kernel": f"tac (g = {g})"}}


def tac_calibration_block(torch, sq, synth, dev, N=8192, C=4096, reps=5):
    """TAC closed-form calibration (App. C, offline) on 8192 paired tokens of width
    4096, at the default block size 16 and at 128: call time and the rate at which
    it consumes the two fp16 inputs (the statistics pass reads each once)."""
    out = {}
    for g in (16, 128):
        zf, zq = synth.tac_calib_pair(N, C, g, synth.rng_for(3, synth.T_CALIB, N, C, g))
        Zf, Zq = torch.from_numpy(zf).to(dev), torch.from_numpy(zq).to(dev)
        ws = torch.empty(sq.tac_calibrate_workspace_bytes(N, C, g), dtype=torch.uint8, device=dev)
        tM = torch.empty((C // g, g, g), dtype=torch.float16, device=dev)
        td = torch.empty((C,), dtype=torch.float16, device=dev)
        sq.tac_calibrate(Zf, Zq, g, tac_M=tM, tac_d=td, ws=ws)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            sq.tac_calibrate(Zf, Zq, g, tac_M=tM, tac_d=td, ws=ws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        byts = 2 * N * C * 2
        out[f"g{g}"] = {"ms_per_call": ms, "input_gbs": byts / ms / 1e6,
                        "stats_fp64_gflop": 4.0 * N * C * g / 1e9}
        del Zf, Zq, ws
    return {"workload": f"TAC calibration, {N} paired tokens x {C} channels, fp64 statistics and closed form",
            "per_block_size": out}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; --gpus must be 1"}), flush=True)
        sys.exit(2)
    import torch
    import paper_2606_04945_amd as sq
    import synth

    sq.lib()                                    # raises if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = synth.CONFIGS[synth.LLADA]
    M = cfg.M
    state_np = synth.config_state(synth.LLADA)
    state = torch.from_numpy(state_np).to(dev)
    t0 = time.time()
    sites = []
    for si, site in enumerate(cfg.sites):
        t = synth.site_tensors(synth.LLADA, si, state_np)
        d = dict(site=site, K=site.K, N=site.N, dm=t.dm, du=t.du,
                 X=torch.from_numpy(t.X).to(dev), P=torch.from_numpy(t.P).to(dev),
                 W=torch.from_numpy(t.W).to(dev))
        if site.tac:
            d.update(tac_M=torch.from_numpy(t.tac_M).to(dev), tac_d=torch.from_numpy(t.tac_d).to(dev), g=t.g)
        sites.append(d)
    print(f"# inputs generated in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    # offline weight preparation (Eq. 12), outside the timed region
    for d in sites:
        d["Wq"], d["s_w"] = sq.sgat_prepare_weights(d["W"], d["P"])
        d["Wf"] = sq.weights_to_frag(d["Wq"])
        K, N = d["K"], d["N"]
        d["z"] = torch.empty((M, K), dtype=torch.float16, device=dev) if "tac_M" in d else None
        d["xp"] = torch.empty((M, K), dtype=torch.float32, device=dev)
        d["Aq"] = torch.empty((M, K // 2), dtype=torch.uint8, device=dev)
        d["s_a"] = torch.empty((M,), dtype=torch.float32, device=dev)
        d["Y"] = torch.empty((M, N), dtype=torch.float16, device=dev)
        nb = sq.gemm_workspace_bytes(M, N, K)
        d["gws"] = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)
        nq = sq.quant_act_workspace_bytes(M, K, False, "tac_M" in d)
        d["qws"] = torch.empty(max(nq, 1), dtype=torch.uint8, device=dev)
    if not args.no_w8:
        for d in sites:
            d["Wq8"], d["s_w8"] = sq.sgat_prepare_weights_w8(d["W"], d["P"])
            K, N = d["K"], d["N"]
            d["Aq8"] = torch.empty((M, K), dtype=torch.int8, device=dev)
            d["gws8"] = torch.empty(max(sq.gemm_workspace_bytes(M, N, K, 8), 1), dtype=torch.uint8, device=dev)
    # rotating copies of the prepared weights for the folded-basis runs (8 x 108 MB
    # of 4-bit, 4 x 216 MB of 8-bit codes), so that the 256 MB last-level cache
    # cannot hold a layer set's weights from one step to the next
    wcopies = [[(d["Wf"].clone(), d["s_w"].clone()) for d in sites] for _ in range(8)]
    w8copies = ([[(d["Wq8"].clone(), d["s_w8"].clone()) for d in sites] for _ in range(4)]
                if not args.no_w8 else [])
    torch.cuda.synchronize()
    timer = Timer(torch)

    def step_dense(tm):
        for d in sites:
            src = d["X"]
            if d["z"] is not None:
                tm.wrap("tac", lambda: sq.tac_apply(d["X"], d["tac_M"], d["tac_d"], d["g"], out=d["z"]))
                src = d["z"]
            tm.wrap("transform/" + d["site"].name,
                    lambda: sq.sgat_transform(src, state, d["P"], d["dm"], d["du"], out=d["xp"]))
            tm.wrap("quant", lambda: sq.sgat_quantize(d["xp"], Aq=d["Aq"], s=d["s_a"]))
            tm.wrap("gemm/" + d["site"].name,
                    lambda: sq.w4a4_gemm_frag(d["Aq"], d["s_a"], d["Wf"], d["s_w"], Y=d["Y"], ws=d["gws"]))

    def step_dense_fast(tm):
        for d in sites:
            src = d["X"]
            if d["z"] is not None:
                tm.wrap("tac", lambda: sq.tac_apply(d["X"], d["tac_M"], d["tac_d"], d["g"], out=d["z"]))
                src = d["z"]
            tm.wrap("ftransform/" + d["site"].name,
                    lambda: sq.sgat_transform_fast(src, state, d["Ps"], d["dm"], d["du"], out=d["xp"]))
            tm.wrap("quant", lambda: sq.sgat_quantize(d["xp"], Aq=d["Aq"], s=d["s_a"]))
            tm.wrap("gemm/" + d["site"].name,
                    lambda: sq.w4a4_gemm_frag(d["Aq"], d["s_a"], d["Wf"], d["s_w"], Y=d["Y"], ws=d["gws"]))

    def step_folded(tm, it):
        ws = wcopies[it % len(wcopies)]
        for d, (Wf, s_w) in zip(sites, ws):
            tm.wrap("quant_act/" + d["site"].name,
                    lambda: sq.sgat_quant_act(d["X"], state, None, d["dm"], d["du"], d.get("tac_M"),
                                              d.get("tac_d"), d.get("g", 0), Aq=d["Aq"], s_a=d["s_a"],
                                              ws=d["qws"]))
            tm.wrap("gemm/" + d["site"].name,
                    lambda: sq.w4a4_gemm_frag(d["Aq"], d["s_a"], Wf, s_w, Y=d["Y"], ws=d["gws"]))

    def step_w8(tm, it):
        for d, (Wq8, s_w8) in zip(sites, w8copies[it % len(w8copies)]):
            tm.wrap("quant_act8/" + d["site"].name,
                    lambda: sq.sgat_quant_act_w8(d["X"], state, None, d["dm"], d["du"], d.get("tac_M"),
                                                 d.get("tac_d"), d.get("g", 0), Aq=d["Aq8"], s_a=d["s_a"],
                                                 ws=d["qws"]))
            tm.wrap("gemm8/" + d["site"].name,
                    lambda: sq.w8a8_gemm(d["Aq8"], d["s_a"], Wq8, s_w8, Y=d["Y"], ws=d["gws8"]))

    def run(step, steps, warmup):
        for i in range(warmup):
            step(Timer(torch), i)
        torch.cuda.synchronize()
        timer.reset()
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        start.record()
        for i in range(steps):
            step(timer, i)
        end.record()
        torch.cuda.synchronize()
        return start.elapsed_time(end) / steps

    out = {}
    flops_tr = {d["site"].name: 2.0 * M * d["K"] * (d["K"] - d["K"] // 32) for d in sites}
    ops_gemm = {d["site"].name: 2.0 * M * d["N"] * d["K"] for d in sites}

    if args.only in ("dense", "both"):
        ms_dense = run(lambda tm, i: step_dense(tm), args.steps, args.warmup)
        tr_ms = sum(timer.ms("transform/" + n)[0] for n in flops_tr)
        tr_flop = sum(flops_tr.values()) * args.steps
        gm_ms = sum(timer.ms("gemm/" + n)[0] for n in ops_gemm)
        gm_ops = sum(ops_gemm.values()) * args.steps
        out["dense"] = dict(ms=ms_dense, transform_ms=tr_ms / args.steps, transform_tflops=tr_flop / tr_ms / 1e9,
                            gemm_ms=gm_ms / args.steps, gemm_tops=gm_ops / gm_ms / 1e9,
                            tac_ms=timer.ms("tac")[0] / args.steps, quant_ms=timer.ms("quant")[0] / args.steps,
                            per_site_transform_ms={n: timer.ms("transform/" + n)[0] / args.steps for n in flops_tr})
    if args.only in ("dense", "both") and not args.no_fast:
        for d in sites:
            d["Ps"] = sq.sgat_split_basis(d["P"])
        # codes of one step through each transform, compared
        step_dense(Timer(torch))
        torch.cuda.synchronize()
        canon = [(d["Aq"].clone(), d["s_a"].clone()) for d in sites]
        step_dense_fast(Timer(torch))
        torch.cuda.synchronize()
        flips = sum(int(((a ^ d["Aq"]) & 0x0F).ne(0).sum() + ((a ^ d["Aq"]) & 0xF0).ne(0).sum())
                    for (a, _), d in zip(canon, sites))
        ncodes = sum(d["Aq"].numel() * 2 for d in sites)
        ms_f = run(lambda tm, i: step_dense_fast(tm), args.steps, args.warmup)
        tr_ms = sum(timer.ms("ftransform/" + n)[0] for n in flops_tr)
        tr_flop = sum(flops_tr.values()) * args.steps
        out["dense_fast"] = dict(ms=ms_f, transform_ms=tr_ms / args.steps, transform_tflops=tr_flop / tr_ms / 1e9,
                                 code_flips=flips, codes=ncodes)
        del canon
    if args.only in ("folded", "both"):
        ms_fold = run(step_folded, args.steps, args.warmup)
        gm_ms = sum(timer.ms("gemm/" + n)[0] for n in ops_gemm)
        gm_ops = sum(ops_gemm.values()) * args.steps
        qa_ms = sum(timer.ms("quant_act/" + d["site"].name)[0] for d in sites)
        out["folded"] = dict(ms=ms_fold, gemm_ms=gm_ms / args.steps, gemm_tops=gm_ops / gm_ms / 1e9,
                             quant_act_ms=qa_ms / args.steps,
                             per_site_gemm_ms={n: timer.ms("gemm/" + n)[0] / args.steps for n in ops_gemm})

    if args.calibrate_copy:
        # a plain device-to-device copy of known size: its FETCH_SIZE / WRITE_SIZE
        # readings scale the counters of the kernels above to bytes
        src = torch.empty(1 << 29, dtype=torch.float16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if not args.no_w8:
        ms_w8 = run(step_w8, args.steps, args.warmup)
        gm_ms = sum(timer.ms("gemm8/" + n)[0] for n in ops_gemm)
        gm_ops = sum(ops_gemm.values()) * args.steps
        out["w8"] = dict(ms=ms_w8, gemm_tops=gm_ops / gm_ms / 1e9,
                         quant_act_ms=sum(timer.ms("quant_act8/" + n)[0] for n in ops_gemm) / args.steps)

    if not args.no_large:
        out["large"] = large_token_block(torch, sq, synth, dev, max(3, args.steps // 4), 1)
    if not args.no_small:
        out["small"] = small_token_block(torch, sq, synth, dev)
    if not args.no_large:
        out["tac_oproj"] = tac_oproj_block(torch, sq, synth, dev)
    if not args.no_sweep:
        out["sweep"] = sweep_block(torch, sq, synth, dev)
    if not args.no_calib:
        out["calib"] = tac_calibration_block(torch, sq, synth, dev)

    # ---------------------------------------------------------------- CPU baseline
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        threads = min(16, os.cpu_count() or 1)
        n = args.cpu_sample
        rows = np.linspace(0, M - 1, n).astype(int)
        rng = np.random.default_rng(0)
        hosts = []
        for d in sites:
            h = dict(X=d["X"][rows].cpu().numpy(), P=d["P"].cpu().numpy(), st=state_np[rows],
                     Wq=rng.integers(0, 256, (d["N"], d["K"] // 2), dtype=np.uint8),
                     s_w=np.ones(d["N"], np.float32))
            if "tac_M" in d:
                h.update(tM=d["tac_M"].cpu().numpy(), td=d["tac_d"].cpu().numpy(), g=d["g"])
            hosts.append((d, h))
        t1 = time.time()
        for d, h in hosts:
            Aq, s_a = O.quant_act(h["X"], h["st"], h["P"], d["dm"], d["du"], h.get("tM"), h.get("td"),
                                  h.get("g", 0), threads=threads)
            O.gemm(Aq, s_a, h["Wq"], h["s_w"], threads=threads)
        el = time.time() - t1
        cpu = {"value": n / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
               "sample": f"{n} of the {M} tokens through the whole dense-P layer set (TAC, transform, "
                         f"quantise, GEMM against all N); weight preparation excluded; {el:.1f} s"}

    dense = out.get("dense")
    fold = out.get("folded")
    main_ms = dense["ms"] if dense else fold["ms"]
    res = {
        "metric": "W4A4 SGAT-linear TOPS & % int8-MFMA peak; layer-set tokens/s per denoise step",
        "value": M / (main_ms / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": main_ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int4xint4->int32 GEMM, fp32 transform, fp16 I/O",
        "data": "synthetic (seeded; random-init weights and orthogonal bases)",
        "weights": "int4 codes in fragment order (sq_weights_to_frag, once, outside the timed region); W8A8 and "
                   "FP6 variants in their own layouts",
        "config": {"workload": "LLaDA-8B-shaped SGAT layer set (QKV, O+TAC g=16, gate+up, down), "
                               "1024 tokens, dense online P" if dense else
                               "LLaDA-8B-shaped SGAT layer set, 1024 tokens, folded P",
                   "tokens": M, "hidden": 4096, "ffn": 12288, "tac_block": 16},
    }
    if dense:
        ach = dense["transform_tflops"]
        res["roofline"] = {"bound": "alu", "achieved": ach, "peak": PEAK_FP32_VALU_TFLOPS, "unit": "TFLOP/s",
                           "frac": ach / PEAK_FP32_VALU_TFLOPS,
                           "traffic": recorded_traffic("transform", "traffic_bytes_per_launch_step_avg"),
                           "kernel": "transform (dense fp32 x P, fixed order)"}
        res["breakdown_ms"] = {k: dense[k] for k in ("transform_ms", "gemm_ms", "tac_ms", "quant_ms")}
        res["gemm"] = {"tops": dense["gemm_tops"], "frac_int8_peak": dense["gemm_tops"] / PEAK_INT8_TOPS}
        res["sgat_linear_tops"] = sum(ops_gemm.values()) / (dense["ms"] / 1e3) / 1e12
    if fold:
        res["folded_P"] = {
            "value": M / (fold["ms"] / 1e3), "unit": "tokens/s", "ms_per_step": fold["ms"],
            "sgat_linear_tops": sum(ops_gemm.values()) / (fold["ms"] / 1e3) / 1e12,
            "roofline": {"bound": "mfma", "achieved": fold["gemm_tops"], "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                         "frac": fold["gemm_tops"] / PEAK_INT8_TOPS, "kernel": "w4a4 gemm"},
            "quant_act_ms": fold["quant_act_ms"], "per_site_gemm_ms": fold["per_site_gemm_ms"]}
        if not dense:
            res["roofline"] = dict(res["folded_P"]["roofline"], traffic=None)
    if "w8" in out:
        w8 = out["w8"]
        res["w8a8_folded_P"] = {"value": M / (w8["ms"] / 1e3), "unit": "tokens/s", "ms_per_step": w8["ms"],
                                "gemm_tops": w8["gemm_tops"], "gemm_frac_int8_peak": w8["gemm_tops"] / PEAK_INT8_TOPS,
                                "quant_act_ms": w8["quant_act_ms"]}
    if "dense_fast" in out:
        f = out["dense_fast"]
        res["dense_P_fast_transform"] = {
            "value": M / (f["ms"] / 1e3), "unit": "tokens/s", "ms_per_step": f["ms"],
            "transform_ms": f["transform_ms"],
            "roofline": {"bound": "mfma", "achieved": f["transform_tflops"], "peak": PEAK_FP16_TFLOPS,
                         "unit": "TFLOP/s", "frac": f["transform_tflops"] / PEAK_FP16_TFLOPS,
                         "traffic": recorded_traffic("transform_fast", "traffic_bytes_per_launch_step_avg"),
                         "kernel": "transform on the fp16 MFMA (hi + lo split: executes 2x the algorithmic flops)"},
            "codes_differing_from_fixed_order": f["code_flips"], "codes": f["codes"]}
    if "large" in out:
        res["large_token"] = out["large"]
    if "small" in out:
        res["small_token"] = out["small"]
    if "tac_oproj" in out:
        res["tac_oproj"] = out["tac_oproj"]
    if "sweep" in out:
        res["token_sweep_gemm"] = out["sweep"]
    if "calib" in out:
        res["tac_calibration"] = out["calib"]
    if cpu:
        res["cpu_baseline"] = cpu
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
