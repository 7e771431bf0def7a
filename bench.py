"""Benchmark: STaR-Quant W4A4 SGAT layer set per denoising step on one MI355X.

Headline workload: the Dream-7B-shaped layer set (Qwen2.5-7B geometry), a batch of
8 sequences x 2048 tokens = 16384 tokens, each sequence with a mask fraction drawn
uniformly in [0.1, 0.9]: QKV 3584->4608, O 3584->3584 with TAC (g = 16) ahead of
it, gate+up 3584->37888, down 18944->3584, all W4A4 SGAT with fp16 in and out.

One step = the whole per-step hot path for every linear of the set:
    [TAC] -> x P G_s (dense fp32 basis applied online, Eq. 11) -> per-token int4
    -> W4A4 GEMM (Eq. 13)
with the weights prepared offline (Eq. 12, outside the timed region) and every
input resident in HBM.  Nested blocks: the same layer set with P folded into the
weights and the upstream activations (the deployment form: [TAC] -> gate -> int4
-> GEMM); the LLaDA-8B-shaped layer set at 1024 tokens (dense, folded, W8A8 and
with the matrix-core transform); the single 128-token linear; TAC at g = 128 ahead
of the O projection (dense and folded, with the identity-block no-op); the 64-step
denoising sweep at 16, 1024 and 16384 tokens; the small-token steps; the GEMM
token-count sweep; the offline TAC calibration; and the oracle timed on the host.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--only-headline]

Prints one JSON line.  Synthetic, seeded inputs (no datasets, no trained weights).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
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
# fp32 vector, published.  Plain (non-packed) v_fmac_f32 reaches it as well:
# two waves of one SIMD issue together, so the rate is 256 CU x 128 FMA lanes x
# 2 flop x 2.4 GHz, not half of it (a kernel of independent FMA chains
# measures 121.5 TFLOP/s at 16 workgroups per CU, 113 at 2)
PEAK_FP32_TFLOPS = 157.3


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
    ap.add_argument("--cpu-rows", type=int, default=64, help="token rows per linear in the all-cores oracle timing")
    ap.add_argument("--cpu-rows-1core", type=int, default=16, help="token rows per linear in the 1-core timing")
    ap.add_argument("--only-headline", action="store_true", help="the headline step only (no nested blocks)")
    ap.add_argument("--no-llada", action="store_true", help="skip the LLaDA-shaped 1024-token blocks")
    ap.add_argument("--no-w8", action="store_true", help="skip the W8A8 (App. D) folded-basis measurement")
    ap.add_argument("--no-small", action="store_true", help="skip the 16/32/64-token steps")
    ap.add_argument("--no-calib", action="store_true", help="skip the TAC calibration timing")
    ap.add_argument("--no-fast", action="store_true", help="skip the dense step with the matrix-core transform")
    ap.add_argument("--no-sweep", action="store_true", help="skip the GEMM token-count sweep")
    ap.add_argument("--no-denoise", action="store_true", help="skip the 64-step denoising sweep")
    ap.add_argument("--no-fp6", action="store_true", help="skip the FP6 variant of the folded Dream step")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (reference for HBM byte counters)")
    return ap.parse_args()


class Timer:
    """HIP event pairs on the launching stream, per label: the sum, the mean and
    the median duration of that label's launches."""

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

    def times(self, label):
        return [s.elapsed_time(e) for s, e in self.pairs.get(label, [])]

    def ms(self, label):
        t = self.times(label)
        return sum(t), len(t)

    def mean(self, label):
        t = self.times(label)
        return sum(t) / len(t) if t else float("nan")

    def median(self, label):
        t = sorted(self.times(label))
        return t[len(t) // 2] if t else float("nan")

    def reset(self):
        self.pairs = {}


class NullTimer:
    """A timer that records nothing (for captured or whole-step timings)."""

    def wrap(self, label, fn):
        fn()


def run_steps(torch, step, steps, warmup):
    """W untimed warm-up steps, then exactly `steps` steps between two HIP events,
    synchronised on both sides.  step(timer, i) enqueues one step.  Returns the
    milliseconds per step and the timer of the timed steps."""
    for i in range(warmup):
        step(Timer(torch), i)
    torch.cuda.synchronize()
    timer = Timer(torch)
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        step(timer, i)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps, timer


LLC_DEFEAT_BYTES = 800 << 20     # weight copies cycled per timing: over 3x the 256 MB last-level cache


def rotating_copies(Wq, s_w, floor=4):
    """(Wq, s_w) followed by enough clones that one pass over them streams at
    least LLC_DEFEAT_BYTES, so that no call finds its weights in the last-level
    cache."""
    n = max(floor, -(-LLC_DEFEAT_BYTES // (Wq.numel() * Wq.element_size() + s_w.numel() * 4)))
    return [(Wq, s_w)] + [(Wq.clone(), s_w.clone()) for _ in range(n - 1)]


def capture(torch, fn, calls):
    """fn(0) .. fn(calls - 1) captured back to back in one HIP graph."""
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
    return g


def replay_ms(torch, g, calls, replays=5):
    """Median over `replays` graph replays of the milliseconds per captured call."""
    g.replay()                                  # warm
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
    return ts[len(ts) // 2]


def graph_ms(torch, fn, calls, replays=5):
    """Median milliseconds per call of fn(i), i = 0 .. calls - 1, captured back to
    back in one HIP graph, so that no host work sits between the launches."""
    g = capture(torch, fn, calls)
    return replay_ms(torch, g, calls, replays), g


def transform_flop(M, K):
    """Algorithmic flop of the dense transform: the other state's band (K/32
    columns) is never needed, so 2 M K (K - K/32)."""
    return 2.0 * M * K * (K - K // 32)


# ------------------------------------------------------------------ layer sets

def load_sites(torch, sq, synth, dev, cid, state_np, *, with_P, keep_host_rows=None):
    """Device tensors of every linear of workload `cid`: activations, weights,
    optional dense basis, TAC parameters, and the output / workspace buffers.
    keep_host_rows: token rows whose host copies (with P and the TAC parameters)
    are kept for the oracle timing."""
    cfg = synth.CONFIGS[cid]
    M = len(state_np)
    sites, hosts = [], []
    for si, site in enumerate(cfg.sites):
        t = synth.site_tensors(cid, si, state_np, with_P=with_P)
        d = dict(name=site.name, K=site.K, N=site.N, dm=t.dm, du=t.du, tac=site.tac,
                 X=torch.from_numpy(t.X).to(dev), W=torch.from_numpy(t.W).to(dev),
                 P=torch.from_numpy(t.P).to(dev) if with_P else None)
        if site.tac:
            d.update(tac_M=torch.from_numpy(t.tac_M).to(dev), tac_d=torch.from_numpy(t.tac_d).to(dev), g=t.g)
        if keep_host_rows is not None:
            h = dict(name=site.name, K=site.K, N=site.N, dm=t.dm, du=t.du, X=t.X[keep_host_rows].copy(),
                     st=state_np[keep_host_rows].copy(), P=t.P)
            if site.tac:
                h.update(tM=t.tac_M, td=t.tac_d, g=t.g)
            hosts.append(h)
        d["Aq"] = torch.empty((M, site.K // 2), dtype=torch.uint8, device=dev)
        d["s_a"] = torch.empty((M,), dtype=torch.float32, device=dev)
        d["Y"] = torch.empty((M, site.N), dtype=torch.float16, device=dev)
        d["gws"] = torch.empty(max(sq.gemm_workspace_bytes(M, site.N, site.K), 1), dtype=torch.uint8, device=dev)
        sites.append(d)
        del t
    return sites, hosts


def prepare(sq, sites, with_P):
    """Offline weight side (Eq. 12) and the fragment order the GEMM streams."""
    for d in sites:
        Wq, d["s_w"] = sq.sgat_prepare_weights(d["W"], d["P"] if with_P else None)
        d["Wf"] = sq.weights_to_frag(Wq)
        d["Wq"] = Wq


def dense_step_fn(sq, state, sites, xp, z):
    """One dense-P step: per linear [TAC] -> transform and gate -> int4 -> GEMM,
    each launch bracketed by HIP events under its own label."""
    def step(tm, i):
        for d in sites:
            src = d["X"]
            if d["tac"]:
                tm.wrap("tac/" + d["name"], lambda: sq.tac_apply(d["X"], d["tac_M"], d["tac_d"], d["g"],
                                                                 out=z[:d["X"].numel()].view_as(d["X"])))
                src = z[:d["X"].numel()].view_as(d["X"])
            xs = xp[:d["X"].numel()].view(d["X"].shape)
            tm.wrap("transform/" + d["name"], lambda: sq.sgat_transform(src, state, d["P"], d["dm"], d["du"], out=xs))
            tm.wrap("quant/" + d["name"], lambda: sq.sgat_quantize(xs, Aq=d["Aq"], s=d["s_a"]))
            tm.wrap("gemm/" + d["name"], lambda: sq.w4a4_gemm_frag(d["Aq"], d["s_a"], d["Wf"], d["s_w"], Y=d["Y"],
                                                                   ws=d["gws"]))
    return step


def dense_report(M, sites, ms, timer):
    """Per-kernel mean and median launch durations of a dense step, the layer
    set's SGAT-linear TOPS, and the transform / GEMM rates."""
    per = {}
    tr_flop = tr_ms = gm_ops = gm_ms = 0.0
    for d in sites:
        n = d["name"]
        f = transform_flop(M, d["K"])
        ops = 2.0 * M * d["N"] * d["K"]
        t_tr, t_gm = timer.mean("transform/" + n), timer.mean("gemm/" + n)
        per[n] = {"K": d["K"], "N": d["N"],
                  "transform_us": t_tr * 1e3, "transform_us_median": timer.median("transform/" + n) * 1e3,
                  "transform_tflops": f / t_tr / 1e9,
                  "quant_us": timer.mean("quant/" + n) * 1e3,
                  "gemm_us": t_gm * 1e3, "gemm_us_median": timer.median("gemm/" + n) * 1e3,
                  "gemm_tops": ops / t_gm / 1e9, "gemm_frac_int8_peak": ops / t_gm / 1e9 / PEAK_INT8_TOPS}
        if d["tac"]:
            per[n]["tac_us"] = timer.mean("tac/" + n) * 1e3
        tr_flop += f
        tr_ms += t_tr
        gm_ops += ops
        gm_ms += t_gm
    return {"tokens": M, "ms_per_step": ms, "tokens_per_s": M / (ms / 1e3),
            "sgat_linear_tops": gm_ops / (ms / 1e3) / 1e12,
            "transform_ms": tr_ms, "transform_tflops": tr_flop / tr_ms / 1e9,
            "gemm_ms": gm_ms, "gemm_tops": gm_ops / gm_ms / 1e9, "gemm_frac_int8_peak": gm_ops / gm_ms / 1e9 /
            PEAK_INT8_TOPS, "per_site": per}


def transform_roofline(M, d, timer, traffic_key):
    n = d["name"]
    ach = transform_flop(M, d["K"]) / timer.mean("transform/" + n) / 1e9
    return {"bound": "mfma", "achieved": ach, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
            "frac": ach / PEAK_FP32_TFLOPS,
            "traffic": recorded_traffic(traffic_key),
            "kernel": f"transform (dense fp32 x P, fixed order, fp32 matrix cores) at the {n} linear, M={M}, K={d['K']}",
            "flop_per_launch": transform_flop(M, d["K"]), "launch_us_mean": timer.mean("transform/" + n) * 1e3}


def workspaces(torch, sites, M, dev):
    """One transform output buffer for the widest linear and one TAC output
    buffer for the linears with TAC; the linears run one after the other on one
    stream, so they share them."""
    xp = torch.empty(M * max(d["K"] for d in sites), dtype=torch.float32, device=dev)
    ktac = [d["K"] for d in sites if d["tac"]]
    z = torch.empty(M * max(ktac), dtype=torch.float16, device=dev) if ktac else None
    return xp, z


def folded_block(torch, sq, sites, state, M, steps, warmup, copies=1):
    """The deployment form (P folded upstream): per linear the gate + int4
    quantiser (TAC fused ahead of O for g <= 16) and the W4A4 GEMM.  `copies`
    rotating sets of prepared weights keep the last-level cache from serving them."""
    for d in sites:
        d["qws"] = torch.empty(max(sq.quant_act_workspace_bytes(M, d["K"], False, d["tac"]), 1), dtype=torch.uint8,
                               device=d["X"].device)
    wsets = [[(d["Wf"], d["s_w"]) for d in sites]] + [[(d["Wf"].clone(), d["s_w"].clone()) for d in sites]
                                                      for _ in range(copies - 1)]

    def step(tm, it):
        for d, (Wf, s_w) in zip(sites, wsets[it % copies]):
            tm.wrap("q/" + d["name"], lambda: sq.sgat_quant_act(d["X"], state, None, d["dm"], d["du"], d.get("tac_M"),
                                                                 d.get("tac_d"), d.get("g", 0), Aq=d["Aq"],
                                                                 s_a=d["s_a"], ws=d["qws"]))
            tm.wrap("g/" + d["name"], lambda: sq.w4a4_gemm_frag(d["Aq"], d["s_a"], Wf, s_w, Y=d["Y"], ws=d["gws"]))
    ms, timer = run_steps(torch, step, steps, warmup)
    # the same steps, one per weight set, captured back to back in one HIP graph
    # (no host work or timing events between the launches)
    graph_ms_step, g = graph_ms(torch, lambda i: step(NullTimer(), i), copies, replays=max(3, min(steps, 10)))
    del g
    per, tot_ops, tot_ms = {}, 0.0, 0.0
    for d in sites:
        n = d["name"]
        gms = timer.mean("g/" + n)
        ops = 2.0 * M * d["N"] * d["K"]
        per[n] = {"M": M, "N": d["N"], "K": d["K"], "gemm_us": gms * 1e3, "gemm_us_median": timer.median("g/" + n) * 1e3,
                  "tops": ops / gms / 1e9, "frac_int8_peak": ops / gms / 1e9 / PEAK_INT8_TOPS,
                  "quant_act_us": timer.mean("q/" + n) * 1e3}
        tot_ops += ops
        tot_ms += gms
    del wsets
    return {"tokens": M, "ms_per_step": ms, "tokens_per_s": M / (ms / 1e3),
            "graph_ms_per_step": graph_ms_step, "graph_tokens_per_s": M / (graph_ms_step / 1e3),
            "sgat_linear_tops": tot_ops / (ms / 1e3) / 1e12,
            "gemm_tops": tot_ops / tot_ms / 1e9, "gemm_frac_int8_peak": tot_ops / tot_ms / 1e9 / PEAK_INT8_TOPS,
            "per_site": per}


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
    """The same folded layer set with the codes carried as e3m2 on the FP6 matrix
    cores: per linear the gate + int4 quantiser, the conversion of the activation
    codes to the FP6 operand layout, and the GEMM on FP6 operands (weights
    converted once, offline).  Its outputs are checked equal to the int4 path's."""
    ref = {d["name"]: d["Y"].clone() for d in sites}
    for d in sites:
        d["W6"] = sq.codes_to_fp6(d["Wq"])
        d["A6"] = torch.empty((M, sq.fp6_row_bytes(d["K"])), dtype=torch.uint8, device=d["Aq"].device)
        d["Y6"] = torch.empty_like(d["Y"])

    def step(tm, i):
        for d in sites:
            tm.wrap("q/" + d["name"], lambda: sq.sgat_quant_act(d["X"], state, None, d["dm"], d["du"], d.get("tac_M"),
                                                                 d.get("tac_d"), d.get("g", 0), Aq=d["Aq"],
                                                                 s_a=d["s_a"], ws=d["qws"]))
            tm.wrap("c/" + d["name"], lambda: sq.codes_to_fp6(d["Aq"], out=d["A6"]))
            tm.wrap("g/" + d["name"], lambda: sq.w4a4_gemm_fp6(d["A6"], d["s_a"], d["W6"], d["s_w"], d["K"],
                                                                Y=d["Y6"]))
    ms, timer = run_steps(torch, step, steps, warmup)
    per, tot_ops, tot_ms = {}, 0.0, 0.0
    for d in sites:
        gms = timer.mean("g/" + d["name"])
        ops = 2.0 * M * d["N"] * d["K"]
        per[d["name"]] = {"gemm_us": gms * 1e3, "tops": ops / gms / 1e9,
                          "frac_fp6_peak": ops / gms / 1e9 / PEAK_FP6_TFLOPS,
                          "frac_int8_peak": ops / gms / 1e9 / PEAK_INT8_TOPS,
                          "convert_us": timer.mean("c/" + d["name"]) * 1e3}
        tot_ops += ops
        tot_ms += gms
    same = all(torch.equal(ref[d["name"]], d["Y6"]) for d in sites)
    dom = max(per, key=lambda n: per[n]["gemm_us"])
    for d in sites:
        del d["W6"], d["A6"], d["Y6"]
    return {"ms_per_step": ms, "tokens_per_s": M / (ms / 1e3), "gemm_tops": tot_ops / tot_ms / 1e9,
            "per_site": per, "outputs_equal_int4_path": same,
            "roofline": {"bound": "mfma", "achieved": per[dom]["tops"], "peak": PEAK_FP6_TFLOPS, "unit": "TFLOP/s",
                         "frac": per[dom]["frac_fp6_peak"],
                         "traffic": recorded_traffic("gemm_fp6_gate_up") if dom == "gate_up" else None,
                         "kernel": f"w4a4 gemm on FP6 operands ({dom})"}}


# ------------------------------------------------------------------ headline

def headline_block(torch, sq, synth, dev, args):
    """Dream-shaped layer set, 8 x 2048 tokens, dense P, TAC g = 16 ahead of O."""
    state_np = synth.config_state(synth.DREAM)
    M = len(state_np)
    rows = np.random.default_rng(synth.SEED).choice(M, size=max(args.cpu_rows, args.cpu_rows_1core), replace=False)
    t0 = time.time()
    sites, hosts = load_sites(torch, sq, synth, dev, synth.DREAM, state_np, with_P=True,
                              keep_host_rows=None if args.no_cpu_baseline else rows)
    print(f"# Dream-shaped inputs generated in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    state = torch.from_numpy(state_np).to(dev)
    prepare(sq, sites, True)
    xp, z = workspaces(torch, sites, M, dev)
    torch.cuda.synchronize()
    ms, timer = run_steps(torch, dense_step_fn(sq, state, sites, xp, z), args.steps, args.warmup)
    rep = dense_report(M, sites, ms, timer)
    down = next(d for d in sites if d["name"] == "down")
    rep["roofline"] = transform_roofline(M, down, timer, "transform_dream_down")
    rep["workload"] = ("Dream-7B-shaped SGAT layer set (QKV 3584->4608, O+TAC g=16 3584->3584, gate+up "
                       "3584->37888, down 18944->3584), 8 x 2048 tokens, dense online P")
    del xp, z
    for d in sites:
        d["P"] = None
    torch.cuda.empty_cache()
    return rep, sites, state, state_np, hosts, rows


def cpu_baseline_block(hosts, M, rows_all, rows_1core):
    """The oracle as it stands, timed on the host: every linear of the Dream-shaped
    dense-P layer set (TAC, transform and gate, quantise, GEMM against all N
    output channels) on a seeded subset of the 16384 token rows; rows are
    independent, so tokens/s scale linearly to the whole batch.  All host cores
    (threads over rows) and one core."""
    from oracle import oracle as O
    nproc = os.cpu_count() or 1
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        pass
    ncpu = min(16, nproc)            # the host share of one GPU
    model = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    rng = np.random.default_rng(0)
    wq = {h["name"]: (rng.integers(0, 256, (h["N"], h["K"] // 2), dtype=np.uint8), np.ones(h["N"], np.float32))
          for h in hosts}

    def run(n, threads):
        t1 = time.time()
        for h in hosts:
            Aq, s_a = O.quant_act(h["X"][:n], h["st"][:n], h["P"], h["dm"], h["du"], h.get("tM"), h.get("td"),
                                  h.get("g", 0), threads=threads)
            O.gemm(Aq, s_a, *wq[h["name"]], threads=threads)
        return time.time() - t1

    el_all = run(rows_all, ncpu)
    el_one = run(rows_1core, 1)
    return {"value": rows_all / el_all, "unit": "tokens/s", "cores": ncpu, "kind": "oracle",
            "sample": f"{rows_all} seeded token rows of the {M} (scaled linearly: rows are independent) through "
                      f"every linear of the Dream-shaped dense-P layer set (TAC g=16 for O, transform and gate, "
                      f"quantise, GEMM against all N); weight preparation excluded; {el_all:.1f} s on "
                      f"{ncpu} threads",
            "value_1core": rows_1core / el_one, "sample_1core": f"{rows_1core} of the same rows on 1 thread, "
                                                                f"{el_one:.1f} s",
            "cpu_model": model, "nproc": nproc}


# ------------------------------------------------------------------ nested blocks

def llada_blocks(torch, sq, synth, dev, args):
    """LLaDA-shaped layer set, 1024 tokens: dense P (the fixed-order transform and
    the matrix-core transform), folded P, and W8A8 folded."""
    state_np = synth.config_state(synth.LLADA)
    M = len(state_np)
    sites, _ = load_sites(torch, sq, synth, dev, synth.LLADA, state_np, with_P=True)
    state = torch.from_numpy(state_np).to(dev)
    prepare(sq, sites, True)
    xp, z = workspaces(torch, sites, M, dev)
    out = {}
    ms, timer = run_steps(torch, dense_step_fn(sq, state, sites, xp, z), max(5, args.steps // 2), 2)
    rep = dense_report(M, sites, ms, timer)
    rep["roofline"] = transform_roofline(M, next(d for d in sites if d["name"] == "down"), timer,
                                         "transform_llada_down")
    rep["workload"] = "LLaDA-8B-shaped SGAT layer set, 1024 tokens, dense online P (TAC g=16 ahead of O)"
    out["dense_P"] = rep
    if not args.no_fast:
        for d in sites:
            d["Ps"] = sq.sgat_split_basis(d["P"])
        canon = [(d["Aq"].clone(), d["s_a"].clone()) for d in sites]

        def step_fast(tm, i):
            for d in sites:
                src = d["X"]
                if d["tac"]:
                    zz = z[:d["X"].numel()].view_as(d["X"])
                    tm.wrap("tac/" + d["name"], lambda: sq.tac_apply(d["X"], d["tac_M"], d["tac_d"], d["g"], out=zz))
                    src = zz
                xs = xp[:d["X"].numel()].view(d["X"].shape)
                tm.wrap("transform/" + d["name"], lambda: sq.sgat_transform_fast(src, state, d["Ps"], d["dm"], d["du"],
                                                                                 out=xs))
                tm.wrap("quant/" + d["name"], lambda: sq.sgat_quantize(xs, Aq=d["Aq"], s=d["s_a"]))
                tm.wrap("gemm/" + d["name"], lambda: sq.w4a4_gemm_frag(d["Aq"], d["s_a"], d["Wf"], d["s_w"],
                                                                       Y=d["Y"], ws=d["gws"]))
        ms, timer = run_steps(torch, step_fast, max(5, args.steps // 2), 2)
        flips = sum(int(((a ^ d["Aq"]) & 0x0F).ne(0).sum() + ((a ^ d["Aq"]) & 0xF0).ne(0).sum())
                    for (a, _), d in zip(canon, sites))
        ncodes = sum(d["Aq"].numel() * 2 for d in sites)
        f = dense_report(M, sites, ms, timer)
        f_ach = f["transform_tflops"]
        out["dense_P_fast_transform"] = {
            "tokens_per_s": f["tokens_per_s"], "ms_per_step": ms, "transform_ms": f["transform_ms"],
            "roofline": {"bound": "mfma", "achieved": f_ach, "peak": PEAK_FP16_TFLOPS, "unit": "TFLOP/s",
                         "frac": f_ach / PEAK_FP16_TFLOPS,
                         "traffic": recorded_traffic("transform_fast", "traffic_bytes_per_launch_step_avg"),
                         "kernel": "transform on the fp16 MFMA (hi + lo split: executes 2x the algorithmic flops)"},
            "codes_differing_from_fixed_order": flips, "codes": ncodes}
        for d in sites:
            del d["Ps"]
        del canon
    del xp, z
    for d in sites:
        d["P"] = None
    torch.cuda.empty_cache()
    # folded P: weights prepared without P (the activations stand for inputs already in the P basis)
    prepare(sq, sites, False)
    fold = folded_block(torch, sq, sites, state, M, args.steps, args.warmup, copies=8)
    fold["workload"] = "LLaDA-8B-shaped SGAT layer set, 1024 tokens, folded P, 8 rotating weight sets"
    fold["roofline"] = {"bound": "mfma", "achieved": fold["gemm_tops"], "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                        "frac": fold["gemm_frac_int8_peak"],
                        "traffic": recorded_traffic("gemm_llada_folded_step", "traffic_bytes_per_step"),
                        "kernel": "w4a4 gemm (all four sites; traffic per step)"}
    out["folded_P"] = fold
    if not args.no_w8:
        # int8 weights in fragment order (as the 4-bit ones), 4 rotating sets
        w8 = []
        for d in sites:
            Wq8, s_w8 = sq.sgat_prepare_weights_w8(d["W"], None)
            w8.append(dict(Wf8=sq.weights_to_frag(Wq8), s_w8=s_w8,
                           Aq8=torch.empty((M, d["K"]), dtype=torch.int8, device=dev),
                           gws8=torch.empty(max(sq.gemm_workspace_bytes(M, d["N"], d["K"], 8), 1), dtype=torch.uint8,
                                            device=dev)))
            del Wq8
        copies = [[(e["Wf8"], e["s_w8"]) for e in w8]] + [[(e["Wf8"].clone(), e["s_w8"].clone()) for e in w8]
                                                          for _ in range(3)]

        def step_w8(tm, it):
            for d, e, (Wf8, s_w8) in zip(sites, w8, copies[it % len(copies)]):
                tm.wrap("q8/" + d["name"], lambda: sq.sgat_quant_act_w8(d["X"], state, None, d["dm"], d["du"],
                                                                       d.get("tac_M"), d.get("tac_d"), d.get("g", 0),
                                                                       Aq=e["Aq8"], s_a=d["s_a"], ws=d["qws"]))
                tm.wrap("g8/" + d["name"], lambda: sq.w8a8_gemm_frag(e["Aq8"], d["s_a"], Wf8, s_w8, Y=d["Y"],
                                                                     ws=e["gws8"]))
        ms, timer = run_steps(torch, step_w8, args.steps, args.warmup)
        graph_ms_step, g = graph_ms(torch, lambda i: step_w8(NullTimer(), i), len(copies),
                                    replays=max(3, min(args.steps, 10)))
        del g
        ops = sum(2.0 * M * d["N"] * d["K"] for d in sites)
        gms = sum(timer.mean("g8/" + d["name"]) for d in sites)
        per = {d["name"]: {"gemm_us": timer.mean("g8/" + d["name"]) * 1e3,
                           "frac_int8_peak": 2.0 * M * d["N"] * d["K"] / timer.mean("g8/" + d["name"]) / 1e9
                           / PEAK_INT8_TOPS} for d in sites}
        out["w8a8_folded_P"] = {"tokens_per_s": M / (ms / 1e3), "ms_per_step": ms,
                                "graph_ms_per_step": graph_ms_step, "graph_tokens_per_s": M / (graph_ms_step / 1e3),
                                "gemm_tops": ops / gms / 1e9,
                                "gemm_frac_int8_peak": ops / gms / 1e9 / PEAK_INT8_TOPS,
                                "quant_act_ms": sum(timer.mean("q8/" + d["name"]) for d in sites),
                                "weights": "int8 in fragment order, 4 rotating sets", "per_site": per}
        del w8, copies
    del sites
    torch.cuda.empty_cache()
    return out


def single_linear_block(torch, sq, synth, dev):
    """The 128-token single linear (K = N = 512), dense P and folded, graph-replayed."""
    state_np = synth.config_state(synth.SINGLE_LINEAR)
    M = len(state_np)
    sites, _ = load_sites(torch, sq, synth, dev, synth.SINGLE_LINEAR, state_np, with_P=True)
    state = torch.from_numpy(state_np).to(dev)
    d = sites[0]
    Wq, s_w = sq.sgat_prepare_weights(d["W"], d["P"])
    Wf = sq.weights_to_frag(Wq)
    qws = torch.empty(sq.quant_act_workspace_bytes(M, d["K"], True, False), dtype=torch.uint8, device=dev)

    def step(i):
        sq.sgat_quant_act(d["X"], state, d["P"], d["dm"], d["du"], Aq=d["Aq"], s_a=d["s_a"], ws=qws)
        sq.w4a4_gemm_frag(d["Aq"], d["s_a"], Wf, s_w, Y=d["Y"], ws=d["gws"])
    ms, g = graph_ms(torch, step, 16, replays=7)
    del g
    ops = 2.0 * M * d["N"] * d["K"]
    return {"workload": "single SGAT W4A4 linear, 128 tokens, K = N = 512, dense P, HIP-graph replay",
            "tokens": M, "us_per_step": ms * 1e3, "tokens_per_s": M / (ms / 1e3),
            "sgat_linear_tops": ops / (ms / 1e3) / 1e12}


def tac_oproj_block(torch, sq, synth, dev, steps=3):
    """TAC (32 blocks of 128) on 8 x 2048 attention outputs of width 4096, then the
    gate + int4 quantiser and the 4096 -> 4096 W4A4 GEMM: dense P (TAC, transform,
    quantise, GEMM) and folded P (TAC, gate + quantise, GEMM), and the
    identity-block case checked to leave the codes of the plain path unchanged."""
    st_np = synth.config_state(synth.TAC_OPROJ)
    M = len(st_np)
    state = torch.from_numpy(st_np).to(dev)
    t = synth.site_tensors(synth.TAC_OPROJ, 0, st_np, with_P=True)
    K, N, g = t.site.K, t.site.N, t.g
    W = torch.from_numpy(t.W).to(dev)
    P = torch.from_numpy(t.P).to(dev)
    X = torch.from_numpy(t.X).to(dev)
    tM, td = torch.from_numpy(t.tac_M).to(dev), torch.from_numpy(t.tac_d).to(dev)
    Z = torch.empty_like(X)
    xp = torch.empty((M, K), dtype=torch.float32, device=dev)
    Aq = torch.empty((M, K // 2), dtype=torch.uint8, device=dev)
    s_a = torch.empty((M,), dtype=torch.float32, device=dev)
    Y = torch.empty((M, N), dtype=torch.float16, device=dev)
    gws = torch.empty(max(sq.gemm_workspace_bytes(M, N, K), 1), dtype=torch.uint8, device=dev)
    out = {"workload": f"TAC g = {g} + O projection {K}->{N}, 8 x 2048 tokens", "tokens": M}
    for mode in ("dense_P", "folded_P"):
        Wq, s_w = sq.sgat_prepare_weights(W, P if mode == "dense_P" else None)
        Wf = sq.weights_to_frag(Wq)
        del Wq

        def step(tm, i):
            tm.wrap("tac", lambda: sq.tac_apply(X, tM, td, g, out=Z))
            if mode == "dense_P":
                tm.wrap("transform", lambda: sq.sgat_transform(Z, state, P, t.dm, t.du, out=xp))
                tm.wrap("q", lambda: sq.sgat_quantize(xp, Aq=Aq, s=s_a))
            else:
                tm.wrap("q", lambda: sq.sgat_quant_act(Z, state, None, t.dm, t.du, Aq=Aq, s_a=s_a))
            tm.wrap("g", lambda: sq.w4a4_gemm_frag(Aq, s_a, Wf, s_w, Y=Y, ws=gws))
        ms, timer = run_steps(torch, step, steps, 1)
        tac_ms, g_ms = timer.mean("tac"), timer.mean("g")
        tac_flop = 2.0 * M * K * g
        rec = {"ms_per_step": ms, "tokens_per_s": M / (ms / 1e3), "tac_ms": tac_ms, "quant_ms": timer.mean("q"),
               "gemm_ms": g_ms, "gemm_frac_int8_peak": 2.0 * M * N * K / g_ms / 1e9 / PEAK_INT8_TOPS,
               "roofline": {"bound": "mfma", "achieved": tac_flop / tac_ms / 1e9, "peak": PEAK_FP32_TFLOPS,
                            "unit": "TFLOP/s", "frac": tac_flop / tac_ms / 1e9 / PEAK_FP32_TFLOPS,
                            "traffic": recorded_traffic("tac_g128") if g == 128 else None,
                            "kernel": f"tac (g = {g})"}}
        if mode == "dense_P":
            tr_ms = timer.mean("transform")
            rec["transform_ms"] = tr_ms
            rec["transform_tflops"] = transform_flop(M, K) / tr_ms / 1e9
        out[mode] = rec
        del Wf
    # identity blocks: TAC is a no-op, so the codes equal those of the plain (no TAC) path
    tI, dI = synth.tac_params(K, g, None, identity=True)
    tIM, tId = torch.from_numpy(tI).to(dev), torch.from_numpy(dI).to(dev)
    sq.tac_apply(X, tIM, tId, g, out=Z)
    Aq_i, s_i = sq.sgat_quant_act(Z, state, None, t.dm, t.du)
    Aq_p, s_p = sq.sgat_quant_act(X, state, None, t.dm, t.du)
    out["identity_blocks_no_op"] = bool(torch.equal(Aq_i, Aq_p) and torch.equal(s_i, s_p))
    del X, Z, xp, P, W, Y
    torch.cuda.empty_cache()
    return out


def denoise_sweep_block(torch, sq, synth, dev, token_counts=(16, 1024, 16384)):
    """The 64-step denoising sweep on the LLaDA-shaped layer set (folded P): at
    each token count, every step t = 0 .. 64 (the mask fraction of the 256-token
    generation block falling linearly from 1 to 0 after a 512-token prompt,
    token i taking position (512 + i) mod 768) and the edge layouts
    (all masked, none masked, alternating), each step graph-replayed.  The TAC
    parameters are fixed across steps and only the state changes, so the
    per-step time should not depend on t: max / min over t is reported.  The
    activations are drawn once per token count (for step 32); only the state
    vector changes from step to step."""
    cfg = synth.CONFIGS[synth.LLADA_SWEEP]
    out = {}
    meta = []
    for si, site in enumerate(cfg.sites):
        t = synth.site_tensors(synth.LLADA_SWEEP, si, synth.config_state(synth.LLADA_SWEEP, M=16, t=32),
                               with_P=False)
        W = torch.from_numpy(t.W).to(dev)
        Wq, s_w = sq.sgat_prepare_weights(W, None)
        meta.append((site, sq.weights_to_frag(Wq), s_w))
        del W, Wq, t
    for M in token_counts:
        st32 = synth.config_state(synth.LLADA_SWEEP, M=M, t=32)
        sites = []
        for si, (site, Wf, s_w) in enumerate(meta):
            t = synth.site_tensors(synth.LLADA_SWEEP, si, st32, with_W=False, with_P=False)
            K, N = site.K, site.N
            d = dict(name=site.name, K=K, N=N, dm=t.dm, du=t.du, X=torch.from_numpy(t.X).to(dev),
                     Aq=torch.empty((M, K // 2), dtype=torch.uint8, device=dev),
                     s_a=torch.empty((M,), dtype=torch.float32, device=dev),
                     Y=torch.empty((M, N), dtype=torch.float16, device=dev),
                     gws=torch.empty(max(sq.gemm_workspace_bytes(M, N, K), 1), dtype=torch.uint8, device=dev),
                     qws=torch.empty(max(sq.quant_act_workspace_bytes(M, K, False, site.tac), 1), dtype=torch.uint8,
                                     device=dev))
            if site.tac:
                d.update(tac_M=torch.from_numpy(t.tac_M).to(dev), tac_d=torch.from_numpy(t.tac_d).to(dev), g=t.g)
            sites.append(d)
            del t
        copies = 8 if M <= 64 else 1        # small steps stream their weights: keep them out of the LLC
        wsets = [[(Wf, s_w) for (_, Wf, s_w) in meta]] + [[(Wf.clone(), s_w.clone()) for (_, Wf, s_w) in meta]
                                                          for _ in range(copies - 1)]
        layouts = [(str(tt), synth.config_state(synth.LLADA_SWEEP, M=M, t=tt)) for tt in range(65)]
        layouts += [(k, synth.state_edge(M, k)) for k in ("all_masked", "none_masked", "alternating")]
        calls = copies if M <= 64 else (4 if M <= 1024 else 1)
        graphs = {}
        for label, st_np in layouts:
            state = torch.from_numpy(st_np).to(dev)

            def step(i, state=state):
                for d, (Wf, s_w) in zip(sites, wsets[i % copies]):
                    sq.sgat_quant_act(d["X"], state, None, d["dm"], d["du"], d.get("tac_M"), d.get("tac_d"),
                                      d.get("g", 0), Aq=d["Aq"], s_a=d["s_a"], ws=d["qws"])
                    sq.w4a4_gemm_frag(d["Aq"], d["s_a"], Wf, s_w, Y=d["Y"], ws=d["gws"])
            graphs[label] = (capture(torch, step, calls), state)
        # every step's graph replayed in turn, several passes (clocks warmed
        # first), and each step's median over the passes: drifts of the clock
        # over the sweep then fall on every step alike
        for g, _ in graphs.values():
            g.replay()
        torch.cuda.synchronize()
        passes = 5 if M <= 1024 else 3
        per = {label: [] for label in graphs}
        for _ in range(passes):
            for label, (g, _) in graphs.items():
                per[label].append(replay_ms(torch, g, calls, replays=1))
        times = {label: sorted(v)[len(v) // 2] * 1e3 for label, v in per.items()}
        del graphs
        steps_us = [times[str(tt)] for tt in range(65)]
        out[str(M)] = {"us_per_step_t0_to_t64": steps_us,
                       "us_per_step_edges": {k: times[k] for k in ("all_masked", "none_masked", "alternating")},
                       "max_over_min_t": max(steps_us) / min(steps_us),
                       "median_us": float(np.median(steps_us)),
                       "tokens_per_s_median": M / (float(np.median(steps_us)) / 1e6)}
        del sites, wsets
        torch.cuda.empty_cache()
    del meta
    torch.cuda.empty_cache()
    return {"workload": "LLaDA-8B-shaped layer set (folded P), denoising steps t = 0..64 (mask fraction 1 -> 0) "
                        "and the edge layouts, at 16, 1024 and 16384 tokens, each step graph-replayed",
            "per_tokens": out}


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


def sweep_block(torch, sq, synth, dev, token_counts=(16, 64, 256, 1024, 4096, 16384)):
    """GEMM token-count sweep (LLaDA shapes, step 32 of 64, folded P): the W4A4
    GEMM of every linear, graph-replayed with rotating weights, as achieved TOP/s
    and algorithmic GB/s, from memory-bound to compute-bound."""
    cfg = synth.CONFIGS[synth.LLADA_SWEEP]
    st_max = synth.config_state(synth.LLADA_SWEEP, M=max(token_counts), t=32)
    meta = []
    for si, site in enumerate(cfg.sites):
        t = synth.site_tensors(synth.LLADA_SWEEP, si, st_max[:16], with_P=False)
        W = torch.from_numpy(t.W).to(dev)
        Wq, s_w = sq.sgat_prepare_weights(W, None)
        meta.append((site, sq.weights_to_frag(Wq), s_w))
        del W, Wq, t
    rots = [rotating_copies(Wf, s_w) for (_, Wf, s_w) in meta]
    out = {}
    for M in token_counts:
        rec = {}
        for si, (site, _, _) in enumerate(meta):
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
    del rots, meta
    torch.cuda.empty_cache()
    return {"workload": "W4A4 GEMMs of the LLaDA-shaped layer set, token counts 16 ... 16384, graph-replayed, "
                        ">= 800 MB of rotating weights per GEMM", "per_tokens": out}


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
        print(json.dumps({"error": "this benchmark runs on exactly one GPU (one GPU's share of the layer set); "
                                   "--gpus must be 1"}), flush=True)
        sys.exit(2)
    import torch
    import paper_2606_04945_amd as sq
    import synth

    sq.lib()                                    # raises if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    head, sites, state, state_np, hosts, rows = headline_block(torch, sq, synth, dev, args)
    M = head["tokens"]
    nested = {}
    if not args.only_headline:
        # the same Dream-shaped inputs with P folded (weights prepared without P)
        prepare(sq, sites, False)
        large = folded_block(torch, sq, sites, state, M, max(3, args.steps // 4), 1)
        large["workload"] = ("Dream-7B-shaped SGAT layer set, 8 x 2048 tokens, folded P (TAC g=16 fused with the "
                             "O quantiser)")
        dom = max(large["per_site"], key=lambda n: large["per_site"][n]["gemm_us"])
        large["roofline"] = {"bound": "mfma", "achieved": large["per_site"][dom]["tops"], "peak": PEAK_INT8_TOPS,
                             "unit": "TOP/s", "frac": large["per_site"][dom]["frac_int8_peak"],
                             "traffic": recorded_traffic("gemm_large") if dom == "gate_up" else None,
                             "kernel": f"w4a4 gemm ({dom})"}
        if not args.no_fp6:
            large["fp6"] = fp6_variant(torch, sq, sites, state, M, max(3, args.steps // 4), 1)
        for d in sites:
            large["per_site"][d["name"]]["vendor_int8_gemm_us"] = vendor_int8_us(torch, M, d["N"], d["K"], dev)
        nested["dream_folded_P"] = large
    del sites
    torch.cuda.empty_cache()

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline_block(hosts, M, min(args.cpu_rows, len(rows)), min(args.cpu_rows_1core, len(rows)))
    del hosts

    if not args.only_headline:
        if not args.no_llada:
            nested.update({"llada_" + k: v for k, v in llada_blocks(torch, sq, synth, dev, args).items()})
        nested["single_linear"] = single_linear_block(torch, sq, synth, dev)
        nested["tac_oproj"] = tac_oproj_block(torch, sq, synth, dev)
        if not args.no_denoise:
            nested["denoise_sweep"] = denoise_sweep_block(torch, sq, synth, dev)
        if not args.no_small:
            nested["small_token"] = small_token_block(torch, sq, synth, dev)
        if not args.no_sweep:
            nested["token_sweep_gemm"] = sweep_block(torch, sq, synth, dev)
        if not args.no_calib:
            nested["tac_calibration"] = tac_calibration_block(torch, sq, synth, dev)
    if args.calibrate_copy:
        # a plain device-to-device copy of known size: its FETCH_SIZE / WRITE_SIZE
        # readings scale the counters of the kernels above to bytes
        src = torch.empty(1 << 29, dtype=torch.float16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    res = {
        "metric": "W4A4 SGAT-linear TOPS & % int8-MFMA peak; layer-set tokens/s per denoise step",
        "value": head["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int4xint4->int32 GEMM, fp32 transform, fp16 I/O",
        "data": "synthetic (seeded; random-init weights and orthogonal bases)",
        "weights": "int4 codes in fragment order (sq_weights_to_frag, once, outside the timed region)",
        "config": {"workload": head["workload"], "tokens": M, "batch": 8, "seq_len": 2048, "hidden": 3584,
                   "ffn": 18944, "tac_block": 16},
        "roofline": head["roofline"],
        "sgat_linear_tops": head["sgat_linear_tops"],
        "gemm": {"tops": head["gemm_tops"], "frac_int8_peak": head["gemm_frac_int8_peak"]},
        "breakdown_ms": {"transform": head["transform_ms"], "gemm": head["gemm_ms"],
                         "quant": sum(v["quant_us"] for v in head["per_site"].values()) / 1e3,
                         "tac": sum(v.get("tac_us", 0.0) for v in head["per_site"].values()) / 1e3},
        "per_site": head["per_site"],
    }
    res.update(nested)
    if cpu:
        res["cpu_baseline"] = cpu
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
