#!/usr/bin/env python3
"""Benchmark of the masked MoE-layer forward (FlexMoE online clipping) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--table NAME]

A step is one flexmoe_layer_forward: routing, dispatch, the gate/up GEMM with
fused SwiGLU (routed experts truncated to k_e channels, plus the shared
expert when the layer has one), the down GEMM and the weighted combine.
Inputs are seeded synthetic tensors already resident in HBM; the weights are
rotated over --copies device copies so that no step finds them in the 256 MB
last-level cache.

Prints ONE JSON line on stdout.  The headline (`value`, `ms_per_step`) is the
Mixtral-8x7B-shaped layer (T = 16384, d = 4096, 8 experts of I = 14336, top-2,
Zipf(1.2) expert load, its own 50 % keep table): tokens/s over exactly K
timed steps, after at least W warm-up steps and --min-warmup-s seconds.
`step_ms` gives the median and p10/p90 of the K steps' individual durations
(a second pass with an event between steps).  `roofline` describes the
dominant kernel, the gate/up GEMM: its algorithmic flops per launch over its
average launch time, measured with HIP events around each launch on its own
stream in a third pass; this layer has no shared expert, so the launch runs
alone.  `cpu_baseline` is the CPU oracle timed on a bounded sample of the
same workload.  `per_budget` repeats the headline layer at the nested
100/80/60/40/20 % tables, each also run offline (compact weights: the
paper's static checkpoint mode) and through the paper's bucketed kernel
design (an ablation).

Further objects, each on its own layer: `qwen2_prefill` (the Qwen2-57B-A14B-
shaped layer, T = 8192, at the five nested budgets), `decode` (the same layer
at 1, 8 and 64 tokens per step with the budget switching every step, the
fixed-table and pointer-switch references and the cost of one budget
switch), and `qwen15` (the Qwen1.5-MoE-A2.7B-shaped layer, T = 4096, with
the device channel saliency of Eq. 2 and one action-learning step).
`dense_gemm_reference` times the vendor library's dense bf16 GEMM
(torch.matmul) on two dense shapes, as context for what a plain contraction
reaches on the same GPU.
"""
import argparse
import contextlib
import gc
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0    # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3      # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
RIDGE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)
DECODE_MAX_T = 64            # the library runs its weight-streaming GEMMs for T <= 64 (bf16)
GEMV_MAX_T = 8               # up to this many tokens the routed experts' GEMMs run on the vector ALUs,
                             # above it on 64-wide matrix-core tiles
DECODE_WIDE_SHARED_T = 5     # above this many tokens the shared expert's take the 64-wide tiles
HEADLINE = "mixtral_8x7b"
EXTRAS = ("qwen2_prefill", "decode", "qwen15")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=100, help="untimed steps first (at least this many)")
    ap.add_argument("--min-warmup-s", type=float, default=2.0,
                    help="warm-up also lasts at least this long: clocks and caches settle over ~100 "
                         "prefill steps, whatever --warmup says")
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--table", default=None, help="keep table (default: the workload's own, else kept100)")
    ap.add_argument("--decode-T", type=int, default=1, help="tokens per step of the decode workload")
    ap.add_argument("--copies", type=int, default=3, help="weight copies rotated over the steps")
    ap.add_argument("--extras", default=",".join(EXTRAS),
                    help="comma list of further sections (%s), or 'none'" % ",".join(EXTRAS))
    ap.add_argument("--extra-steps", type=int, default=0,
                    help="timed steps of the further sections (default: --steps, at least 20)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baselines")
    ap.add_argument("--no-per-budget", action="store_true")
    ap.add_argument("--no-saliency", action="store_true", help="skip the channel-saliency measurement")
    ap.add_argument("--saliency-T", type=int, default=0,
                    help="tokens per calibration batch of the saliency (default: the workload's T)")
    ap.add_argument("--saliency-steps", type=int, default=10)
    ap.add_argument("--no-action", action="store_true", help="skip the action-learning step measurement")
    ap.add_argument("--graphs", action="store_true",
                    help="decode workload: replay each step from a HIP graph (captured through "
                         "torch.cuda.graph); measured no faster than eager calls")
    ap.add_argument("--action-steps", type=int, default=10)
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target work of the main CPU baseline")
    ap.add_argument("--bucket-align", type=int, default=128,
                    help="k_align of the bucketed ablation in the per-budget results")
    ap.add_argument("--no-dense-reference", action="store_true",
                    help="skip timing the vendor library's dense bf16 GEMM (torch.matmul) on two reference shapes")
    ap.add_argument("--dense-reference-only", action="store_true",
                    help="only time the dense reference GEMMs (for a counter run of the vendor kernel)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after timing, copy this many MiB device-to-device once, so that a "
                         "counter run sees a plain copy of known size (HBM byte calibration)")
    return ap.parse_args(argv)


@contextlib.contextmanager
def no_gc():
    """Run a timed region with Python's cyclic garbage collector paused, as
    the standard library's timeit does: a full collection inside a loop of
    decode-sized steps stalls the host that feeds the GPU for milliseconds,
    and the GPU idles meanwhile."""
    was = gc.isenabled()
    gc.disable()
    try:
        yield
    finally:
        if was:
            gc.enable()


def kernel_src_hash(read=None):
    """Hash of the gate/up kernels' sources with // comments and blank lines
    removed, so that an edit of a comment keeps the counter records valid.
    `read(name)` returns a file's text (default: the working tree)."""
    read = read or (lambda f: open(os.path.join(ROOT, "paper_2606_27866_amd", "csrc", f)).read())
    h = hashlib.sha256()
    for f in ("gemm_bf16_big.hip", "gemm_decode.hip", "gemv_decode.hip", "common.h", "kernels.h", "mfma_tile.h"):
        for line in read(f).splitlines():
            code = line.split("//", 1)[0].rstrip()
            if code:
                h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def traffic_file(workload, T):
    name = workload if workload != "qwen2_57b_a14b_decode" else "%s_T%d" % (workload, T)
    return os.path.join(ROOT, "profiles", "gate_up_gemm_traffic_%s.json" % name)


def load_traffic(workload, T, table):
    """HBM bytes per gate/up-GEMM launch from committed rocprofv3 counter
    runs, or None if absent or taken on a different kernel source, token
    count or keep table."""
    path = traffic_file(workload, T)
    if not os.path.exists(path):
        return None
    d = json.load(open(path))
    if (d.get("kernel_src_sha") != kernel_src_hash() or d.get("table") != table
            or d.get("T") != T):
        return None
    return d.get("hbm_bytes_per_launch")


def step_stats(ms_list):
    """Median, p10, p90, mean of per-step durations (ms)."""
    a = np.asarray(ms_list, dtype=np.float64)
    return dict(median=float(np.median(a)), p10=float(np.percentile(a, 10)), p90=float(np.percentile(a, 90)),
                mean=float(a.mean()), n=int(a.size))


def cpu_info():
    model = platform.processor() or "unknown"
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return dict(cpu_model=model, nproc=os.cpu_count(), usable_cpus=usable)


class Workload:
    """Host inputs + device copies of one layer configuration.  `weights`
    ((w_gate, w_up, w_down), (ws_gate, ws_up, ws_down)) and `dev` (the
    device copies of another Workload of the same layer) let several token
    counts share one layer."""

    def __init__(self, cfg, table_name, copies, decode_T=None, weights=None, dev=None):
        import torch
        from paper_2606_27866_amd import flexmoe as fm
        from paper_2606_27866_amd import synth
        self.cfg, self.fm, self.synth, self.torch = cfg, fm, synth, torch
        t0 = time.time()
        self.tables = synth.config_keep_tables(cfg)
        if table_name is None:
            table_name = "own" if "own" in self.tables else "kept100"
        self.table_name = table_name
        self.decode = decode_T is not None
        self.T = decode_T if self.decode else cfg.T
        bias = synth.router_bias(cfg)
        if self.decode:
            self.batches = [synth.make_tokens(cfg, T=self.T, batch=b, bias=bias) for b in range(64)]
        else:
            self.batches = [synth.make_tokens(cfg, bias=bias)]
        if weights is None:
            weights = synth.make_layer_weights(cfg)
        self.w, self.s = weights
        log("[bench] %s: host inputs ready in %.1fs" % (cfg.name, time.time() - t0))
        self.layer = fm.Layer(cfg.d, cfg.E, cfg.I, cfg.top_k, cfg.I_shared, cfg.dtype, cfg.norm_topk,
                              max_tokens=self.T)
        if dev is None:
            dev_w = [fm.to_device(a) for a in self.w]
            dev_s = [fm.to_device(a) if a is not None else None for a in self.s]
            dev = [(dev_w, dev_s)]
            for _ in range(copies - 1):
                dev.append(([t.clone() for t in dev_w], [t.clone() if t is not None else None for t in dev_s]))
        self.copies = dev
        self.xd = [(fm.to_device(x), fm.to_device(lg)) for x, lg in self.batches]
        self.y = torch.empty((self.T, cfg.d), dtype=self.layer.tdtype, device="cuda")
        self.keep_dev = {n: fm.to_device(t) for n, t in self.tables.items()}
        torch.cuda.synchronize()
        log("[bench] %s: device buffers ready (%d weight copies) in %.1fs" % (cfg.name, len(dev), time.time() - t0))

    def use_copy(self, i):
        w, s = self.copies[i % len(self.copies)]
        self.layer.set_weights(*w, *s)

    def counts(self, batch, keep_name):
        """Per-expert routed token counts n_e from the GPU's own dispatch."""
        torch = self.torch
        c = torch.empty(self.cfg.E, dtype=torch.int32, device="cuda")
        x, lg = self.xd[batch]
        self.use_copy(0)
        self.layer.forward(x, lg, y=self.y, keep=self.keep_dev[keep_name], dbg={"counts": c})
        torch.cuda.synchronize()
        return c.cpu().numpy().astype(np.int64)

    def algorithmic(self, n, keep):
        """Flops and HBM bytes of the whole layer and of the gate/up GEMM."""
        cfg = self.cfg
        d, Is, T = cfg.d, cfg.I_shared, self.T
        sw = 2 if cfg.dtype == self.synth.BF16 else 4
        k = keep.astype(np.int64)
        act = (n > 0) & (k > 0)
        nk = int((n * k)[act].sum())
        F = 6 * d * nk + 6 * d * T * Is
        B = 3 * d * int(k[act].sum()) * sw + 3 * d * Is * sw + 2 * T * d * sw + 4 * T * cfg.E
        F1 = 4 * d * (nk + T * Is)
        B1 = 2 * d * (int(k[act].sum()) + Is) * sw + T * d * sw + (nk + T * Is) * sw
        lw_keep = float((n * k).sum()) / max(1, int(n.sum()) * cfg.I)
        return dict(F=F, B=B, F1=F1, B1=B1, load_weighted_keep=lw_keep)

    def _step(self, i, keep_names, mode):
        """One step: weight copy i, batch i; mode 'fixed' (one device table),
        'upload' (flexmoe_set_budget of the next table before the forward)
        or 'pointer' (a different resident device table each step)."""
        self.use_copy(i)
        name = keep_names[i % len(keep_names)]
        if mode == "upload":
            self.layer.set_budget(self.tables[name])
            keep = None
        else:
            keep = self.keep_dev[name]
        x, lg = self.xd[i % len(self.xd)]
        self.layer.forward(x, lg, y=self.y, keep=keep)

    def run(self, steps, keep_names, with_kernel_times=False, mode=None):
        """Time `steps` forwards; the keep table cycles over keep_names (by
        default one budget upload per step when there are several)."""
        torch, fm = self.torch, self.fm
        mode = mode or ("upload" if len(keep_names) > 1 else "fixed")
        if with_kernel_times:
            fm.flexmoe_timing_enable(True)
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        with no_gc():
            ev0.record()
            for i in range(steps):
                self._step(i, keep_names, mode)
            ev1.record()
            torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1)
        kt = None
        if with_kernel_times:
            kt = fm.flexmoe_timing_read()
            fm.flexmoe_timing_enable(False)
        return ms, kt

    def run_per_step(self, steps, keep_names, mode=None):
        """Per-step durations (ms): an event on the stream between steps."""
        torch = self.torch
        mode = mode or ("upload" if len(keep_names) > 1 else "fixed")
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        with no_gc():
            for i in range(steps):
                ev[i].record()
                self._step(i, keep_names, mode)
            ev[steps].record()
            torch.cuda.synchronize()
        return [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]

    def warm(self, args, keep_names, mode=None, min_steps=None, warm_s=None):
        """At least --warmup steps and --min-warmup-s seconds of them (or
        min_steps and warm_s)."""
        n, t0 = 0, time.time()
        want = args.warmup if min_steps is None else min_steps
        secs = args.min_warmup_s if warm_s is None else warm_s
        while n < want or time.time() - t0 < secs:
            k = max(1, min(50, want - n)) if n < want else 20
            self.run(k, keep_names, mode=mode)
            n += k
        return n

    def capture_graphs(self, keep_names, n):
        """One HIP graph per step of a period of n decode steps: the budget
        upload (when tables switch) and the layer forward of batch b with
        weight copy b % copies, captured through torch.cuda.graph."""
        torch = self.torch
        switching = len(keep_names) > 1
        self.graphs = []
        for b in range(n):
            self.use_copy(b)
            x, lg = self.xd[b % len(self.xd)]
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                if switching:
                    self.layer.set_budget(self.tables[keep_names[b % len(keep_names)]])
                self.layer.forward(x, lg, y=self.y, keep=None if switching else self.keep_dev[keep_names[0]])
            self.graphs.append(g)
        torch.cuda.synchronize()

    def run_graphs(self, steps):
        torch = self.torch
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        with no_gc():
            ev0.record()
            for i in range(steps):
                self.graphs[i % len(self.graphs)].replay()
            ev1.record()
            torch.cuda.synchronize()
        return ev0.elapsed_time(ev1)

    def run_bucketed(self, steps, table_name, k_align):
        """Time `steps` forwards of the bucketed ablation (width groups, one
        launch pair each, widths aligned up to k_align)."""
        torch = self.torch
        keep = self.tables[table_name]
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        with no_gc():
            ev0.record()
            for i in range(steps):
                self.use_copy(i)
                x, lg = self.xd[i % len(self.xd)]
                self.layer.forward(x, lg, y=self.y, bucketed=(keep, k_align))
            ev1.record()
            torch.cuda.synchronize()
        return ev0.elapsed_time(ev1)

    def export_clipped(self, table_name):
        """Offline clipping: each weight copy packed for one budget."""
        cws = []
        for c in range(len(self.copies)):
            self.use_copy(c)
            cws.append(self.layer.export_clipped(self.tables[table_name]))
        self.torch.cuda.synchronize()
        return cws

    def run_clipped(self, steps, cws):
        """Time `steps` forwards of the offline-clipped subnetwork (packed
        weights rotated like the ranked ones)."""
        torch = self.torch
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        with no_gc():
            ev0.record()
            for i in range(steps):
                self.use_copy(i)  # shared expert of this copy
                x, lg = self.xd[i % len(self.xd)]
                self.layer.forward(x, lg, y=self.y, clipped=cws[i % len(cws)])
            ev1.record()
            torch.cuda.synchronize()
        return ev0.elapsed_time(ev1)

    def release(self):
        del self.copies, self.xd, self.y, self.keep_dev, self.layer
        self.torch.cuda.synchronize()
        self.torch.cuda.empty_cache()


def gate_up_kernel_name(cfg, T):
    """The kernel the library runs for the gate/up GEMM at T tokens (its own
    thresholds, kernels.h)."""
    if cfg.dtype != 1:
        return "gemm1_f32_kernel"
    if T > DECODE_MAX_T:
        return "gemm1_big_kernel"
    routed = "gemm1_decode_wide_kernel" if T > GEMV_MAX_T else "gemv1_kernel"
    if not cfg.I_shared:
        return routed
    shared = "gemm1_decode_wide_kernel" if T > DECODE_WIDE_SHARED_T else "gemv1_kernel"
    if routed == shared:
        return routed
    return "%s for the routed experts, %s for the shared expert" % (routed, shared)


def roofline_of(wl, alg, kt, steps, bf16, workload, keep_label):
    """Roofline of the gate/up GEMM from the event-timed launches: the
    algorithmic flops (prefill) or bytes (decode) of one launch over its
    average duration.  With the shared expert on the side stream there are
    two concurrent launches per step; then each duration includes the time
    the two share the chip, and the layer-level fraction is the defensible
    figure (`layer_frac`)."""
    gu_ms = kt["gate_up"][0] + kt["gate_up_shared"][0]
    gu_n = kt["gate_up"][1] + kt["gate_up_shared"][1]
    gu_avg = gu_ms / max(gu_n, 1)
    per_step = gu_n / steps
    gu_step = gu_avg * per_step
    peak_flops = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
    mfma = alg["F1"] / alg["B1"] >= RIDGE and not wl.decode
    if mfma:
        roof = dict(bound="mfma", achieved=alg["F1"] / per_step / (gu_avg / 1e3) / 1e12, peak=peak_flops,
                    unit="TFLOP/s", flops_per_launch=alg["F1"] / per_step)
    else:
        roof = dict(bound="hbm", achieved=alg["B1"] / per_step / (gu_avg / 1e3) / 1e9, peak=PEAK_HBM_GBS,
                    unit="GB/s", bytes_per_launch=alg["B1"] / per_step)
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = load_traffic(workload, wl.T, keep_label)
    roof["kernel"] = "gate_up GEMM (%s)" % gate_up_kernel_name(wl.cfg, wl.T)
    roof["avg_launch_ms"] = gu_avg
    roof["launches_per_step"] = per_step
    roof["summed_launch_ms_per_step"] = gu_step
    roof["timing"] = "HIP events around each launch, on its stream, over a separate pass of the K steps"
    roof["concurrent_launches"] = bool(kt["gate_up_shared"][1])
    if kt["gate_up_shared"][1]:
        roof["note"] = ("the shared expert's gate/up launch runs on a side stream concurrently with the "
                        "routed one; each launch's duration includes the time the two share the chip, so "
                        "this per-launch figure is a lower bound; layer_frac is the layer-level fraction")
    return roof


def forward_section(wl, args, keep_names, mode=None, workload=None, steps=None, label=None, warm_s=None):
    """Warm-up, K timed steps, per-step percentiles, per-kernel times, the
    gate/up roofline and the layer's rates for one workload and table list."""
    steps = steps or args.steps
    bf16 = wl.cfg.dtype == wl.synth.BF16
    workload = workload or wl.cfg.name
    if wl.decode:
        per = []
        for b in range(min(64, steps + args.warmup)):
            name = keep_names[b % len(keep_names)]
            per.append(wl.algorithmic(wl.counts(b, name), wl.tables[name]))
        alg = {k: float(np.mean([p[k] for p in per])) for k in per[0]}
    else:
        alg = wl.algorithmic(wl.counts(0, keep_names[0]), wl.tables[keep_names[0]])
    nwarm = wl.warm(args, keep_names, mode=mode, warm_s=warm_s)
    # the timed region: exactly K steps, no instrumentation inside
    ms, _ = wl.run(steps, keep_names, mode=mode)
    per_step = wl.run_per_step(steps, keep_names, mode=mode)
    # per-kernel durations: the same K steps again, each kernel bracketed by
    # a HIP event pair on the stream it runs on (a few microseconds per kernel)
    ms_inst, kt = wl.run(steps, keep_names, with_kernel_times=True, mode=mode)
    ms_step = ms / steps
    peak_flops = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
    layer_s = ms_step / 1e3
    layer = dict(tflops=alg["F"] / layer_s / 1e12, frac_mfma=alg["F"] / layer_s / 1e12 / peak_flops,
                 gbs=alg["B"] / layer_s / 1e9, frac_hbm=alg["B"] / layer_s / 1e9 / PEAK_HBM_GBS,
                 flops_per_step=alg["F"], bytes_per_step=alg["B"],
                 load_weighted_keep=alg["load_weighted_keep"],
                 kernels_ms={k: v[0] / max(v[1], 1) for k, v in kt.items() if v[1]})
    roof = roofline_of(wl, alg, kt, steps, bf16, workload, label or "+".join(keep_names))
    roof["layer_frac"] = layer["frac_hbm"] if roof["bound"] == "hbm" else layer["frac_mfma"]
    out = dict(T=wl.T, steps=steps, warmup_steps=nwarm, ms_per_step=ms_step, tokens_per_s=wl.T / layer_s,
               step_ms=step_stats(per_step), ms_per_step_instrumented=ms_inst / steps,
               roofline=roof, layer=layer)
    log("[bench] %s T=%d %s: %.4f ms/step (median %.4f, p10 %.4f, p90 %.4f), %.0f tokens/s, layer %.1f TFLOP/s "
        "(%.3f of bf16 peak) %.0f GB/s (%.3f of HBM); gate/up %.4f ms/launch (%s %.3f)"
        % (workload, wl.T, "+".join(keep_names), ms_step, out["step_ms"]["median"], out["step_ms"]["p10"],
           out["step_ms"]["p90"], wl.T / layer_s, layer["tflops"], layer["frac_mfma"], layer["gbs"],
           layer["frac_hbm"], roof["avg_launch_ms"], roof["bound"], roof["frac"]))
    for kname, v in layer["kernels_ms"].items():
        log("[bench]   %-17s %8.4f ms avg" % (kname, v))
    return out


def per_budget_section(wl, args):
    """The nested tables on the headline layer: online (ranked weights and a
    device keep table), offline (compact weights of that budget) and the
    bucketed ablation."""
    cfg, synth, fm = wl.cfg, wl.synth, wl.fm
    peak_flops = PEAK_BF16_TFLOPS if cfg.dtype == synth.BF16 else PEAK_F32_TFLOPS
    steps_b = max(5, args.steps // 2)
    per_budget = []
    for name in ["kept%d" % int(round(f * 100)) for f in synth.NESTED_FRACTIONS]:
        a = wl.algorithmic(wl.counts(0, name), wl.tables[name])
        wl.run(3, [name])
        sb = wl.run(steps_b, [name])[0] / steps_b / 1e3
        med = step_stats(wl.run_per_step(steps_b, [name]))["median"]
        cws = wl.export_clipped(name)
        wl.run_clipped(2, cws)
        so = wl.run_clipped(steps_b, cws) / steps_b / 1e3
        del cws
        wl.run_bucketed(2, name, args.bucket_align)
        sk = wl.run_bucketed(steps_b, name, args.bucket_align) / steps_b / 1e3
        per_budget.append(dict(table=name, kept=synth.keep_fraction(wl.tables[name], cfg.I),
                               load_weighted_keep=a["load_weighted_keep"],
                               ms=sb * 1e3, median_ms=med, tokens_per_s=wl.T / sb,
                               tflops=a["F"] / sb / 1e12, frac_mfma=a["F"] / sb / 1e12 / peak_flops,
                               frac_hbm=a["B"] / sb / 1e9 / PEAK_HBM_GBS,
                               offline_ms=so * 1e3, offline_tokens_per_s=wl.T / so, online_over_offline=so / sb,
                               bucketed_ms=sk * 1e3, bucketed_k_align=args.bucket_align,
                               ragged_over_bucketed=sk / sb))
        log("[bench]   budget %-7s %.4f ms  %.0f tok/s  %.1f TFLOP/s | offline %.4f ms, online/offline %.3f"
            " | bucketed(%d) %.4f ms, ragged/bucketed %.3f" %
            (name, sb * 1e3, wl.T / sb, a["F"] / sb / 1e12, so * 1e3, so / sb, args.bucket_align, sk * 1e3, sk / sb))
    # the bucketed ablation on keep tables drawn from the paper's action set
    # {0.1, 0.4, 0.7, 1.0} (at most four width groups, as in its deployments)
    ablation = []
    levels = [fm.flexmoe_keep_from_ratio(r, cfg.I) for r in synth.ACTION_RATIOS]
    for f in (0.75, 0.5, 0.25):
        name = "action%d" % int(round(f * 100))
        wl.tables[name] = synth.action_keep_table(cfg.E, levels, 1000 * cfg.config_id + synth._TID_ACTION, f)
        wl.keep_dev[name] = fm.to_device(wl.tables[name])
        wl.run(2, [name])
        sb = wl.run(steps_b, [name])[0] / steps_b / 1e3
        wl.run_bucketed(2, name, args.bucket_align)
        sk = wl.run_bucketed(steps_b, name, args.bucket_align) / steps_b / 1e3
        widths = sorted(set(int(v) for v in wl.tables[name] if v > 0))
        ablation.append(dict(table=name, kept=synth.keep_fraction(wl.tables[name], cfg.I), widths=widths,
                             ragged_ms=sb * 1e3, bucketed_ms=sk * 1e3, bucketed_k_align=args.bucket_align,
                             ragged_over_bucketed=sk / sb))
        log("[bench]   action-set table %-9s kept %.3f widths %s: ragged %.4f ms, bucketed(%d) %.4f ms, "
            "ragged/bucketed %.3f" % (name, synth.keep_fraction(wl.tables[name], cfg.I), widths, sb * 1e3,
                                      args.bucket_align, sk * 1e3, sk / sb))
    return per_budget, ablation


def cpu_baselines(wl, keep, args):
    """The oracle on a bounded sample of the workload's tokens: the fp64
    parity build with all OpenMP threads (the reported baseline), and the same
    source at 1 thread and with fp32 accumulators at -O3 -march=native (1
    thread and all threads)."""
    import oracle
    cfg = wl.cfg
    x, lg = wl.batches[0]
    T = x.shape[0]
    allt = oracle.num_threads()

    def measure(variant, threads, target_s):
        oracle.set_threads(threads, variant)
        used = oracle.num_threads(variant)

        def run(S):
            t0 = time.time()
            oracle.layer_forward(x[:S], lg[:S], *wl.w, keep, cfg.top_k, cfg.norm_topk, *wl.s, variant=variant)
            return time.time() - t0

        S0 = min(16 if threads == 1 else 64, T)
        t0 = run(S0)
        S = int(min(T, max(S0, S0 * target_s / max(t0, 1e-3))))
        t = run(S) if S != S0 else t0
        passes = 1
        while S == T and t < 0.6 * target_s and passes < 4:
            t += run(S)
            passes += 1
        what = ("%d pass%s over all %d tokens" % (passes, "es" if passes > 1 else "", T) if S == T
                else "first %d of %d tokens" % (S, T))
        return dict(value=S * passes / t, unit="tokens/s", cores=used, kind="oracle",
                    build=("fp64 accumulation, gcc -O2 -fopenmp (the parity build)" if variant == "fp64" else
                           "fp32 accumulation, gcc -O3 -march=native -fopenmp (timing build of the same source)"),
                    sample="%s of the workload, same weights and keep table, %.1f s" % (what, t))

    main = measure("fp64", allt, args.cpu_seconds)
    builds = [dict(main), measure("fp64", 1, args.cpu_seconds / 3), measure("f32acc", allt, args.cpu_seconds / 3),
              measure("f32acc", 1, args.cpu_seconds / 3)]
    oracle.set_threads(allt)
    oracle.set_threads(allt, "f32acc")
    main.update(cpu_info())
    main["builds"] = builds
    for b in builds:
        log("[bench] CPU oracle %-70s %2d threads: %.2f tokens/s" % (b["build"], b["cores"], b["value"]))
    return main


def saliency_section(wl, args, T=None, with_cpu=True):
    """Channel ranking on the device (Eq. 2 saliency over calibration batches,
    then the reorder of Eq. 3), timed per calibration batch."""
    torch, fm, synth, cfg = wl.torch, wl.fm, wl.synth, wl.cfg
    T = T or args.saliency_T or wl.T
    bias = synth.router_bias(cfg)
    nb = 4
    batches = []
    for b in range(nb):
        x, lg = synth.make_calibration_batch(cfg, b, T, bias=bias)
        batches.append((fm.to_device(x), fm.to_device(lg), fm.to_device(synth.make_target(cfg, T, batch=b))))
    wl.use_copy(0)
    sal = fm.Saliency(wl.layer, T)
    steps = args.saliency_steps

    def run(k, timed_kernels=False):
        if timed_kernels:
            fm.flexmoe_timing_enable(True)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(k):
            x, lg, tg = batches[i % nb]
            sal.add_batch(x, lg, tg, scale=1.0 / k)
        e1.record()
        torch.cuda.synchronize()
        kt = None
        if timed_kernels:
            kt = fm.flexmoe_timing_read()
            fm.flexmoe_timing_enable(False)
        return e0.elapsed_time(e1), kt

    run(2)
    sal.scores.zero_()
    ms, _ = run(steps)
    _, kt = run(steps, timed_kernels=True)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    ranked = sal.rank_reorder()
    e1.record()
    torch.cuda.synchronize()
    rank_ms = e0.elapsed_time(e1)
    del ranked
    ms_b = ms / steps
    A = T * cfg.top_k
    d, I, Is = cfg.d, cfg.I, cfg.I_shared
    f_fwd = 6 * d * A * I + 6 * d * T * Is
    f_dgrad = 2 * d * A * I
    f_wgrad = 6 * d * A * I           # three weight gradients, every routed expert at full width
    f_all = f_fwd + f_dgrad + f_wgrad
    wg_ms, wg_n = kt["sal_wgrad"]
    dg_ms, dg_n = kt["sal_dgrad"]
    kms = {k: v[0] / max(v[1], 1) for k, v in kt.items() if v[1]}
    wg_avg = wg_ms / max(wg_n, 1)
    roof = dict(kernel="wgrad GEMMs + Eq. 2 reduction (sal_wgrad_kernel)", bound="mfma",
                achieved=f_wgrad / (wg_avg / 1e3) / 1e12, peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                avg_launch_ms=wg_avg, flops_per_launch=f_wgrad,
                theta_bytes_per_launch=3 * cfg.E * I * d * 2)
    roof["frac"] = roof["achieved"] / roof["peak"]
    dg_avg = dg_ms / max(dg_n, 1)
    out = dict(calibration_tokens=T, batches_timed=steps, ms_per_batch=ms_b, tokens_per_s=T / (ms_b / 1e3),
               tflops=f_all / (ms_b / 1e3) / 1e12, frac_mfma=f_all / (ms_b / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
               flops_per_batch=f_all, rank_reorder_ms=rank_ms, roofline_wgrad=roof,
               dgrad_tflops=f_dgrad / (dg_avg / 1e3) / 1e12, kernels_ms=kms,
               loss="1/2 sum_t ||Y_t - target_t||^2 with a seeded Gaussian target (std 0.05)",
               w_down_t="made once for the ranking set (flexmoe_transpose_weights), not per batch")
    log("[bench] saliency: %d tokens/batch, %.4f ms/batch, %.0f tokens/s, %.1f TFLOP/s overall; wgrad %.4f ms "
        "(%.1f TFLOP/s), dgrad %.4f ms (%.1f TFLOP/s); rank+reorder %.3f ms"
        % (T, ms_b, T / (ms_b / 1e3), out["tflops"], wg_avg, roof["achieved"], dg_avg, out["dgrad_tflops"],
           rank_ms))
    for k, v in kms.items():
        log("[bench]   saliency %-17s %8.4f ms" % (k, v))
    del sal, batches
    torch.cuda.empty_cache()
    if with_cpu and not args.no_cpu:
        out["cpu_baseline"] = saliency_cpu_baseline(wl, T, args.cpu_seconds)
        log("[bench] saliency CPU oracle: %.2f tokens/s on %d threads" % (out["cpu_baseline"]["value"],
                                                                           out["cpu_baseline"]["cores"]))
    return out


def action_section(wl, args):
    """One action-learning step of the layer on the device (Sec. 3.2): the
    Gumbel-max sample of every expert's width (Eq. 5), the sampled subnet's
    forward, its backward for a fixed synthetic upstream gradient, and the
    action-logit gradient (Eqs. 6-8).  Fresh Gumbel draws every step, so the
    widths change from step to step."""
    torch, fm, synth, cfg = wl.torch, wl.fm, wl.synth, wl.cfg
    T = wl.T
    ratios = synth.ACTION_RATIOS
    K = len(ratios)
    nsteps = 8
    alpha, _ = synth.make_action_inputs(cfg, K)
    gumbels = [fm.to_device(synth.make_action_inputs(cfg, K, step=i)[1]) for i in range(nsteps)]
    ad = fm.to_device(alpha)
    x, lg = wl.xd[0]
    dy = fm.to_device(synth.make_target(cfg, T, std=1e-3))   # a fixed upstream gradient dL/dY
    wl.use_copy(0)
    lr = fm.ActionLearner(wl.layer, T, ratios)
    lr.transpose_weights()
    y = torch.empty((T, cfg.d), dtype=wl.layer.tdtype, device="cuda")
    tau, lam, beta = 1.0, 0.1, 0.01

    def step(i):
        lr.sample(ad, gumbels[i % nsteps])
        lr.forward(x, lg, y=y)
        _, _, dm = lr.backward(lg, dy)
        lr.action_grad(ad, gumbels[i % nsteps], tau, lam, beta, dm)

    def run(k, timed_kernels=False):
        if timed_kernels:
            fm.flexmoe_timing_enable(True)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(k):
            step(i)
        e1.record()
        torch.cuda.synchronize()
        kt = None
        if timed_kernels:
            kt = fm.flexmoe_timing_read()
            fm.flexmoe_timing_enable(False)
        return e0.elapsed_time(e1), kt

    run(2)
    steps = args.action_steps
    ms, _ = run(steps)
    _, kt = run(steps, timed_kernels=True)
    # algorithmic work of the average step: the sampled widths of each step
    # and the routed counts (fixed: the batch does not change)
    n = wl.counts(0, "kept100")
    A_I = 0
    nk = 0
    for i in range(steps):
        keep, _, _ = _sample_host(synth, cfg, ratios, alpha, i % nsteps)
        nk += int((n * keep).sum())
        A_I += int(n.sum()) * cfg.I
    nk /= steps
    A_I /= steps
    d, Is = cfg.d, cfg.I_shared
    f_fwd = 4 * d * A_I + 2 * d * nk + 6 * d * T * Is        # gate/up at full width, down at the kept width
    f_dgrad = 2 * d * A_I + 2 * d * T * Is
    f_dx = 4 * d * nk + 4 * d * T * Is
    f_all = f_fwd + f_dgrad + f_dx
    ms_s = ms / steps
    kms = {k: v[0] / max(v[1], 1) for k, v in kt.items() if v[1]}
    dg_ms = kms.get("act_dgrad", float("nan"))
    dx_ms = kms.get("act_dx", float("nan"))
    gu_ms = kms.get("gate_up", float("nan"))
    out = dict(tokens=T, steps_timed=steps, ms_per_step=ms_s, tokens_per_s=T / (ms_s / 1e3),
               tflops=f_all / (ms_s / 1e3) / 1e12, frac_mfma=f_all / (ms_s / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
               flops_per_step=f_all, mean_kept_fraction=nk / A_I, ratios=list(ratios),
               roofline_dgrad=dict(kernel="dgrad + SwiGLU backward + mask gradient (dgrad_kernel<2>)",
                                   bound="mfma", achieved=f_dgrad / (dg_ms / 1e3) / 1e12, peak=PEAK_BF16_TFLOPS,
                                   unit="TFLOP/s", frac=f_dgrad / (dg_ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS,
                                   avg_launch_ms=dg_ms, flops_per_launch=f_dgrad),
               dx_tflops=f_dx / (dx_ms / 1e3) / 1e12, gate_up_tflops=4 * d * (A_I + T * Is) / (gu_ms / 1e3) / 1e12,
               kernels_ms=kms,
               upstream_gradient="fixed seeded Gaussian dL/dY (std 1e-3); Gumbel draws change every step")
    log("[bench] action step: %.4f ms/step, %.0f tokens/s, %.1f TFLOP/s; dgrad %.4f ms (%.1f TFLOP/s), dx %.4f ms "
        "(%.1f TFLOP/s), gate/up %.4f ms; mean kept fraction %.3f"
        % (ms_s, T / (ms_s / 1e3), out["tflops"], dg_ms, out["roofline_dgrad"]["achieved"], dx_ms,
           out["dx_tflops"], gu_ms, nk / A_I))
    for k, v in kms.items():
        log("[bench]   action %-17s %8.4f ms" % (k, v))
    return out


def _sample_host(synth, cfg, ratios, alpha, step):
    """The widths the device samples at `step` (same fp32 argmax), for the
    algorithmic flop count."""
    _, gumbel = synth.make_action_inputs(cfg, len(ratios), step=step)
    widths = np.array([int(np.ceil(r * cfg.I - 1e-9)) for r in ratios], np.int64)
    act = np.argmax(alpha + gumbel, axis=1)
    return widths[act], act, None


def saliency_cpu_baseline(wl, T, target_s):
    """The oracle's Eq. 2 on the first S tokens of calibration batch 0."""
    import oracle
    cfg, synth = wl.cfg, wl.synth
    x, lg = synth.make_calibration_batch(cfg, 0, T)
    tg = synth.make_target(cfg, T, batch=0)

    def run(S):
        t0 = time.time()
        oracle.channel_saliency([(x[:S], lg[:S], tg[:S])], *wl.w, cfg.top_k, cfg.norm_topk, *wl.s)
        return time.time() - t0

    # a per-batch fixed part (the Eq. 2 sums over every weight) plus a
    # per-token part: two probe sizes size the timed sample
    Sa, Sb = min(64, T), min(256, T)
    ta = run(Sa)
    tb = run(Sb) if Sb != Sa else ta
    c = max((tb - ta) / max(Sb - Sa, 1), 1e-6)
    f = max(ta - c * Sa, 0.0)
    S = int(min(T, max(Sb, (target_s - f) / c)))
    t = run(S) if S != Sb else tb
    return dict(value=S / t, unit="tokens/s", cores=oracle.num_threads(), kind="oracle",
                sample="first %d of %d tokens of calibration batch 0, %.1f s (fp64); the whole batch would take "
                       "about %.0f s (%.1f s per batch + %.2f ms per token)" % (S, T, t, f + c * T, f, c * 1e3))


DENSE_SHAPES = ((8192, 8192, 8192), (16384, 28672, 4096))


def dense_reference(reps=25):
    """The vendor library's dense bf16 GEMM (torch.matmul -> hipBLASLt) on two
    dense shapes, the second one the Mixtral-shaped gate/up with every token
    on one expert: the rate a plain contraction reaches on this GPU, as
    context for the layer's roofline.  Not part of the layer's path."""
    import torch
    out = []
    for M, N, K in DENSE_SHAPES:
        g = torch.Generator(device="cuda")
        g.manual_seed(M + N + K)
        a = torch.randn(M, K, device="cuda", dtype=torch.bfloat16, generator=g)
        b = torch.randn(N, K, device="cuda", dtype=torch.bfloat16, generator=g)
        c = a @ b.t()
        torch.cuda.synchronize()
        t0 = time.time()
        while time.time() - t0 < 1.0:
            c = a @ b.t()
            torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            c = a @ b.t()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        tf = 2.0 * M * N * K / (ms / 1e3) / 1e12
        out.append(dict(M=M, N=N, K=K, ms=ms, tflops=tf, frac=tf / PEAK_BF16_TFLOPS))
        log("[bench] dense reference (torch.matmul bf16) %dx%dx%d: %.4f ms, %.1f TFLOP/s (%.3f of bf16 peak)"
            % (M, N, K, ms, tf, tf / PEAK_BF16_TFLOPS))
        del a, b, c
    torch.cuda.empty_cache()
    return out


def qwen2_prefill_section(args):
    """The Qwen2-57B-A14B-shaped layer (T = 8192, 64 experts of 2560
    channels, top-8, shared expert of 20480) at the five nested budgets.
    Its shared expert fills more than four waves of gate/up tiles, so it runs
    as segment 0 of the same launch: one gate/up launch per step."""
    from paper_2606_27866_amd import synth
    cfg = synth.CONFIGS["qwen2_57b_a14b_prefill"]
    wl = Workload(cfg, "kept100", args.copies)
    steps = args.extra_steps or max(args.steps, 20)
    out = []
    for i, name in enumerate("kept%d" % int(round(f * 100)) for f in synth.NESTED_FRACTIONS):
        r = forward_section(wl, args, [name], steps=steps, warm_s=args.min_warmup_s if i == 0 else 0.5)
        r["table"] = name
        r["kept"] = synth.keep_fraction(wl.tables[name], cfg.I)
        out.append(r)
    wl.release()
    return dict(workload=cfg.name, d=cfg.d, E=cfg.E, I=cfg.I, top_k=cfg.top_k, I_shared=cfg.I_shared,
                per_budget=out)


def decode_section(args):
    """The Qwen2-57B-A14B-shaped layer at 1, 8 and 64 tokens per step, weight
    streaming.  For each T: the budget cycling through the five nested tables
    with one flexmoe_set_budget upload per step (the measured configuration);
    the same cycle as a pointer switch between five resident device tables;
    each table held fixed; and the cost of one switch."""
    import torch
    from paper_2606_27866_amd import synth
    cfg = synth.CONFIGS["qwen2_57b_a14b_decode"]
    names = ["kept%d" % int(round(f * 100)) for f in synth.NESTED_FRACTIONS]
    t0 = time.time()
    weights = synth.make_layer_weights(cfg)
    log("[bench] decode layer weights drawn in %.1fs" % (time.time() - t0))
    steps = max(args.steps, 200)
    out = dict(workload=cfg.name, d=cfg.d, E=cfg.E, I=cfg.I, top_k=cfg.top_k, I_shared=cfg.I_shared,
               tables=names, steps=steps, by_T={})
    dev = None
    for T in (1, 8, 64):
        wl = Workload(cfg, None, args.copies, decode_T=T, weights=weights, dev=dev)
        dev = wl.copies
        sw = forward_section(wl, args, names, mode="upload", workload=cfg.name, steps=steps,
                             warm_s=args.min_warmup_s if T == 1 else 1.0)
        wl.warm(args, names, mode="pointer", min_steps=20, warm_s=0.3)
        ptr = step_stats(wl.run_per_step(steps, names, mode="pointer"))
        fixed = {}
        for n in names:
            wl.run(10, [n])
            fixed[n] = step_stats(wl.run_per_step(steps, [n]))
        fixed_med = float(np.mean([v["median"] for v in fixed.values()]))
        # host latency of one flexmoe_set_budget call through the binding
        torch.cuda.synchronize()
        nh = 500
        with no_gc():
            h0 = time.perf_counter()
            for i in range(nh):
                wl.layer.set_budget(wl.tables[names[i % len(names)]])
            host_us = (time.perf_counter() - h0) / nh * 1e6
            torch.cuda.synchronize()
        # GPU time of the upload kernel: a burst of launches on an idle stream
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with no_gc():
            e0.record()
            for i in range(nh):
                wl.layer.set_budget(wl.tables[names[i % len(names)]])
            e1.record()
            torch.cuda.synchronize()
        gpu_us = e0.elapsed_time(e1) / nh * 1e3
        cost = dict(set_budget_host_us=host_us, set_keep_kernel_gpu_us_burst=gpu_us,
                    cycling_minus_fixed_us=(sw["step_ms"]["median"] - fixed_med) * 1e3,
                    cycling_minus_pointer_us=(sw["step_ms"]["median"] - ptr["median"]) * 1e3,
                    pointer_minus_fixed_us=(ptr["median"] - fixed_med) * 1e3,
                    note="medians of per-step durations; fixed = mean over the five tables of each held "
                         "fixed; the upload carries the table in the kernel's arguments (no host-to-device "
                         "copy); the burst figure is launches back to back on an idle stream")
        log("[bench] decode T=%d: cycling %.4f ms, pointer %.4f ms, fixed(mean) %.4f ms; set_budget host %.2f us, "
            "GPU %.2f us; cycling-fixed %.2f us" % (T, sw["step_ms"]["median"], ptr["median"], fixed_med, host_us,
                                                    gpu_us, cost["cycling_minus_fixed_us"]))
        out["by_T"]["T%d" % T] = dict(switching=sw, pointer_switch=ptr, fixed=fixed, fixed_median_mean=fixed_med,
                                      switch_cost=cost)
        wl.release()
    del dev
    torch.cuda.empty_cache()
    return out


def qwen15_section(args):
    """The Qwen1.5-MoE-A2.7B-shaped layer (T = 4096, 60 experts of 1408
    channels, top-4, shared expert of 5632 on the side stream) at its own
    50 % table, with the device channel saliency (Eq. 2) and one
    action-learning step of the same layer."""
    from paper_2606_27866_amd import synth
    cfg = synth.CONFIGS["qwen15_moe_a27b"]
    wl = Workload(cfg, None, args.copies)
    r = forward_section(wl, args, [wl.table_name], steps=args.extra_steps or max(args.steps, 20))
    r.update(workload=cfg.name, d=cfg.d, E=cfg.E, I=cfg.I, top_k=cfg.top_k, I_shared=cfg.I_shared,
             keep_table=wl.table_name)
    if not args.no_saliency:
        r["saliency"] = saliency_section(wl, args)
        if not args.saliency_T:
            r["saliency"]["batch_x4"] = saliency_section(wl, args, T=4 * wl.T, with_cpu=False)
    if not args.no_action:
        r["action_learning"] = action_section(wl, args)
    wl.release()
    return r


def main(argv=None):
    args = parse(argv)
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(the layer shards by tokens or experts; see the design notes). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_27866_amd import flexmoe as fm
    from paper_2606_27866_amd import synth
    torch.cuda.set_device(0)
    fm.lib()
    if args.dense_reference_only:
        print(json.dumps({"dense_reference": dense_reference()}), flush=True)
        return
    t_start = time.time()
    cfg = synth.CONFIGS[args.workload]
    decode_T = args.decode_T if args.workload == "qwen2_57b_a14b_decode" else None
    wl = Workload(cfg, args.table, args.copies, decode_T)
    bf16 = cfg.dtype == synth.BF16
    if wl.decode:
        keep_names = ["kept%d" % int(round(f * 100)) for f in synth.NESTED_FRACTIONS]
    else:
        keep_names = [wl.table_name]
    head = forward_section(wl, args, keep_names, workload=args.workload)
    ms_step = head["ms_per_step"]
    value = head["tokens_per_s"]
    eager_ms_step = ms_step
    graphs = False
    if wl.decode and args.graphs:
        wl.capture_graphs(keep_names, 64)
        wl.run_graphs(args.warmup)
        ms_g = wl.run_graphs(args.steps)
        graphs = True
        ms_step = ms_g / args.steps
        value = wl.T * args.steps / (ms_g / 1e3)
        log("[bench] %s: %.4f ms/step replayed from HIP graphs (eager %.4f ms/step)"
            % (args.workload, ms_step, eager_ms_step))

    per_budget = ablation = None
    if not args.no_per_budget and not wl.decode:
        per_budget, ablation = per_budget_section(wl, args)
    saliency = action = None
    if args.workload != HEADLINE and bf16 and not wl.decode:
        if not args.no_saliency:
            saliency = saliency_section(wl, args)
        if not args.no_action:
            action = action_section(wl, args)

    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    cpu = None
    if not args.no_cpu:
        log("[bench] CPU oracle baselines ...")
        cpu = cpu_baselines(wl, wl.tables[keep_names[0]], args)
    wl.release()

    extras = {}
    wanted = args.extras.split(",") if args.extras and args.extras != "none" else []
    if args.workload != HEADLINE and args.extras == ",".join(EXTRAS):
        wanted = []   # a single-workload run unless extras are named
    for name in wanted:
        if name not in EXTRAS:
            raise SystemExit("unknown extra section %r" % name)
        t0 = time.time()
        extras[name] = {"qwen2_prefill": qwen2_prefill_section, "decode": decode_section,
                        "qwen15": qwen15_section}[name](args)
        log("[bench] section %s done in %.1fs" % (name, time.time() - t0))

    dense = None
    if not args.no_dense_reference and args.workload == HEADLINE:
        dense = dense_reference()

    out = {
        "metric": "masked MoE-layer tokens/s + % bf16 MFMA peak / % HBM BW, per budget",
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded PCG64; random-init weights of the layer's shape)",
        "config": {"workload": args.workload, "T": wl.T, "d": cfg.d, "E": cfg.E, "I": cfg.I,
                   "top_k": cfg.top_k, "I_shared": cfg.I_shared,
                   "keep_table": "+".join(keep_names) if wl.decode else wl.table_name,
                   "weight_copies": args.copies, "hip_graphs": graphs},
        "step_ms": head["step_ms"],
        "warmup_steps_run": head["warmup_steps"],
        "eager_ms_per_step": eager_ms_step,
        "roofline": head["roofline"],
        "layer": head["layer"],
        "per_budget": per_budget,
        "action_set_ablation": ablation,
        "cpu_baseline": cpu,
    }
    if saliency is not None:
        out["saliency"] = saliency
    if action is not None:
        out["action_learning"] = action
    out.update(extras)
    if dense is not None:
        out["dense_gemm_reference"] = dense
    out["wall_s"] = time.time() - t_start
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
