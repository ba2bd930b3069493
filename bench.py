#!/usr/bin/env python3
"""Benchmark of the masked MoE-layer forward (FlexMoE online clipping) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--table NAME]

A step is one flexmoe_layer_forward: routing, dispatch, the gate/up GEMM with
fused SwiGLU (routed experts truncated to k_e channels, plus the shared
expert), the down GEMM and the weighted combine.  Inputs are seeded synthetic
tensors already resident in HBM; the weights are rotated over --copies
device copies so that no step finds them in the 256 MB last-level cache.

Prints ONE JSON line on stdout.  `value` is tokens/s of the whole layer;
`roofline` describes the dominant kernel (the gate/up GEMM) with its
algorithmic flops or bytes per launch over its average launch time, measured
with HIP events around each launch in a second pass of the same K steps (the
first, uninstrumented pass gives the step time); `cpu_baseline` is
the CPU oracle timed on a bounded sample of the same workload.  Per-budget
results (the nested 100/80/60/40/20 % tables) go into `per_budget`, each with
the same budget run offline (exported as compact weights: the paper's static
checkpoint mode) and the online/offline throughput ratio, and with the
paper's bucketed kernel design (width groups, aligned widths) as an ablation.
`saliency` times the one-time channel ranking on the device: the Eq. 2
saliency of every routed channel over calibration batches of the workload's
size (a layer-level squared-error loss against a seeded target), with the
roofline of its dominant kernel (the weight-gradient GEMMs with the fused
saliency reduction), the reorder of Eq. 3, and the oracle on a sample.
`action_learning` times one action-learning step of the layer on the device:
the Gumbel-max width sample of every expert, the sampled subnet's forward,
its backward for a fixed upstream gradient, and the action-logit gradient.
"""
import argparse
import hashlib
import json
import os
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
DECODE_WIDE_T = 16           # above this many tokens the routed experts' take 64-wide tiles once T*k >= 8*E
DECODE_WIDE_SHARED_T = 5     # above this many tokens the shared expert's take them


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=100,
                    help="untimed steps first (the clocks and caches settle over ~100 steps)")
    ap.add_argument("--workload", default="qwen15_moe_a27b")
    ap.add_argument("--table", default=None, help="keep table (default: the workload's own, else kept100)")
    ap.add_argument("--decode-T", type=int, default=1, help="tokens per step of the decode workload")
    ap.add_argument("--copies", type=int, default=3, help="weight copies rotated over the steps")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-per-budget", action="store_true")
    ap.add_argument("--no-saliency", action="store_true", help="skip the channel-saliency measurement")
    ap.add_argument("--saliency-T", type=int, default=0,
                    help="tokens per calibration batch of the saliency (default: the workload's T)")
    ap.add_argument("--saliency-steps", type=int, default=10)
    ap.add_argument("--no-action", action="store_true", help="skip the action-learning step measurement")
    ap.add_argument("--graphs", action="store_true",
                    help="decode: replay each step from a HIP graph (captured through torch.cuda.graph); "
                         "measured no faster than eager calls, whose launches already overlap")
    ap.add_argument("--action-steps", type=int, default=10)
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU-baseline work")
    ap.add_argument("--bucket-align", type=int, default=128,
                    help="k_align of the bucketed ablation in the per-budget results")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after timing, copy this many MiB device-to-device once, so that a "
                         "counter run sees a plain copy of known size (HBM byte calibration)")
    return ap.parse_args()


def kernel_src_hash():
    h = hashlib.sha256()
    for f in ("gemm_bf16_big.hip", "gemm_decode.hip", "common.h", "kernels.h", "mfma_tile.h"):
        h.update(open(os.path.join(ROOT, "paper_2606_27866_amd", "csrc", f), "rb").read())
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


class Workload:
    """Host inputs + device copies of one layer configuration."""

    def __init__(self, cfg, table_name, copies, decode_T=None):
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
        self.w = synth.make_expert_weights(cfg)
        self.s = synth.make_shared_weights(cfg)
        log("[bench] host inputs ready in %.1fs" % (time.time() - t0))
        self.layer = fm.Layer(cfg.d, cfg.E, cfg.I, cfg.top_k, cfg.I_shared, cfg.dtype, cfg.norm_topk,
                              max_tokens=self.T)
        dev_w = [fm.to_device(a) for a in self.w]
        dev_s = [fm.to_device(a) if a is not None else None for a in self.s]
        self.copies = [(dev_w, dev_s)]
        for _ in range(copies - 1):
            self.copies.append(([t.clone() for t in dev_w], [t.clone() if t is not None else None for t in dev_s]))
        self.xd = [(fm.to_device(x), fm.to_device(lg)) for x, lg in self.batches]
        self.y = torch.empty((self.T, cfg.d), dtype=self.layer.tdtype, device="cuda")
        self.keep_dev = {n: fm.to_device(t) for n, t in self.tables.items()}
        torch.cuda.synchronize()
        log("[bench] device buffers ready (%d weight copies) in %.1fs" % (copies, time.time() - t0))

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

    def run(self, steps, keep_names, with_kernel_times=False):
        """Time `steps` forwards; the keep table cycles over keep_names (one
        budget switch per step when there are several)."""
        torch, fm = self.torch, self.fm
        switching = len(keep_names) > 1
        if with_kernel_times:
            fm.flexmoe_timing_enable(True)
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record()
        for i in range(steps):
            self.use_copy(i)
            if switching:
                self.layer.set_budget(self.tables[keep_names[i % len(keep_names)]])
                keep = None
            else:
                keep = self.keep_dev[keep_names[0]]
            x, lg = self.xd[i % len(self.xd)]
            self.layer.forward(x, lg, y=self.y, keep=keep)
        ev1.record()
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1)
        kt = None
        if with_kernel_times:
            kt = fm.flexmoe_timing_read()
            fm.flexmoe_timing_enable(False)
        return ms, kt

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
        ev0.record()
        for i in range(steps):
            self.use_copy(i)  # shared expert of this copy
            x, lg = self.xd[i % len(self.xd)]
            self.layer.forward(x, lg, y=self.y, clipped=cws[i % len(cws)])
        ev1.record()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1)


def cpu_baseline(wl, keep, target_s):
    """The oracle, untouched, on the first S tokens of the workload."""
    import oracle
    cfg = wl.cfg
    x, lg = wl.batches[0]
    s = wl.s

    def run(S):
        t0 = time.time()
        oracle.layer_forward(x[:S], lg[:S], *wl.w, keep, cfg.top_k, cfg.norm_topk, *s)
        return time.time() - t0

    T = x.shape[0]
    S0 = min(64, T)
    t0 = run(S0)
    S = int(min(T, max(S0, S0 * target_s / max(t0, 1e-3))))
    t = run(S) if S != S0 else t0
    passes = 1
    # the whole batch may take less than the target: repeat it (at most 4 passes)
    while S == T and t < 0.6 * target_s and passes < 4:
        t += run(S)
        passes += 1
    what = ("%d pass%s over all %d tokens" % (passes, "es" if passes > 1 else "", T) if S == T
            else "first %d of %d tokens" % (S, T))
    return dict(value=S * passes / t, unit="tokens/s", cores=oracle.num_threads(), kind="oracle",
                sample="%s of the workload, same weights and keep table, %.1f s (fp64 accumulation)"
                       % (what, t))


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
               roofline_dgrad=dict(kernel="dgrad + SwiGLU backward + mask gradient (act_dgrad_kernel)",
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


def main():
    args = parse()
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
    cfg = synth.CONFIGS[args.workload]
    decode_T = args.decode_T if args.workload == "qwen2_57b_a14b_decode" else None
    wl = Workload(cfg, args.table, args.copies, decode_T)
    bf16 = cfg.dtype == synth.BF16

    if wl.decode:
        # decode: a pool of 64 batches, the 5 nested tables switching every step
        names = ["kept%d" % int(round(f * 100)) for f in synth.NESTED_FRACTIONS]
        per = []
        for b in range(min(64, args.steps + args.warmup)):
            n = wl.counts(b, names[b % len(names)])
            per.append(wl.algorithmic(n, wl.tables[names[b % len(names)]]))
        alg = {k: float(np.mean([p[k] for p in per])) for k in per[0]}
        keep_names = names
    else:
        n = wl.counts(0, wl.table_name)
        alg = wl.algorithmic(n, wl.tables[wl.table_name])
        keep_names = [wl.table_name]

    wl.run(args.warmup, keep_names)
    # The timed region: exactly K steps, no instrumentation inside.
    ms, _ = wl.run(args.steps, keep_names)
    # Per-kernel durations for the roofline: the same K steps again, each
    # kernel bracketed by a HIP event pair on the stream it runs on (the
    # events add a few microseconds per kernel, so this pass is not the one
    # whose step time is reported).
    ms_inst, kt = wl.run(args.steps, keep_names, with_kernel_times=True)
    ms_step = ms / args.steps
    value = wl.T * args.steps / (ms / 1e3)
    log("[bench] %s: %.4f ms/step, %.0f tokens/s (%.4f ms/step with per-kernel events)"
        % (args.workload, ms_step, value, ms_inst / args.steps))
    eager_ms_step = ms_step
    graphs = False
    if wl.decode and args.graphs:
        # decode steps are short: replaying each step's launches from a HIP
        # graph removes the host's launch gaps between its kernels
        wl.capture_graphs(keep_names, 64)
        wl.run_graphs(args.warmup)
        ms_g = wl.run_graphs(args.steps)
        graphs = True
        ms_step = ms_g / args.steps
        value = wl.T * args.steps / (ms_g / 1e3)
        log("[bench] %s: %.4f ms/step, %.0f tokens/s replayed from HIP graphs (eager %.4f ms/step)"
            % (args.workload, ms_step, value, eager_ms_step))
    for kname, (kms, cnt) in kt.items():
        if cnt:
            log("[bench]   %-17s %8.4f ms avg over %d launches" % (kname, kms / cnt, cnt))

    # The gate/up GEMM is one kernel launched once per step over all segments,
    # or twice (routed experts, then the shared expert on the side stream).
    # Its average launch carries the step's gate/up work divided by the
    # launches per step; per launch, achieved = that work / the average
    # launch duration, i.e. the step's gate/up work / the summed durations.
    gu_ms = kt["gate_up"][0] + kt["gate_up_shared"][0]
    gu_n = kt["gate_up"][1] + kt["gate_up_shared"][1]
    gu_avg = gu_ms / max(gu_n, 1)
    gu_per_step = gu_n / args.steps
    gu_avg_step = gu_avg * gu_per_step  # summed gate/up launch time per step
    intensity = alg["F1"] / alg["B1"]
    peak_flops = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
    if intensity >= RIDGE and not wl.decode:
        roof = dict(bound="mfma", achieved=alg["F1"] / (gu_avg_step / 1e3) / 1e12, peak=peak_flops,
                    unit="TFLOP/s")
    else:
        roof = dict(bound="hbm", achieved=alg["B1"] / (gu_avg_step / 1e3) / 1e9, peak=PEAK_HBM_GBS,
                    unit="GB/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = load_traffic(args.workload, wl.T, "+".join(keep_names))
    if not bf16:
        roof["kernel"] = "gate_up GEMM (gemm1_f32_kernel)"
    elif wl.T <= DECODE_WIDE_SHARED_T or (wl.T <= DECODE_MAX_T and not cfg.I_shared and
                                          not (wl.T > DECODE_WIDE_T and wl.T * cfg.top_k >= 8 * cfg.E)):
        roof["kernel"] = "gate_up GEMM (gemm1_decode_kernel)"
    elif wl.T <= DECODE_MAX_T and wl.T > DECODE_WIDE_T and wl.T * cfg.top_k >= 8 * cfg.E:
        roof["kernel"] = "gate_up GEMM (gemm1_decode_wide_kernel)"
    elif wl.T <= DECODE_MAX_T:
        roof["kernel"] = ("gate_up GEMM (gemm1_decode_kernel for the routed experts, "
                          "gemm1_decode_wide_kernel for the shared expert)")
    else:
        roof["kernel"] = "gate_up GEMM (gemm1_big_kernel)"
    roof["avg_launch_ms"] = gu_avg
    roof["launches_per_step"] = gu_per_step
    roof["timing"] = "HIP events around each launch, on its stream, over a second pass of the K steps"
    if kt["gate_up_shared"][1]:
        roof["note"] = ("the shared expert's gate/up launch runs on a side stream concurrently with the "
                        "routed one; each launch's duration includes the time the two share the chip, so "
                        "this per-launch figure is below the layer's own (layer.tflops)")

    layer_s = ms_step / 1e3
    layer = dict(tflops=alg["F"] / layer_s / 1e12, frac_mfma=alg["F"] / layer_s / 1e12 / peak_flops,
                 gbs=alg["B"] / layer_s / 1e9, frac_hbm=alg["B"] / layer_s / 1e9 / PEAK_HBM_GBS,
                 flops_per_step=alg["F"], bytes_per_step=alg["B"],
                 load_weighted_keep=alg["load_weighted_keep"],
                 kernels_ms={k: v[0] / max(v[1], 1) for k, v in kt.items()})

    per_budget = None
    if not args.no_per_budget and not wl.decode:
        per_budget = []
        steps_b = max(5, args.steps // 2)
        for name in ["kept%d" % int(round(f * 100)) for f in synth.NESTED_FRACTIONS]:
            nb = wl.counts(0, name)
            a = wl.algorithmic(nb, wl.tables[name])
            wl.run(2, [name])
            msb, _ = wl.run(steps_b, [name])
            sb = msb / steps_b / 1e3
            # the same budget exported offline (compact weights, Table 2 mode)
            cws = wl.export_clipped(name)
            wl.run_clipped(2, cws)
            so = wl.run_clipped(steps_b, cws) / steps_b / 1e3
            del cws
            # the paper's bucketed design (Alg. 2) as an ablation
            wl.run_bucketed(2, name, args.bucket_align)
            sk = wl.run_bucketed(steps_b, name, args.bucket_align) / steps_b / 1e3
            per_budget.append(dict(table=name, kept=synth.keep_fraction(wl.tables[name], cfg.I),
                                   ms=sb * 1e3, tokens_per_s=wl.T / sb,
                                   tflops=a["F"] / sb / 1e12,
                                   frac_mfma=a["F"] / sb / 1e12 / peak_flops,
                                   frac_hbm=a["B"] / sb / 1e9 / PEAK_HBM_GBS,
                                   offline_ms=so * 1e3, offline_tokens_per_s=wl.T / so,
                                   online_over_offline=so / sb,
                                   bucketed_ms=sk * 1e3, bucketed_k_align=args.bucket_align,
                                   ragged_over_bucketed=sk / sb))
            log("[bench]   budget %-7s %.4f ms  %.0f tok/s  %.1f TFLOP/s | offline %.4f ms, online/offline %.3f"
                " | bucketed(%d) %.4f ms, ragged/bucketed %.3f" %
                (name, sb * 1e3, wl.T / sb, a["F"] / sb / 1e12, so * 1e3, so / sb, args.bucket_align,
                 sk * 1e3, sk / sb))

    # The bucketed ablation on keep tables drawn from the paper's action set
    # {0.1, 0.4, 0.7, 1.0} (at most four width groups, as in its deployments).
    action_ablation = None
    if not args.no_per_budget and not wl.decode:
        action_ablation = []
        levels = [fm.flexmoe_keep_from_ratio(r, cfg.I) for r in synth.ACTION_RATIOS]
        steps_b = max(5, args.steps // 2)
        for f in (0.75, 0.5, 0.25):
            name = "action%d" % int(round(f * 100))
            wl.tables[name] = synth.action_keep_table(cfg.E, levels, 1000 * cfg.config_id + synth._TID_ACTION,
                                                      f)
            wl.keep_dev[name] = fm.to_device(wl.tables[name])
            wl.run(2, [name])
            sb = wl.run(steps_b, [name])[0] / steps_b / 1e3
            wl.run_bucketed(2, name, args.bucket_align)
            sk = wl.run_bucketed(steps_b, name, args.bucket_align) / steps_b / 1e3
            widths = sorted(set(int(v) for v in wl.tables[name] if v > 0))
            action_ablation.append(dict(table=name, kept=synth.keep_fraction(wl.tables[name], cfg.I),
                                        widths=widths, ragged_ms=sb * 1e3, bucketed_ms=sk * 1e3,
                                        bucketed_k_align=args.bucket_align, ragged_over_bucketed=sk / sb))
            log("[bench]   action-set table %-9s kept %.3f widths %s: ragged %.4f ms, bucketed(%d) %.4f ms, "
                "ragged/bucketed %.3f" % (name, synth.keep_fraction(wl.tables[name], cfg.I), widths, sb * 1e3,
                                          args.bucket_align, sk * 1e3, sk / sb))

    saliency = None
    if not args.no_saliency and bf16 and not wl.decode:
        saliency = saliency_section(wl, args)
        if not args.saliency_T:
            # a calibration batch four times the workload's: Eq. 2 reads every
            # weight once per batch, which larger batches amortise
            saliency["batch_x4"] = saliency_section(wl, args, T=4 * wl.T, with_cpu=False)
    action = None
    if not args.no_action and bf16 and not wl.decode:
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
        log("[bench] CPU oracle baseline ...")
        cpu = cpu_baseline(wl, wl.tables[keep_names[0]], args.cpu_seconds)
        log("[bench] CPU oracle: %.2f tokens/s on %d threads" % (cpu["value"], cpu["cores"]))

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
        "eager_ms_per_step": eager_ms_step,
        "roofline": roof,
        "layer": layer,
        "per_budget": per_budget,
        "action_set_ablation": action_ablation,
        "saliency": saliency,
        "action_learning": action,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
