"""Host logic of bench.py that needs no GPU: the one-GPU guard, the
algorithmic flop and byte counts behind the reported TFLOP/s, GB/s and
roofline, the staleness check of the committed HBM-traffic records, and the
token-count thresholds that name the roofline's kernel."""
import json
import os
import re
import subprocess
import sys
import types

import numpy as np
import pytest

import bench
from paper_2606_27866_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""  # no JSON line for a configuration that was not measured


def _fake_workload(cfg, T):
    return types.SimpleNamespace(cfg=cfg, T=T, synth=synth)


def _brute_force_counts(cfg, T, idx, keep):
    """Flops and bytes summed assignment by assignment: each routed token of
    expert e multiplies d x k_e gate, d x k_e up and k_e x d down weights
    (2 flops per multiply-add); the shared expert does the same over I_s for
    every token.  An expert's weights are read once if it has any token and
    any kept channel; x and y once per token; the fp32 logits once."""
    sw = 2 if cfg.dtype == synth.BF16 else 4
    F = F1 = 0
    touched = set()
    for t in range(T):
        for e in idx[t]:
            ke = int(keep[e])
            if ke == 0:
                continue
            touched.add(int(e))
            F1 += 2 * cfg.d * ke * 2          # gate and up
            F += 2 * cfg.d * ke * 2 + 2 * ke * cfg.d
        F1 += 2 * cfg.d * cfg.I_shared * 2
        F += 2 * cfg.d * cfg.I_shared * 3
    kept_w = sum(int(keep[e]) for e in touched)
    B = (3 * cfg.d * kept_w * sw + 3 * cfg.d * cfg.I_shared * sw + T * cfg.d * sw + T * cfg.d * sw
         + T * cfg.E * 4)
    # gate/up GEMM alone: its weights, x, and the activations it writes
    h_elems = sum(int(keep[e]) for t in range(T) for e in idx[t]) + T * cfg.I_shared
    B1 = 2 * cfg.d * (kept_w + cfg.I_shared) * sw + T * cfg.d * sw + h_elems * sw
    return F, B, F1, B1


@pytest.mark.parametrize("I_shared,dtype", [(0, synth.F32), (96, synth.BF16)])
def test_algorithmic_counts_match_a_count_per_assignment(I_shared, dtype):
    rng = np.random.default_rng(7)
    T, d, E, I, k = 37, 48, 9, 160, 3
    cfg = synth.small_config("count", T=T, d=d, E=E, I=I, top_k=k, I_shared=I_shared, dtype=dtype)
    # expert 4 gets no token: its weights are not read
    candidates = [e for e in range(E) if e != 4]
    idx = np.stack([rng.choice(candidates, size=k, replace=False) for _ in range(T)])
    keep = rng.integers(1, I + 1, size=E)
    keep[2] = 0            # pruned expert: its tokens cost nothing
    keep[7] = I            # unpruned expert
    n = np.bincount(idx.ravel(), minlength=E).astype(np.int64)
    got = bench.Workload.algorithmic(_fake_workload(cfg, T), n, keep)
    F, B, F1, B1 = _brute_force_counts(cfg, T, idx, keep)
    assert (got["F"], got["B"], got["F1"], got["B1"]) == (F, B, F1, B1)
    routed = [(t, e) for t in range(T) for e in idx[t]]
    assert got["load_weighted_keep"] == pytest.approx(sum(int(keep[e]) for _, e in routed) / (len(routed) * I))


def test_full_budget_counts_equal_the_unpruned_layer():
    cfg = synth.CONFIGS["qwen15_moe_a27b"]
    T = 4096
    n = np.full(cfg.E, T * cfg.top_k // cfg.E, dtype=np.int64)
    n[: T * cfg.top_k - int(n.sum())] += 1
    got = bench.Workload.algorithmic(_fake_workload(cfg, T), n, np.full(cfg.E, cfg.I))
    # every routed token runs a full I-wide SwiGLU expert, every token the shared one
    assert got["F"] == 6 * cfg.d * (T * cfg.top_k * cfg.I + T * cfg.I_shared)
    assert got["load_weighted_keep"] == 1.0


def _write_record(path, **kw):
    rec = dict(kernel_src_sha=bench.kernel_src_hash(), table="own", T=4096, hbm_bytes_per_launch=123456789)
    rec.update(kw)
    with open(path, "w") as f:
        json.dump(rec, f)


@pytest.mark.parametrize("change,expect", [
    ({}, 123456789),
    ({"kernel_src_sha": "0" * 16}, None),   # counters taken on other kernel sources
    ({"table": "kept100"}, None),
    ({"T": 8192}, None),
])
def test_traffic_record_is_used_only_for_the_same_kernels_table_and_T(tmp_path, monkeypatch, change, expect):
    path = str(tmp_path / "rec.json")
    _write_record(path, **change)
    monkeypatch.setattr(bench, "traffic_file", lambda workload, T: path)
    assert bench.load_traffic("qwen15_moe_a27b", 4096, "own") == expect


def test_kernel_hash_ignores_comments_but_not_code():
    """A comment edit keeps the counter records valid; a code edit does not."""
    src = {}

    def read(f):
        if f not in src:
            src[f] = open(os.path.join(bench.ROOT, "paper_2606_27866_amd", "csrc", f)).read()
        return src[f]

    base = bench.kernel_src_hash(read)
    assert base == bench.kernel_src_hash()
    text = read("gemm_bf16_big.hip")
    src["gemm_bf16_big.hip"] = "// a new comment line\n\n" + text.replace("namespace flexmoe {", "namespace flexmoe {  // note", 1)
    assert bench.kernel_src_hash(read) == base
    src["gemm_bf16_big.hip"] = text.replace("constexpr int NSB = 2;", "constexpr int NSB = 3;", 1)
    assert src["gemm_bf16_big.hip"] != text
    assert bench.kernel_src_hash(read) != base


def test_missing_traffic_record_gives_null(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "traffic_file", lambda workload, T: str(tmp_path / "absent.json"))
    assert bench.load_traffic("qwen15_moe_a27b", 4096, "own") is None


def test_kernel_thresholds_match_the_library():
    """The roofline names its kernel from the token count with the library's
    own thresholds; they must be the ones the dispatch uses."""
    src = open(os.path.join(ROOT, "paper_2606_27866_amd", "csrc", "kernels.h")).read()

    def const(name):
        m = re.search(r"constexpr int %s = (\d+);" % name, src)
        assert m, name
        return int(m.group(1))

    assert bench.DECODE_MAX_T == const("kDecodeMaxT")
    assert bench.GEMV_MAX_T == const("kGemvMaxT")
    assert bench.DECODE_WIDE_SHARED_T == const("kDecodeWideSharedT")


def test_traffic_records_name_their_workload():
    for wl, T in (("qwen15_moe_a27b", 4096), ("qwen2_57b_a14b_decode", 1), ("qwen2_57b_a14b_decode", 64)):
        p = bench.traffic_file(wl, T)
        assert os.path.dirname(p) == os.path.join(ROOT, "profiles")
        assert wl in os.path.basename(p)
    assert bench.traffic_file("qwen2_57b_a14b_decode", 8).endswith("_T8.json")


def test_default_run_is_the_largest_single_gpu_layer():
    """With no flags the headline is the Mixtral-8x7B-shaped layer (T = 16384,
    the largest configuration), with the further sections after it."""
    a = bench.parse([])
    assert a.workload == "mixtral_8x7b" and a.gpus == 1
    cfg = synth.CONFIGS[a.workload]
    assert cfg.T == max(c.T for c in synth.CONFIGS.values())
    assert set(a.extras.split(",")) == {"qwen2_prefill", "decode", "qwen15"}
    assert a.min_warmup_s >= 1.0   # warm-up lasts a while whatever --warmup says


def test_step_stats_are_order_statistics_of_the_steps():
    rng = np.random.default_rng(3)
    ms = rng.uniform(1.0, 2.0, size=101)
    st = bench.step_stats(list(ms))
    s = np.sort(ms)
    assert st["median"] == s[50] and st["n"] == 101
    assert st["p10"] == pytest.approx(s[10]) and st["p90"] == pytest.approx(s[90])
    assert st["p10"] <= st["median"] <= st["p90"]
    assert st["mean"] == pytest.approx(ms.mean())


@pytest.mark.parametrize("T,name", [(1, "gemv1_kernel"), (5, "gemv1_kernel"),
                                    (8, "gemv1_kernel for the routed experts, gemm1_decode_wide_kernel "
                                        "for the shared expert"),
                                    (9, "gemm1_decode_wide_kernel"),
                                    (64, "gemm1_decode_wide_kernel"), (65, "gemm1_big_kernel")])
def test_gate_up_kernel_named_from_the_library_thresholds(T, name):
    cfg = synth.CONFIGS["qwen2_57b_a14b_decode"]
    assert bench.gate_up_kernel_name(cfg, T) == name
    assert bench.gate_up_kernel_name(synth.CONFIGS["mixtral_8x7b"], 16384) == "gemm1_big_kernel"
    assert bench.gate_up_kernel_name(synth.CONFIGS["tiny_fp32"], 64) == "gemm1_f32_kernel"


def test_cpu_info_names_the_model_and_counts():
    info = bench.cpu_info()
    assert info["nproc"] >= 1 and 1 <= info["usable_cpus"] <= info["nproc"]
    assert isinstance(info["cpu_model"], str) and info["cpu_model"]
