"""Parity at the full sizes of the benchmark workloads, in the launch
configuration bench.py times.

Routing and dispatch are checked bit-exactly for every token against the
oracle's routing and dispatch; y is checked on sampled rows, which the oracle
computes one by one (a token's output depends on that token only).  The
prefill rows include, for every active expert, the tokens of its first
routed row, of the first row of its last (partial) 256-row tile and of its
last routed row, so that every expert's tile edges are compared element by
element.
"""
import functools

import numpy as np
import pytest

import oracle
from paper_2606_27866_amd import synth
from tests.gpu_util import BF16_TOL, GpuLayer, check_y, say

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=1)
def layer_inputs(name):
    cfg = synth.CONFIGS[name]
    say("generating", name)
    w, s = synth.make_layer_weights(cfg)
    return cfg, w, s


@functools.lru_cache(maxsize=1)
def gpu_layer(name):
    cfg, w, s = layer_inputs(name)
    return GpuLayer(cfg.d, cfg.E, cfg.I, cfg.top_k, cfg.I_shared, cfg.dtype, cfg.norm_topk,
                    cfg.T, *w, *s)


def edge_rows(cfg, lg, keep, tile_rows=256):
    """Tokens at every active expert's segment edges in the oracle's own
    dispatch: its first routed row, the first row of its last row tile and
    its last routed row."""
    idx, _ = oracle.route(lg, cfg.top_k, cfg.norm_topk)
    _, offsets, perm, _ = oracle.dispatch(idx, keep, cfg.E)
    rows = []
    for e in range(cfg.E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi > lo:
            last_tile = lo + (hi - lo - 1) // tile_rows * tile_rows
            rows += [perm[lo] // cfg.top_k, perm[last_tile] // cfg.top_k, perm[hi - 1] // cfg.top_k]
    return np.array(rows, dtype=np.int64)


def check_all_routing(cfg, lg, keep, r):
    idx, w = oracle.route(lg, cfg.top_k, cfg.norm_topk)
    counts, offsets, perm, pos = oracle.dispatch(idx, keep, cfg.E)
    np.testing.assert_array_equal(r["topk_idx"], idx)
    np.testing.assert_allclose(r["topk_w"], w, rtol=0, atol=1e-6)
    np.testing.assert_array_equal(r["counts"], counts)
    np.testing.assert_array_equal(r["offsets"], offsets)
    np.testing.assert_array_equal(r["perm"], perm)
    np.testing.assert_array_equal(r["pos"], pos)


CASES = [("qwen15_moe_a27b", "own"), ("qwen15_moe_a27b", "kept20"),
         ("qwen2_57b_a14b_prefill", "kept100"), ("qwen2_57b_a14b_prefill", "kept40"),
         ("mixtral_8x7b", "own"), ("mixtral_8x7b", "kept20")]


@pytest.mark.parametrize("name,table", CASES, ids=["%s-%s" % c for c in CASES])
def test_full_size_prefill(name, table):
    cfg, w, s = layer_inputs(name)
    x, lg = synth.make_tokens(cfg)
    keep = synth.config_keep_tables(cfg)[table]
    g = gpu_layer(name)
    say(name, table, "forward")
    y, r = g.forward(x, lg, keep)
    check_all_routing(cfg, lg, keep, r)
    rng = np.random.default_rng(7)
    rows = np.unique(np.concatenate([[0, cfg.T - 1], rng.choice(cfg.T, 8, replace=False),
                                     edge_rows(cfg, lg, keep)]))
    say(name, table, "oracle on rows", rows.tolist())
    ref = oracle.layer_forward(x[rows], lg[rows], *w, keep, cfg.top_k, cfg.norm_topk, *s)
    check_y(y[rows], ref, BF16_TOL)


@pytest.mark.parametrize("T", [1, 8, 64])
def test_decode_budget_cycling(T):
    """Decode batches of the Qwen2-shaped layer; the budget switches every
    step through the five nested tables."""
    name = "qwen2_57b_a14b_decode"
    cfg, w, s = layer_inputs(name)
    g = gpu_layer(name)
    tables = synth.config_keep_tables(cfg)
    names = ["kept%d" % int(round(f * 100)) for f in synth.NESTED_FRACTIONS]
    bias = synth.router_bias(cfg)
    for step in range(5):
        x, lg = synth.make_tokens(cfg, T=T, batch=step, bias=bias)
        keep = tables[names[step]]
        say("decode T=%d step %d table %s" % (T, step, names[step]))
        y, r = g.forward(x, lg, keep)
        check_all_routing(cfg, lg, keep, r)
        rows = np.arange(T) if T <= 8 else np.arange(0, T, 9)
        ref = oracle.layer_forward(x[rows], lg[rows], *w, keep, cfg.top_k, cfg.norm_topk, *s)
        check_y(y[rows], ref, BF16_TOL)
