"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars: routing ids, counts, offsets, dispatch permutation and inverse are
bit-exact; router weights within 1e-6; y within 2e-2 * max|ref| for bf16
inputs and 1e-5 * max|ref| in fp32 mode (oracle in fp64, unrounded).
"""
import numpy as np
import pytest

import oracle
from paper_2606_27866_amd import flexmoe as fm
from paper_2606_27866_amd import synth
from tests.gpu_util import (BF16_TOL, F32_TOL, GpuLayer, check_route, check_y, mini_layer,
                            oracle_ref, say, y_to_f64)

pytestmark = pytest.mark.gpu


def gpu_layer_for(cfg, w, s, max_tokens=None):
    return GpuLayer(cfg.d, cfg.E, cfg.I, cfg.top_k, cfg.I_shared, cfg.dtype, cfg.norm_topk,
                    max_tokens or cfg.T, *w, *s)


def test_native_library_is_the_one_loaded():
    L = fm.lib()
    assert L._name.endswith("paper_2606_27866_amd/libflexmoe.so")


# --------------------------------------------------------------------------
# tiny fp32 layer: every keep table, 1e-5
# --------------------------------------------------------------------------
def tiny_tables(cfg):
    t = dict(synth.config_keep_tables(cfg))
    t["edges_a"] = np.array([0, 1, 15, 16, 17, 63, 64, 65], np.int32)
    t["edges_b"] = np.array([cfg.I - 1, cfg.I, 0, 1, 17, 100, 511, 512], np.int32)
    t["one_channel"] = np.ones(cfg.E, np.int32)
    return t


def test_tiny_fp32_all_tables():
    cfg = synth.CONFIGS["tiny_fp32"]
    x, lg = synth.make_tokens(cfg)
    w = synth.make_expert_weights(cfg)
    g = gpu_layer_for(cfg, w, (None, None, None))
    for name, keep in tiny_tables(cfg).items():
        say("tiny_fp32 table", name, keep.tolist())
        y, r = g.forward(x, lg, keep)
        ref, rr = oracle_ref(cfg, x, lg, w, (None, None, None), keep)
        check_route(r, rr)
        check_y(y, ref, F32_TOL)


def test_fp32_multi_chunk_dispatch():
    """fp32 layer whose T*top_k exceeds one dispatch workgroup."""
    cfg, x, lg, w, s = mini_layer("f32_big", 600, 64, 8, 96, 2, 32, dtype=synth.F32, config_id=77)
    g = gpu_layer_for(cfg, w, s)
    keep = np.array([96, 0, 17, 64, 65, 1, 96, 33], np.int32)
    y, r = g.forward(x, lg, keep)
    ref, rr = oracle_ref(cfg, x, lg, w, s, keep)
    check_route(r, rr)
    check_y(y, ref, F32_TOL)


def test_tiny_fp32_zero_budget_is_exact_zero():
    cfg = synth.CONFIGS["tiny_fp32"]
    x, lg = synth.make_tokens(cfg)
    w = synth.make_expert_weights(cfg)
    g = gpu_layer_for(cfg, w, (None, None, None))
    y, r = g.forward(x, lg, np.zeros(cfg.E, np.int32))
    assert np.all(y == 0.0)
    assert np.all(r["pos"] == -1) and r["offsets"][-1] == 0


# --------------------------------------------------------------------------
# bf16 layers of several tiles with ragged tails
# --------------------------------------------------------------------------
MINIS = [
    # name, T, d, E, I, k, I_s, norm
    ("m_a", 300, 256, 8, 320, 2, 0, 1),
    ("m_b", 200, 512, 60, 192, 4, 256, 0),
    ("m_topk_eq_E", 129, 128, 16, 136, 16, 0, 1),
    ("m_top1", 77, 64, 5, 64, 1, 0, 1),
    ("m_256_experts", 100, 64, 256, 64, 8, 64, 0),
    ("m_shared_wide", 150, 192, 6, 72, 2, 520, 1),
    # T*top_k = 1024 is the largest batch dispatched by one workgroup, 1026
    # takes the three-kernel dispatch path
    ("m_dispatch_1024", 512, 64, 8, 64, 2, 0, 1),
    ("m_dispatch_1026", 513, 64, 8, 64, 2, 64, 0),
    # a decode-sized batch with 16 experts per token (T*top_k = 1024)
    ("m_decode_top16", 64, 128, 24, 72, 16, 64, 0),
    # few down tiles and a wide shared expert: its reduction is split into
    # chunks (2 of 1024 channels; 3 of 1088, 1088 and 904)
    ("m_shared_split2", 300, 256, 8, 128, 2, 2048, 1),
    ("m_shared_split3", 200, 128, 4, 64, 2, 3080, 0),
    # 10 chunks of 1024: the combine adds the shared row sets in two batches
    # of 8 (the prefill combine's top-2 variant)
    ("m_shared_split10", 200, 128, 4, 64, 2, 10240, 1),
    # a shared expert with 16 x 64 = 1024 gate/up tiles fills the GPU on its
    # own: it runs as segment 0 of the routed experts' launches (no side
    # stream), and its down reduction is split into 8 chunks
    ("m_shared_one_launch", 4096, 64, 8, 64, 2, 8192, 1),
]


@pytest.mark.parametrize("spec", MINIS, ids=[m[0] for m in MINIS])
def test_bf16_mini(spec):
    name, T, d, E, I, k, I_s, norm = spec
    cfg, x, lg, w, s = mini_layer(name, T, d, E, I, k, I_s, norm=norm, config_id=60 + MINIS.index(spec))
    g = gpu_layer_for(cfg, w, s)
    rng = np.random.default_rng(len(name))
    tables = [np.full(E, I, np.int32), rng.integers(0, I + 1, size=E).astype(np.int32)]
    edge = np.array([0, 1, 15, 16, 17, 63, 64, 65, I - 1, I], np.int32)
    tables.append(np.minimum(np.resize(edge, E), I))
    for keep in tables:
        say(name, "keep", keep[:12].tolist())
        y, r = g.forward(x, lg, keep)
        ref, rr = oracle_ref(cfg, x, lg, w, s, keep)
        check_route(r, rr)
        check_y(y, ref, BF16_TOL)


@pytest.mark.parametrize("T", [1, 2, 63, 64, 65, 129])
def test_bf16_token_counts(T):
    cfg, x, lg, w, s = mini_layer("t%d" % T, 129, 128, 8, 96, 2, 64, config_id=70)
    x, lg = x[:T], lg[:T]
    g = gpu_layer_for(cfg, w, s, max_tokens=129)
    keep = np.array([96, 0, 17, 64, 65, 1, 96, 33], np.int32)
    y, r = g.forward(x, lg, keep)
    ref, rr = oracle_ref(cfg, x, lg, w, s, keep)
    check_route(r, rr)
    check_y(y, ref, BF16_TOL)


def test_bf16_decode_shared_partial_rows_fit_a_smaller_token_count():
    """The shared expert's down reduction at decode is split into chunks of
    I channels up to 16 tokens and of 2I above: a workspace sized for 24
    tokens (4 partial rows per token) must also hold 16 tokens' 8 each."""
    cfg, x, lg, w, s = mini_layer("osrows", 24, 64, 4, 64, 2, 512, config_id=75)
    g = gpu_layer_for(cfg, w, s, max_tokens=24)
    keep = np.array([64, 7, 0, 40], np.int32)
    for T in (16, 24, 16):
        y, r = g.forward(x[:T], lg[:T], keep)
        ref, rr = oracle_ref(cfg, x[:T], lg[:T], w, s, keep)
        check_route(r, rr)
        check_y(y, ref, BF16_TOL)


@pytest.mark.parametrize("T", [5, 6, 8, 17, 31, 33, 49, 64])
def test_bf16_shared_expert_wide_decode_tiles(T):
    """6..64 tokens: the shared expert's GEMMs take 64-wide tiles (the routed
    experts' too from 24 tokens on at this E and k; 5 tokens: neither).  d = 264
    leaves a partial 256-deep K batch, I_s = 216 a partial channel tile and a
    ragged last reduction chunk (chunks of I = 40 channels), and T a partial
    16-token block."""
    cfg, x, lg, w, s = mini_layer("wide%d" % T, 64, 264, 6, 40, 2, 216, config_id=72)
    x, lg = x[:T], lg[:T]
    g = gpu_layer_for(cfg, w, s, max_tokens=64)
    for keep in (np.full(6, 40, np.int32), np.array([40, 0, 17, 8, 1, 33], np.int32)):
        y, r = g.forward(x, lg, keep)
        ref, rr = oracle_ref(cfg, x, lg, w, s, keep)
        check_route(r, rr)
        check_y(y, ref, BF16_TOL)


@pytest.mark.parametrize("T", [1, 4, 6, 16, 17, 40, 64])
def test_bf16_decode_with_shared_expert_every_output_written(T):
    """Decode-sized batches with a shared expert whose down reduction is
    split into many row sets (chunks of I or 2I channels), across the 16- and
    64-wide tile choices.  d = 328 leaves a last 64-column tile of 8 columns;
    the tables prune every routed expert (the shared row sets alone make y),
    keep one expert, mix widths, keep all.  Each call is repeated into
    outputs filled with NaN and must write every element with the same bits."""
    import torch
    E, I = 12, 96
    cfg, x, lg, w, s = mini_layer("dsh%d" % T, 64, 328, E, I, 4, 1184, config_id=91)
    x, lg = x[:T], lg[:T]
    g = gpu_layer_for(cfg, w, s, max_tokens=64)
    one = np.zeros(E, np.int32)
    one[int(np.argmax(lg[0]))] = I  # the first token's top expert
    rng = np.random.default_rng(T)
    tables = (np.zeros(E, np.int32), one, rng.integers(0, I + 1, size=E).astype(np.int32),
              np.full(E, I, np.int32))
    for keep in tables:
        say("decode T", T, "keep", keep.tolist())
        y, r = g.forward(x, lg, keep)
        ref, rr = oracle_ref(cfg, x, lg, w, s, keep)
        check_route(r, rr)
        check_y(y, ref, BF16_TOL)
        # the same call again, into outputs filled with NaN: every element
        # is written, with the same bits
        xd, ld = fm.to_device(x), fm.to_device(np.ascontiguousarray(lg, np.float32))
        for _ in range(3):
            yb = torch.full((T, cfg.d), float("nan"), dtype=torch.bfloat16, device="cuda")
            g.layer.forward(xd, ld, y=yb)
            torch.cuda.synchronize()
            assert np.array_equal(y, y_to_f64(fm.to_host(yb)))


@pytest.mark.parametrize("T", [1, 2, 3, 5, 7, 8])
def test_bf16_vector_alu_decode_tiles(T):
    """Up to 8 tokens the 16-wide weight-streaming tiles run on the vector
    ALUs: each segment's rows are a template bound of 1, 2, 4 or 8 (T = 3, 5,
    7 leave rows past the segment's), d = 776 ends in a 256-deep K batch with
    one 8-wide chunk, I = 264 and I_s = 520 end in partial 16-channel tiles,
    and the widths cross every chunk and tile edge.  One pass sends every
    token to expert 2 first, so a routed segment holds all T rows."""
    E, I = 6, 264
    cfg, x, lg, w, s = mini_layer("valu%d" % T, 8, 776, E, I, 2, 520, config_id=93)
    x, lg = x[:T], lg[:T]
    g = gpu_layer_for(cfg, w, s, max_tokens=8)
    skew = np.ascontiguousarray(lg + np.array([0, 0, 50, 0, 0, 0], np.float32))
    tables = (np.full(E, I, np.int32), np.array([1, 7, 9, 15, 17, 263], np.int32),
              np.array([8, 16, 0, 255, 256, 257], np.int32))
    for logits in (lg, skew):
        for keep in tables:
            say("valu T", T, "keep", keep.tolist())
            y, r = g.forward(x, logits, keep)
            ref, rr = oracle_ref(cfg, x, logits, w, s, keep)
            check_route(r, rr)
            check_y(y, ref, BF16_TOL)


def test_all_tokens_on_one_expert_and_ties():
    cfg, x, lg, w, s = mini_layer("skew", 257, 128, 8, 128, 2, 0, config_id=71)
    g = gpu_layer_for(cfg, w, s)
    keep = np.array([128, 77, 0, 128, 5, 64, 128, 1], np.int32)
    cases = {
        "one_expert": lg + np.array([50, 0, 0, 0, 0, 0, 0, 0], np.float32),
        "quantised_ties": np.round(lg * 2) / 2,
        "all_equal": np.zeros_like(lg),
        "nan_logit": np.where(np.arange(lg.shape[1])[None, :] == 3, np.float32(np.nan), lg),
        # -0 and +0 compare equal: every token ties everywhere, so experts 0 and 1
        "signed_zeros": np.where((np.arange(lg.shape[1])[None, :] + np.arange(lg.shape[0])[:, None]) % 2 == 0,
                                 np.float32(-0.0), np.float32(0.0)).astype(np.float32),
        # +inf first, -inf after every finite logit, NaN after -inf
        "infinities": np.where(np.arange(lg.shape[1])[None, :] == 2, np.float32(-np.inf),
                               np.where((np.arange(lg.shape[1])[None, :] == 5) & (np.arange(lg.shape[0])[:, None] % 2 == 0),
                                        np.float32(np.inf),
                                        np.where((np.arange(lg.shape[1])[None, :] == 6)
                                                 & (np.arange(lg.shape[0])[:, None] % 3 == 0), np.float32(np.nan), lg))),
    }
    for name, l2 in cases.items():
        say("routing case", name)
        l2 = np.ascontiguousarray(l2, np.float32)
        y, r = g.forward(x, l2, keep)
        ref, rr = oracle_ref(cfg, x, l2, w, s, keep)
        np.testing.assert_array_equal(r["topk_idx"], rr["idx"])
        np.testing.assert_array_equal(r["perm"], rr["perm"])
        np.testing.assert_array_equal(r["pos"], rr["pos"])
        if name not in ("nan_logit", "infinities"):  # weights of those rows are not finite
            check_route(r, rr)
            check_y(y, ref, BF16_TOL)


def test_zero_budget_bf16_exact_zero_and_shared_only():
    cfg, x, lg, w, s = mini_layer("zero", 100, 128, 8, 64, 2, 0, config_id=72)
    g = gpu_layer_for(cfg, w, s)
    y, _ = g.forward(x, lg, np.zeros(cfg.E, np.int32))
    assert np.all(y == 0.0)
    cfg2, x2, lg2, w2, s2 = mini_layer("zero_sh", 100, 128, 8, 64, 2, 96, config_id=73)
    g2 = gpu_layer_for(cfg2, w2, s2)
    y2, _ = g2.forward(x2, lg2, np.zeros(cfg2.E, np.int32))
    ref = oracle.layer_forward(x2, lg2, *w2, np.zeros(cfg2.E, np.int32), cfg2.top_k, 1, *s2)
    check_y(y2, ref, BF16_TOL)


def test_deterministic_bits():
    cfg, x, lg, w, s = mini_layer("det", 333, 256, 16, 128, 4, 128, config_id=74)
    g = gpu_layer_for(cfg, w, s)
    keep = np.arange(16, dtype=np.int32) * 8
    y1, r1 = g.forward(x, lg, keep)
    y2, r2 = g.forward(x, lg, keep)
    assert np.array_equal(y1, y2)
    for k in r1:
        assert np.array_equal(r1[k], r2[k])


def test_budget_switch_stream_ordered():
    """Five nested tables set with flexmoe_set_budget between forwards queued
    on one stream with no host sync in between: each output matches the
    oracle for its own table."""
    import torch
    cfg, x, lg, w, s = mini_layer("switch", 256, 256, 8, 256, 2, 128, config_id=75)
    g = gpu_layer_for(cfg, w, s)
    fam = synth.nested_keep_family(cfg.E, cfg.I, seed=99, grid=16)
    xd, ld = fm.to_device(x), fm.to_device(lg)
    ys = []
    for keep in fam:
        g.layer.set_budget(keep)
        ys.append(g.layer.forward(xd, ld))
    torch.cuda.synchronize()
    for keep, yd in zip(fam, ys):
        y = synth.bf16_bits_to_f32(fm.to_host(yd)).astype(np.float64)
        ref = oracle.layer_forward(x, lg, *w, keep, cfg.top_k, cfg.norm_topk, *s)
        check_y(y, ref, BF16_TOL)
    # zero-copy switch: a different device keep table per forward
    tables = [fm.to_device(k) for k in fam]
    outs = [g.layer.forward(xd, ld, keep=t) for t in tables]
    torch.cuda.synchronize()
    for a, b in zip(ys, outs):
        assert torch.equal(a, b)


# --------------------------------------------------------------------------
# rank + reorder (Eq. 3)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_rank_reorder(dtype):
    import torch
    cfg, x, lg, w, s = mini_layer("rr", 64, 128, 6, 200, 2, 0, dtype=dtype, config_id=76)
    rng = np.random.default_rng(3)
    scores = np.abs(rng.standard_normal((cfg.E, cfg.I))).astype(np.float32)
    scores[1] = np.round(scores[1] * 4) / 4  # ties
    scores[2, 7] = np.nan
    wg_r, wu_r, wd_r, perm = oracle.rank_reorder(scores, *w)
    desc = fm.make_desc(cfg.d, cfg.E, cfg.I, cfg.top_k, 0, dtype, cfg.norm_topk, cfg.T)
    dev = [fm.to_device(a) for a in w]
    outs = [torch.empty_like(t) for t in dev]
    pd = torch.empty((cfg.E, cfg.I), dtype=torch.int32, device="cuda")
    fm.flexmoe_rank_reorder(desc, fm.to_device(scores), *dev, *outs, pd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(pd.cpu().numpy(), perm)
    for o, ref in zip(outs, (wg_r, wu_r, wd_r)):
        assert np.array_equal(fm.to_host(o), ref)
    # permutation invariance on the GPU: ranked full layer == original full layer
    full = np.full(cfg.E, cfg.I, np.int32)
    g0 = gpu_layer_for(cfg, w, s)
    g1 = gpu_layer_for(cfg, (wg_r, wu_r, wd_r), s)
    y0, _ = g0.forward(x, lg, full)
    y1, _ = g1.forward(x, lg, full)
    tol = F32_TOL if dtype == synth.F32 else BF16_TOL
    check_y(y1, y0, tol)
