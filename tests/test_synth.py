"""Input generator: determinism, bf16 rounding, keep-table properties."""
import numpy as np
import pytest

from paper_2606_27866_amd import synth


def test_bf16_round_to_nearest_even():
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9, -2.5, 0.0, -0.0, np.inf,
                     3.4028235e38, np.nan], dtype=np.float32)
    b = synth.f32_to_bf16_bits(vals)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa wins (1.0)
    assert b[1] == 0x3F80
    # 1 + 3*2^-9 rounds up to 1 + 2^-7
    assert b[2] == 0x3F81
    assert b[3] == 0xC020 and b[4] == 0 and b[5] == 0x8000 and b[6] == 0x7F80
    assert b[7] == 0x7F80  # above the largest bf16: rounds to inf
    assert b[8] == 0x7FC0
    back = synth.bf16_bits_to_f32(b[:7])
    assert back[0] == 1.0 and back[3] == -2.5


def test_generation_is_deterministic():
    cfg = synth.small_config("det", T=8, d=16, E=4, I=32, top_k=2, config_id=77, bias_std=0.5)
    a = synth.make_tokens(cfg)
    b = synth.make_tokens(cfg)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    w1 = synth.make_expert_weights(cfg)
    w2 = synth.make_expert_weights(cfg)
    for p, q in zip(w1, w2):
        assert p.dtype == np.uint16 and np.array_equal(p, q)


@pytest.mark.parametrize("name", ["tiny_fp32", "qwen15_moe_a27b", "qwen2_57b_a14b_prefill",
                                  "mixtral_8x7b"])
def test_keep_tables(name):
    cfg = synth.CONFIGS[name]
    tables = synth.config_keep_tables(cfg)
    fam = [tables["kept%d" % int(round(f * 100))] for f in synth.NESTED_FRACTIONS]
    for a, b in zip(fam, fam[1:]):
        assert np.all(a >= b)  # nested: a subset chain of kept channels
    for f, t in zip(synth.NESTED_FRACTIONS, fam):
        assert t.min() >= 0 and t.max() <= cfg.I and np.all(t % 64 == 0)
        assert abs(synth.keep_fraction(t, cfg.I) - f) <= 64 / (cfg.E * cfg.I)
    if name == "tiny_fp32":
        own = tables["own"]
        for v in (0, cfg.I, 1, 17, 100, cfg.I - 1):
            assert v in own
    if name == "qwen15_moe_a27b":
        own = tables["own"]
        assert own.sum() == cfg.E * cfg.I // 2 and 0 in own and cfg.I in own
        assert np.all(own % 64 == 0)
    if name == "mixtral_8x7b":
        own = tables["own"]
        assert set(own.tolist()) <= {cfg.I // 4, cfg.I // 2, 3 * cfg.I // 4, cfg.I}
        assert own.sum() * 2 == cfg.E * cfg.I


def test_zipf_bias_gives_zipf_load():
    cfg = synth.CONFIGS["mixtral_8x7b"]
    b = synth.router_bias(cfg)
    g = np.random.default_rng(0)
    lg = g.standard_normal((40000, cfg.E)).astype(np.float32) + b
    top2 = np.argsort(-lg, axis=1)[:, :2]
    share = np.bincount(top2.reshape(-1), minlength=cfg.E) / top2.size
    want = np.sort(synth.zipf_shares(cfg.E, 1.2))[::-1]
    np.testing.assert_allclose(np.sort(share)[::-1], want, atol=0.01)


def test_action_keep_table_uses_only_action_widths():
    levels = [141, 564, 986, 1408]
    for f in (0.9, 0.75, 0.5, 0.25, 0.05):
        t = synth.action_keep_table(60, levels, 7, f)
        assert set(t.tolist()) <= set(levels)
        kept = t.sum() / (60 * 1408)
        # at most the target, unless every expert already sits at the narrowest action
        assert kept <= f + 1e-12 or (t == levels[0]).all()
        # one step wider on any expert would exceed the target (the walk stops at the first fit)
        assert kept > f - (levels[-1] - levels[0]) / (60 * 1408) - 1e-12 or (t == levels[0]).all()


def test_concurrent_draws_equal_serial_draws():
    """The weights drawn concurrently (one thread per tensor) are the bytes of
    drawing each tensor alone, in any order, over several generation chunks."""
    cfg = synth.small_config("conc", T=8, d=1024, E=3, I=6000, top_k=2, I_shared=4096, config_id=78)
    (wg, wu, wd), (sg, su, sd) = synth.make_layer_weights(cfg)
    assert wg.size > synth._CHUNK  # more than one chunk per tensor
    serial = [synth._as_dtype(synth._normal(cfg.config_id, tid, a.size, cfg.w_std).reshape(a.shape), cfg.dtype)
              for tid, a in ((synth._TID_SDOWN, sd), (synth._TID_WUP, wu), (synth._TID_WGATE, wg),
                             (synth._TID_SGATE, sg), (synth._TID_WDOWN, wd), (synth._TID_SUP, su))]
    for got, ref in zip((sd, wu, wg, sg, wd, su), serial):
        assert got.dtype == np.uint16 and np.array_equal(got, ref)
    assert all(np.array_equal(p, q) for p, q in zip(synth.make_expert_weights(cfg), (wg, wu, wd)))
    assert all(np.array_equal(p, q) for p, q in zip(synth.make_shared_weights(cfg), (sg, su, sd)))
