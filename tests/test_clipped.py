"""Offline clipping (Sec. 4.4, Table 2): one budget exported as compact weights.

CPU tests pin the oracle's packing (oracle.export_clipped) and the host side
of the C ABI.  GPU tests check the library's export against that packing
byte for byte, and its clipped forward against the online forward on the
ranked weights (bit for bit) and against the oracle.
"""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2606_27866_amd import flexmoe as fm
from paper_2606_27866_amd import synth
from tests.bruteforce import f64, random_layer, router_weights, silu, topk_by_sort
from tests.gpu_util import BF16_TOL, F32_TOL, check_route, check_y, mini_layer, oracle_ref, say


def dense_from_packed(x, logits, gc, uc, dc, keep, E, d, top_k, norm_topk):
    """The MoE layer evaluated straight from packed buffers: expert e uses its
    whole packed block (kp_e channels, no mask) at channel offset ch0_e."""
    X = f64(x)
    T = X.shape[0]
    G = np.zeros((T, E))
    idx = topk_by_sort(logits, top_k)
    w = router_weights(logits, idx, norm_topk)
    G[np.repeat(np.arange(T), top_k), idx.reshape(-1)] = w.reshape(-1)
    Gc, Uc, Dc = f64(gc), f64(uc), f64(dc)
    Y = np.zeros((T, d))
    c0 = 0
    for e in range(E):
        kp = oracle.packed_width(keep[e])
        if kp:
            Wg = Gc[c0 * d:(c0 + kp) * d].reshape(kp, d)
            Wu = Uc[c0 * d:(c0 + kp) * d].reshape(kp, d)
            Wd = Dc[c0 * d:(c0 + kp) * d].reshape(d, kp)
            Y += G[:, e:e + 1] * ((silu(X @ Wg.T) * (X @ Wu.T)) @ Wd.T)
        c0 += kp
    return Y


KEEPS = [[0, 1, 7, 8, 9, 40, 17, 3], [40, 40, 40, 40, 40, 40, 40, 40], [0] * 8, [33, 0, 0, 24, 5, 40, 2, 16]]


@pytest.mark.parametrize("keep", KEEPS)
@pytest.mark.parametrize("bf16", [False, True])
def test_export_pin_packed_layer_equals_masked_layer(keep, bf16):
    """The packed subnetwork, evaluated without any mask, is the masked layer
    of Eq. 4 with the same budget (so no kept channel is lost, misplaced or
    duplicated, and the padding contributes nothing)."""
    rng = np.random.default_rng(31 + len(str(keep)) + bf16)
    T, d, E, I, k = 7, 24, 8, 40, 2
    x, lg, wg, wu, wd, _ = random_layer(rng, T, d, E, I, k, 0, bf16)
    keep = np.asarray(keep, np.int32)
    gc, uc, dc = oracle.export_clipped(keep, wg, wu, wd)
    P = sum(oracle.packed_width(v) for v in keep)
    assert gc.shape == uc.shape == dc.shape == (P * d,)
    ref = oracle.layer_forward(x, lg, wg, wu, wd, keep, k, 1)
    y = dense_from_packed(x, lg, gc, uc, dc, keep, E, d, k, 1)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12 * max(1.0, np.abs(ref).max()))


def test_export_pin_padding_is_zero_and_blocks_in_order():
    rng = np.random.default_rng(5)
    E, I, d = 4, 24, 16
    wg = rng.standard_normal((E, I, d)).astype(np.float32)
    wu = rng.standard_normal((E, I, d)).astype(np.float32)
    wd = rng.standard_normal((E, d, I)).astype(np.float32)
    keep = np.array([3, 0, 24, 9], np.int32)
    gc, uc, dc = oracle.export_clipped(keep, wg, wu, wd)
    c0 = 0
    for e in range(E):
        k, kp = int(keep[e]), oracle.packed_width(keep[e])
        g = gc[c0 * d:(c0 + kp) * d].reshape(kp, d)
        dn = dc[c0 * d:(c0 + kp) * d].reshape(d, kp)
        assert np.array_equal(g[:k], wg[e, :k]) and not g[k:].any()
        assert np.array_equal(dn[:, :k], wd[e, :, :k]) and not dn[:, k:].any()
        c0 += kp
    assert c0 * d == gc.size


# --------------------------------------------------------------------------
# host side of the ABI (no GPU)
# --------------------------------------------------------------------------
def desc_for(E=8, I=40, d=24, dtype=fm.FLEXMOE_BF16):
    return fm.make_desc(d, E, I, 2, 0, dtype, 1, 16)


def test_clipped_channels_host():
    desc = desc_for()
    for keep in KEEPS:
        assert fm.flexmoe_clipped_channels(desc, keep) == sum(oracle.packed_width(v) for v in keep)


@pytest.mark.parametrize("bad", [[-1] + [0] * 7, [41] + [0] * 7])
def test_clipped_rejects_bad_keep(bad):
    desc = desc_for()
    with pytest.raises(fm.FlexMoEError) as ei:
        fm.flexmoe_clipped_channels(desc, bad)
    assert ei.value.code == -3
    with pytest.raises(fm.FlexMoEError) as ei:
        fm.flexmoe_export_clipped(desc, bad, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, stream=0)
    assert ei.value.code == -3


def test_clipped_forward_rejects_bad_packed_count():
    desc = desc_for()
    for P in (-8, 8 * 40 + 8):
        with pytest.raises(fm.FlexMoEError) as ei:
            fm.flexmoe_layer_forward_clipped(desc, 1, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, P,
                                             None, None, None, 0x1000, 0x1000, workspace_bytes=1 << 30,
                                             stream=0)
        assert ei.value.code == -1


# --------------------------------------------------------------------------
# GPU: export bytes, clipped forward == online forward == oracle
# --------------------------------------------------------------------------
CASES = [
    # name, T, d, E, I, k, I_s, dtype, norm
    ("c_f32", 50, 64, 8, 72, 2, 0, synth.F32, 1),
    ("c_f32_shared", 90, 64, 6, 48, 2, 64, synth.F32, 0),
    ("c_prefill", 300, 256, 8, 320, 2, 0, synth.BF16, 1),
    ("c_prefill_shared", 200, 512, 16, 192, 4, 256, synth.BF16, 0),
    ("c_decode", 8, 256, 16, 200, 4, 128, synth.BF16, 0),
    ("c_decode64", 64, 128, 24, 72, 8, 64, synth.BF16, 1),
]


def case_keeps(E, I, seed):
    rng = np.random.default_rng(seed)
    ks = [rng.integers(0, I + 1, size=E).astype(np.int32)]
    edge = np.array([0, 1, 7, 8, 9, I - 1, I, 17] * ((E + 7) // 8), np.int32)[:E]
    ks.append(np.minimum(edge, I))
    return ks


@pytest.mark.gpu
@pytest.mark.parametrize("spec", CASES, ids=[c[0] for c in CASES])
def test_gpu_clipped_matches_online_and_oracle(spec):
    import torch
    name, T, d, E, I, k, I_s, dtype, norm = spec
    cfg, x, lg, w, s = mini_layer(name, T, d, E, I, k, I_s, dtype=dtype, norm=norm,
                                  config_id=120 + CASES.index(spec))
    layer = fm.Layer(d, E, I, k, I_s, dtype, norm, max_tokens=T)
    dev = [fm.to_device(a) if a is not None else None for a in (*w, *s)]
    layer.set_weights(*dev)
    xd, ld = fm.to_device(x), fm.to_device(lg)
    for keep in case_keeps(E, I, 7 + CASES.index(spec)):
        say(name, "keep", keep.tolist())
        cw = layer.export_clipped(keep)
        torch.cuda.synchronize()
        # the export is a pure rearrangement: byte-exact against the oracle's
        gc, uc, dc = oracle.export_clipped(keep, *w)
        P = cw.packed_channels
        for got, ref in zip((cw.w_gate_c, cw.w_up_c, cw.w_down_c), (gc, uc, dc)):
            assert np.array_equal(fm.to_host(got)[:P * d], ref)
        A = T * k
        i32 = dict(dtype=torch.int32, device="cuda")
        dbg_on, dbg_off = ({n: torch.empty(A, **i32) for n in ("topk_idx", "perm", "pos")} for _ in range(2))
        for dbg in (dbg_on, dbg_off):
            dbg["offsets"] = torch.empty(E + 1, **i32)
        layer.set_budget(keep)
        y_on = layer.forward(xd, ld, dbg=dbg_on)
        y_off = layer.forward(xd, ld, clipped=cw, dbg=dbg_off)
        torch.cuda.synchronize()
        # same data multiplied in the same order: identical bits
        assert torch.equal(y_on.view(torch.int16) if y_on.dtype == torch.bfloat16 else y_on,
                           y_off.view(torch.int16) if y_off.dtype == torch.bfloat16 else y_off)
        for key in ("topk_idx", "pos", "offsets"):
            assert torch.equal(dbg_on[key], dbg_off[key]), key
        n_perm = int(dbg_on["offsets"][E])  # entries past P are unspecified
        assert torch.equal(dbg_on["perm"][:n_perm], dbg_off["perm"][:n_perm])
        ref = oracle.layer_forward(x, lg, *w, keep, k, norm, *s)
        yo = synth.bf16_bits_to_f32(fm.to_host(y_off)).astype(np.float64) if dtype == synth.BF16 \
            else fm.to_host(y_off).astype(np.float64)
        check_y(yo, ref, BF16_TOL if dtype == synth.BF16 else F32_TOL)


@pytest.mark.gpu
@pytest.mark.parametrize("T", [40, 300])
def test_gpu_clipped_wrong_table_stays_inside_the_buffers(T):
    """keep_dev wider than the exported budget: experts whose packed block
    would end past packed_channels are skipped, the others read the packed
    buffers with the table's own offsets -- exactly what a dense evaluation of
    that addressing gives (so every access stayed inside the buffers)."""
    import torch
    d, E, I, k = 128, 8, 64, 2
    cfg, x, lg, w, s = mini_layer("c_wrong", T, d, E, I, k, 0, dtype=synth.BF16, norm=1, config_id=140)
    layer = fm.Layer(d, E, I, k, 0, synth.BF16, 1, max_tokens=T)
    layer.set_weights(*[fm.to_device(a) for a in w])
    exported = np.array([16, 8, 0, 24, 8, 40, 8, 16], np.int32)
    wrong = np.array([24, 16, 8, 24, 16, 40, 8, 64], np.int32)
    cw = layer.export_clipped(exported)
    P = cw.packed_channels
    keep_dev = fm.to_device(wrong)
    y = layer.forward(fm.to_device(x), fm.to_device(lg), clipped=cw, keep=keep_dev)
    torch.cuda.synchronize()
    # the addressing the kernels follow, evaluated in NumPy
    gc, uc, dc = (fm.to_host(t)[:P * d] for t in (cw.w_gate_c, cw.w_up_c, cw.w_down_c))
    wg_e, wu_e, wd_e = (np.zeros((E, I, d), np.uint16), np.zeros((E, I, d), np.uint16),
                        np.zeros((E, d, I), np.uint16))
    keep_eff = np.zeros(E, np.int32)
    c0 = 0
    for e in range(E):
        kk, kp = int(wrong[e]), oracle.packed_width(wrong[e])
        if c0 + kp <= P:
            keep_eff[e] = kk
            wg_e[e, :kk] = gc[c0 * d:(c0 + kk) * d].reshape(kk, d)
            wu_e[e, :kk] = uc[c0 * d:(c0 + kk) * d].reshape(kk, d)
            wd_e[e, :, :kk] = dc[c0 * d:(c0 + kp) * d].reshape(d, kp)[:, :kk]
        c0 += kp
    assert keep_eff.tolist() == [24, 16, 8, 24, 16, 0, 0, 0]
    ref = oracle.layer_forward(x, lg, wg_e, wu_e, wd_e, keep_eff, k, 1)
    check_y(synth.bf16_bits_to_f32(fm.to_host(y)).astype(np.float64), ref, BF16_TOL)


@pytest.mark.gpu
def test_gpu_clipped_full_size_qwen15():
    """The benchmark workload's own table, offline vs online, bit for bit."""
    import torch
    cfg = synth.CONFIGS["qwen15_moe_a27b"]
    g = torch.Generator(device="cuda")
    g.manual_seed(3)

    def rnd(*shape):
        return (torch.randn(*shape, device="cuda", generator=g) * 0.02).to(torch.bfloat16)

    x, lg = synth.make_tokens(cfg)
    keep = synth.config_keep_tables(cfg)["own"]
    layer = fm.Layer(cfg.d, cfg.E, cfg.I, cfg.top_k, cfg.I_shared, cfg.dtype, cfg.norm_topk, cfg.T)
    layer.set_weights(rnd(cfg.E, cfg.I, cfg.d), rnd(cfg.E, cfg.I, cfg.d), rnd(cfg.E, cfg.d, cfg.I),
                      rnd(cfg.I_shared, cfg.d), rnd(cfg.I_shared, cfg.d), rnd(cfg.d, cfg.I_shared))
    layer.set_budget(keep)
    cw = layer.export_clipped(keep)
    xd, ld = fm.to_device(x), fm.to_device(lg)
    y_on = layer.forward(xd, ld)
    y_off = layer.forward(xd, ld, clipped=cw)
    torch.cuda.synchronize()
    assert torch.equal(y_on.view(torch.int16), y_off.view(torch.int16))
