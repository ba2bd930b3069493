"""The no-allocation forward (flexmoe_layer_forward_noalloc) against the
workspace forward (flexmoe_layer_forward), both through the C ABI, on the
same seeded inputs.

Each case makes calls in a row with decreasing T (the static scratch keeps
the previous call's contents), checks the routing and dispatch copies bit
for bit against the workspace forward's, y within the bar of the dtype
(2e-2 * max|ref| in bf16, 1e-5 in fp32) against the workspace forward's y,
and y against the oracle at the same bar.  Decode-sized batches cover the
16- and 64-wide weight-streaming tiles with the shared expert's split down
reduction in the same launches as the routed experts; larger batches the
prefill tiles.
"""
import numpy as np
import pytest

from paper_2606_27866_amd import flexmoe as fm
from paper_2606_27866_amd import synth
from tests.gpu_util import BF16_TOL, F32_TOL, check_route, check_y, oracle_ref, say, y_to_f64

pytestmark = pytest.mark.gpu

CASES = [
    # name, d, E, I, k, I_s, norm, dtype, token counts (called in this order)
    ("decode_shared", 512, 16, 256, 4, 1024, 0, synth.BF16, (48, 8, 1)),
    ("prefill_shared", 512, 60, 192, 4, 256, 0, synth.BF16, (200, 70)),
    ("no_shared", 256, 8, 320, 2, 0, 1, synth.BF16, (300, 3)),
    ("fp32", 256, 8, 512, 2, 64, 1, synth.F32, (64, 9)),
]


def _route_bufs(torch, T, k, E):
    A = max(T * k, 1)
    i32 = dict(dtype=torch.int32, device="cuda")
    return dict(topk_idx=torch.full((A,), -7, **i32),
                topk_w=torch.full((A,), -7.0, dtype=torch.float32, device="cuda"),
                counts=torch.full((E,), -7, **i32), offsets=torch.full((E + 1,), -7, **i32),
                perm=torch.full((A,), -7, **i32), pos=torch.full((A,), -7, **i32))


def _route_host(dbg, T, k):
    r = {n: v.cpu().numpy() for n, v in dbg.items()}
    r["topk_idx"] = r["topk_idx"][:T * k].reshape(T, k)
    r["topk_w"] = r["topk_w"][:T * k].reshape(T, k)
    r["pos"] = r["pos"][:T * k]
    r["perm"] = r["perm"][:int(r["offsets"][-1])]
    return r


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_workspace_forward(case):
    import torch
    name, d, E, I, k, I_s, norm, dtype, Ts = case
    Tmax = max(Ts)
    cfg = synth.LayerConfig("noalloc_" + name, 64, T=Tmax, d=d, E=E, I=I, top_k=k, I_shared=I_s, dtype=dtype,
                            norm_topk=norm, bias_std=0.5, w_std=0.05)
    (wg, wu, wd), (sg, su, sd) = synth.make_layer_weights(cfg)
    layer = fm.Layer(d, E, I, k, I_s, dtype, norm, max_tokens=Tmax)
    dev = [fm.to_device(a) if a is not None else None for a in (wg, wu, wd, sg, su, sd)]
    layer.set_weights(*dev)
    rng = np.random.default_rng(11)
    tol = BF16_TOL if dtype == synth.BF16 else F32_TOL
    bias = synth.router_bias(cfg)
    for i, T in enumerate(Ts):
        x, lg = synth.make_tokens(cfg, T=T, batch=i, bias=bias)
        keep = rng.integers(0, I + 1, size=E).astype(np.int32)
        keep[rng.integers(0, E)] = 0
        keep[rng.integers(0, E)] = I
        say("noalloc", name, "T", T, "keep", keep.tolist())
        layer.set_budget(keep)
        xd, ld = fm.to_device(x), fm.to_device(lg)
        dbg_ws, dbg_na = _route_bufs(torch, T, k, E), _route_bufs(torch, T, k, E)
        y_ws = layer.forward(xd, ld, dbg=dbg_ws)
        y_na = torch.full((T, d), float("nan"), dtype=layer.tdtype, device="cuda")
        fm.flexmoe_layer_forward_noalloc(layer.desc, T, xd, ld, *dev[:3], layer.keep, *dev[3:], y_na, dbg=dbg_na)
        torch.cuda.synchronize()
        r_ws, r_na = _route_host(dbg_ws, T, k), _route_host(dbg_na, T, k)
        for n in ("topk_idx", "topk_w", "counts", "offsets", "perm", "pos"):
            np.testing.assert_array_equal(r_na[n], r_ws[n], err_msg=n)
        yw, yn = y_to_f64(fm.to_host(y_ws)), y_to_f64(fm.to_host(y_na))
        assert np.isfinite(yn).all()
        e_ws = check_y(yn, yw, tol)
        ref, rr = oracle_ref(cfg, x, lg, (wg, wu, wd), (sg, su, sd), keep)
        check_route(r_na, rr)
        e_ref = check_y(yn, ref, tol)
        say("  max|y_noalloc - y_workspace| / max|y_workspace| = %.3e, vs oracle %.3e" % (e_ws, e_ref))


def test_noalloc_zero_tokens_and_zero_budget():
    """T = 0 enqueues nothing; an all-zero budget gives exact zeros (no shared expert)."""
    import torch
    cfg = synth.LayerConfig("noalloc_zero", 65, T=16, d=128, E=4, I=64, top_k=2, I_shared=0, dtype=synth.BF16,
                            norm_topk=1, bias_std=0.5, w_std=0.05)
    (wg, wu, wd), _ = synth.make_layer_weights(cfg)
    layer = fm.Layer(cfg.d, cfg.E, cfg.I, cfg.top_k, 0, synth.BF16, 1, max_tokens=16)
    dev = [fm.to_device(a) for a in (wg, wu, wd)]
    x, lg = synth.make_tokens(cfg)
    y = torch.full((16, cfg.d), 3.0, dtype=torch.bfloat16, device="cuda")
    fm.flexmoe_layer_forward_noalloc(layer.desc, 0, fm.to_device(x), fm.to_device(lg), *dev, layer.keep,
                                     None, None, None, y)
    torch.cuda.synchronize()
    assert bool((y == 3.0).all())
    layer.set_budget(np.zeros(cfg.E, np.int32))
    fm.flexmoe_layer_forward_noalloc(layer.desc, 16, fm.to_device(x), fm.to_device(lg), *dev, layer.keep,
                                     None, None, None, y)
    torch.cuda.synchronize()
    assert bool((y == 0).all())
