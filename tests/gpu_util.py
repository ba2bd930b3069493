"""Helpers of the GPU parity tests: run the HIP path through the C ABI and
the oracle on the same seeded inputs, and compare."""
import sys

import numpy as np

import oracle
from paper_2606_27866_amd import flexmoe as fm
from paper_2606_27866_amd import synth

BF16_TOL = 2e-2     # max|y - ref| <= 2e-2 * max|ref|   (bf16 inputs, fp32 accumulation)
F32_TOL = 1e-5      # max|y - ref| <= 1e-5 * max|ref|   (fp32 mode, fp64 oracle)
W_TOL = 1e-6        # router weights, absolute


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def y_to_f64(y_host):
    return synth.bf16_bits_to_f32(y_host).astype(np.float64) if y_host.dtype == np.uint16 \
        else y_host.astype(np.float64)


class GpuLayer:
    """Weights uploaded once; forward through flexmoe_layer_forward."""

    def __init__(self, d, E, I, top_k, I_shared, dtype, norm_topk, max_tokens, wg, wu, wd,
                 sg=None, su=None, sd=None):
        import torch
        self.torch = torch
        self.layer = fm.Layer(d, E, I, top_k, I_shared, dtype, norm_topk, max_tokens)
        dev = [fm.to_device(a) if a is not None else None for a in (wg, wu, wd, sg, su, sd)]
        self.layer.set_weights(*dev)
        self.E, self.top_k, self.d = E, top_k, d

    def forward(self, x, logits, keep, with_route=True):
        torch = self.torch
        T = x.shape[0]
        self.layer.set_budget(np.asarray(keep, np.int32))
        xd = fm.to_device(x)
        ld = fm.to_device(np.ascontiguousarray(logits, np.float32))
        A = max(T * self.top_k, 1)
        dbg = None
        if with_route:
            i32 = dict(dtype=torch.int32, device="cuda")
            dbg = dict(topk_idx=torch.full((A,), -7, **i32),
                       topk_w=torch.full((A,), -7.0, dtype=torch.float32, device="cuda"),
                       counts=torch.full((self.E,), -7, **i32),
                       offsets=torch.full((self.E + 1,), -7, **i32),
                       perm=torch.full((A,), -7, **i32), pos=torch.full((A,), -7, **i32))
        y = self.layer.forward(xd, ld, dbg=dbg)
        torch.cuda.synchronize()
        out = y_to_f64(fm.to_host(y))
        if not with_route:
            return out, None
        r = {k: v.cpu().numpy() for k, v in dbg.items()}
        r["topk_idx"] = r["topk_idx"][:T * self.top_k].reshape(T, self.top_k)
        r["topk_w"] = r["topk_w"][:T * self.top_k].reshape(T, self.top_k)
        r["pos"] = r["pos"][:T * self.top_k]
        P = int(r["offsets"][-1]) if T > 0 else 0
        r["perm"] = r["perm"][:P]
        return out, r


def check_route(r, ref):
    np.testing.assert_array_equal(r["topk_idx"], ref["idx"])
    np.testing.assert_allclose(r["topk_w"], ref["w"], rtol=0, atol=W_TOL)
    np.testing.assert_array_equal(r["counts"], ref["counts"])
    np.testing.assert_array_equal(r["offsets"], ref["offsets"])
    np.testing.assert_array_equal(r["perm"], ref["perm"])
    np.testing.assert_array_equal(r["pos"], ref["pos"])


def check_y(y, ref, tol):
    scale = np.abs(ref).max()
    err = np.abs(y - ref).max() if y.size else 0.0
    assert err <= tol * max(scale, 1e-30), "max|err| = %.3e > %.1e * max|ref| (%.3e)" % (err, tol, scale)
    return err / max(scale, 1e-30)


def mini_layer(name, T, d, E, I, k, I_s=0, dtype=synth.BF16, norm=1, config_id=60, bias_std=0.5,
               w_std=0.05):
    cfg = synth.LayerConfig(name, config_id, T=T, d=d, E=E, I=I, top_k=k, I_shared=I_s,
                            dtype=dtype, norm_topk=norm, bias_std=bias_std, w_std=w_std)
    x, lg = synth.make_tokens(cfg)
    wg, wu, wd = synth.make_expert_weights(cfg)
    sg, su, sd = synth.make_shared_weights(cfg)
    return cfg, x, lg, (wg, wu, wd), (sg, su, sd)


def oracle_ref(cfg, x, lg, w, s, keep):
    return oracle.layer_forward(x, lg, *w, keep, cfg.top_k, cfg.norm_topk, *s, want_route=True)
