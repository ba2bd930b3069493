"""Action learning on the device (Sec. 3.2, Eqs. 5-8) against the oracle.

One training step of a layer's per-expert width actions through the C ABI:
the hard Gumbel-softmax sample (bit-exact: the same fp32 argmax), the
sampled subnet's forward, the backward for an upstream gradient (input,
router-logit and mask gradients) and the action-logit gradient with the
cost and entropy terms.

Tolerances: the forward as for the inference path (2e-2 of max|ref|, bf16
operands, fp32 accumulation).  The backward rounds its MFMA operands (dO,
g, u, dG, dU) to bf16 once each, like the forward's h: 2e-2 of the largest
reference magnitude of each output (per expert for the mask gradient).  The
action-logit gradient from a given mask gradient is fp32 arithmetic on
E*K values: 1e-4 relative.
"""
import numpy as np
import pytest

import oracle
from paper_2606_27866_amd import flexmoe as fm
from paper_2606_27866_amd import synth
from tests.gpu_util import BF16_TOL, check_y, mini_layer, say

RATIOS = synth.ACTION_RATIOS
BWD_TOL = 2e-2


def test_action_api_rejects_bad_arguments_on_host():
    f32 = fm.make_desc(64, 4, 64, 2, 0, fm.FLEXMOE_F32, 1, 16)
    bf = fm.make_desc(64, 4, 64, 2, 0, fm.FLEXMOE_BF16, 1, 16)
    cases = [
        (lambda: fm.flexmoe_sample_actions(f32, fm.make_actions(RATIOS), 0x1000, 0x1000, 0x1000, stream=0), -5),
        (lambda: fm.flexmoe_sample_actions(bf, fm.make_actions([0.5, 0.0]), 0x1000, 0x1000, 0x1000, stream=0), -1),
        (lambda: fm.flexmoe_sample_actions(bf, fm.make_actions([0.5, 1.5]), 0x1000, 0x1000, 0x1000, stream=0), -1),
        (lambda: fm.flexmoe_sample_actions(bf, fm.make_actions([]), 0x1000, 0x1000, 0x1000, stream=0), -1),
        (lambda: fm.flexmoe_action_grad(bf, 8, fm.make_actions(RATIOS), 0x1000, 0x1000, 0.0, 0.1, 0.1, 0x1000,
                                        0x1000, None, 0x1000, workspace_bytes=1 << 30, stream=0), -1),
        (lambda: fm.flexmoe_train_forward(bf, 16, *([0x1000] * 6), None, None, None, 0x1000, 0x1000,
                                          workspace_bytes=256, stream=0), -4),
        (lambda: fm.flexmoe_train_backward(bf, 17, *([0x1000] * 5), None, None, None, 0x1000, 0x1000, 0x1000,
                                           0x1000, workspace_bytes=1 << 30, stream=0), -2),
    ]
    for f, code in cases:
        with pytest.raises(fm.FlexMoEError) as ei:
            f()
        assert ei.value.code == code
    assert fm.flexmoe_train_workspace_bytes(bf, 0) < fm.flexmoe_train_workspace_bytes(bf, 16)


def check_max(a, ref, tol, what):
    a = np.asarray(a, np.float64)
    scale = np.abs(ref).max()
    err = np.abs(a - ref).max() if a.size else 0.0
    assert err <= tol * max(scale, 1e-30), "%s: max|err| %.3e > %.1e * %.3e" % (what, err, tol, scale)
    return err / max(scale, 1e-30)


CASES = [
    # name, T, d, E, I, k, I_s, norm
    ("a_small", 60, 64, 8, 96, 2, 32, 1),        # one-workgroup dispatch, ragged tiles
    ("a_ragged", 600, 256, 16, 200, 4, 128, 0),  # routing kernels, I % 256 != 0, narrow actions
    ("a_tiles", 1100, 520, 8, 264, 2, 0, 1),     # two row tiles per expert, d % 256 != 0, no shared expert
]


@pytest.mark.gpu
@pytest.mark.parametrize("spec", CASES, ids=[c[0] for c in CASES])
def test_gpu_action_step_matches_oracle(spec):
    import torch
    name, T, d, E, I, k, I_s, norm = spec
    cid = 190 + CASES.index(spec)
    cfg, x, lg, w, s = mini_layer(name, T, d, E, I, k, I_s, norm=norm, config_id=cid)
    alpha, gumbel = synth.make_action_inputs(cfg, len(RATIOS))
    tau, lam, beta = 0.8, 0.3, 0.05
    tgt = synth.make_target(cfg, T)

    layer = fm.Layer(d, E, I, k, I_s, synth.BF16, norm, max_tokens=T)
    layer.set_weights(*[fm.to_device(a) if a is not None else None for a in (*w, *s)])
    # the middle case runs in a workspace sized for more tokens than the step has
    learner = fm.ActionLearner(layer, T + (37 if CASES.index(spec) == 1 else 0), RATIOS)
    say(name, "T", T, "d", d, "E", E, "I", I, "k", k, "I_s", I_s)
    learner.transpose_weights()
    ad, gd = fm.to_device(alpha), fm.to_device(gumbel)
    learner.sample(ad, gd)
    torch.cuda.synchronize()
    keep_ref, act_ref, _ = oracle.sample_actions(RATIOS, I, alpha, gumbel, tau)
    np.testing.assert_array_equal(learner.keep.cpu().numpy(), keep_ref)
    np.testing.assert_array_equal(learner.action.cpu().numpy(), act_ref)

    xd, ld = fm.to_device(x), fm.to_device(lg)
    y = learner.forward(xd, ld)
    torch.cuda.synchronize()
    y_ref = oracle.layer_forward(x, lg, *w, keep_ref, k, norm, *s)
    check_y(synth.bf16_bits_to_f32(fm.to_host(y)).astype(np.float64), y_ref, BF16_TOL)

    dy = (y_ref - tgt).astype(np.float32)   # the quality loss's upstream gradient, same on both sides
    dx, dl, dm = learner.backward(ld, fm.to_device(dy))
    torch.cuda.synchronize()
    dx_ref, dl_ref, dm_ref = oracle.masked_backward(x, lg, *w, keep_ref, k, norm, dy, *s)
    ex = check_max(dx.cpu().numpy(), dx_ref, BWD_TOL, "dx")
    el = check_max(dl.cpu().numpy(), dl_ref, BWD_TOL, "dlogits")
    dmh = dm.cpu().numpy()
    em = max(check_max(dmh[e], dm_ref[e], BWD_TOL, "dmask[%d]" % e) for e in range(E) if np.abs(dm_ref[e]).max() > 0)
    say(name, "rel err dx %.2e dlogits %.2e dmask %.2e" % (ex, el, em))

    # repeated backward: the same bits
    dx2, dl2, dm2 = learner.backward(ld, fm.to_device(dy))
    torch.cuda.synchronize()
    for a, b in ((dx, dx2), (dl, dl2), (dm, dm2)):
        np.testing.assert_array_equal(a.cpu().numpy(), b.cpu().numpy())

    dalpha, stats = learner.action_grad(ad, gd, tau, lam, beta, dm)
    torch.cuda.synchronize()
    counts = np.bincount(oracle.route(lg, k, norm)[0].reshape(-1), minlength=E).astype(np.int32)
    # the action-logit gradient from the device's own mask gradient
    da_ref, C, H = oracle.action_grad(RATIOS, I, alpha, gumbel, tau, dmh.astype(np.float64), counts, T * k, lam,
                                      beta)
    np.testing.assert_allclose(dalpha.cpu().numpy(), da_ref, rtol=1e-4, atol=1e-5 * np.abs(da_ref).max())
    st = stats.cpu().numpy()
    assert st[0] == pytest.approx(C, rel=1e-5)
    assert st[1] == pytest.approx(H, rel=1e-5)
    # end to end against the oracle's own mask gradient
    da_full, _, _ = oracle.action_grad(RATIOS, I, alpha, gumbel, tau, dm_ref, counts, T * k, lam, beta)
    check_max(dalpha.cpu().numpy(), da_full, BWD_TOL, "dalpha")


@pytest.mark.gpu
def test_gpu_zero_width_expert_is_skipped():
    """A keep table with k_e = 0 (not produced by the action sets, allowed by
    the forward): the expert adds nothing and gets no mask gradient."""
    import torch
    T, d, E, I, k = 200, 128, 6, 64, 2
    cfg, x, lg, w, s = mini_layer("a_zero", T, d, E, I, k, 0, norm=0, config_id=199)
    keep = np.array([64, 0, 7, 64, 0, 33], np.int32)
    layer = fm.Layer(d, E, I, k, 0, synth.BF16, 0, max_tokens=T)
    layer.set_weights(*[fm.to_device(a) for a in w])
    learner = fm.ActionLearner(layer, T, RATIOS)
    learner.transpose_weights()
    kd = fm.to_device(keep)
    xd, ld = fm.to_device(x), fm.to_device(lg)
    say("zero-width experts", keep.tolist())
    y = learner.forward(xd, ld, keep=kd)
    y_ref = oracle.layer_forward(x, lg, *w, keep, k, 0)
    dy = (y_ref - synth.make_target(cfg, T)).astype(np.float32)
    dx, dl, dm = learner.backward(ld, fm.to_device(dy))
    torch.cuda.synchronize()
    check_y(synth.bf16_bits_to_f32(fm.to_host(y)).astype(np.float64), y_ref, BF16_TOL)
    dx_ref, dl_ref, dm_ref = oracle.masked_backward(x, lg, *w, keep, k, 0, dy)
    check_max(dx.cpu().numpy(), dx_ref, BWD_TOL, "dx")
    check_max(dl.cpu().numpy(), dl_ref, BWD_TOL, "dlogits")
    dmh = dm.cpu().numpy()
    assert np.all(dmh[1] == 0) and np.all(dmh[4] == 0)
    for e in (0, 2, 3, 5):
        check_max(dmh[e], dm_ref[e], BWD_TOL, "dmask[%d]" % e)
