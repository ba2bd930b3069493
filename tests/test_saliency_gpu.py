"""Channel saliency on the device (Sec. 3.1, Eq. 2) against the oracle.

The HIP path (forward keeping g, u, h; dgrad with the SwiGLU backward; wgrad
GEMMs reducing (theta * g)^2 per channel) is compared score by score with the
oracle's fp64 chain-rule gradients on the same seeded inputs.  Then the
device rank/reorder of Eq. 3 is run on the device scores and must equal the
oracle's reorder of those same scores bit for bit.

Tolerance of a score (bf16 operands, fp32 accumulation): every gradient entry
is a sum of products of operands rounded once or twice to bf16 (relative
error <= 2^-9 each, so <= ~4 * 2^-9 per product); a score is a sum of squares
of theta * g, which doubles the relative error of a coherent error: <= 1.6 %.
The test allows 3 % of the score plus 1e-4 of the expert's largest score
(entries whose gradient is dominated by cancellation).
"""
import numpy as np
import pytest

import oracle
from paper_2606_27866_amd import flexmoe as fm
from paper_2606_27866_amd import synth
from tests.gpu_util import mini_layer, say

REL_TOL = 3e-2
ABS_TOL = 1e-4   # times the expert's largest score


def test_saliency_rejects_bad_arguments_on_host():
    f32 = fm.make_desc(64, 4, 64, 2, 0, fm.FLEXMOE_F32, 1, 16)
    with pytest.raises(fm.FlexMoEError) as ei:
        fm.flexmoe_channel_saliency(f32, 4, *([0x1000] * 9), 0x1000, 1.0, 0x1000, 0x1000,
                                    workspace_bytes=1 << 30, stream=0)
    assert ei.value.code == -5
    bf = fm.make_desc(64, 4, 64, 2, 0, fm.FLEXMOE_BF16, 1, 16)
    with pytest.raises(fm.FlexMoEError) as ei:  # T above max_tokens
        fm.flexmoe_channel_saliency(bf, 17, *([0x1000] * 5), None, None, None, None, 0x1000, 1.0, 0x1000, 0x1000,
                                    workspace_bytes=1 << 30, stream=0)
    assert ei.value.code == -2
    with pytest.raises(fm.FlexMoEError) as ei:  # workspace too small
        fm.flexmoe_channel_saliency(bf, 16, *([0x1000] * 5), None, None, None, None, 0x1000, 1.0, 0x1000, 0x1000,
                                    workspace_bytes=256, stream=0)
    assert ei.value.code == -4
    with pytest.raises(fm.FlexMoEError) as ei:  # shared weights without a shared expert
        fm.flexmoe_channel_saliency(bf, 16, *([0x1000] * 9), 0x1000, 1.0, 0x1000, 0x1000,
                                    workspace_bytes=1 << 30, stream=0)
    assert ei.value.code == -1
    # the workspace grows with T and T = 0 needs only the fixed part
    assert fm.flexmoe_saliency_workspace_bytes(bf, 0) < fm.flexmoe_saliency_workspace_bytes(bf, 16)


def check_scores(s_gpu, s_ref):
    s_gpu = np.asarray(s_gpu, np.float64)
    top = s_ref.max(axis=1, keepdims=True)
    err = np.abs(s_gpu - s_ref)
    bound = REL_TOL * s_ref + ABS_TOL * top
    bad = err > bound
    assert not bad.any(), "score %s: gpu %.6e ref %.6e (%d bad of %d)" % (
        np.argwhere(bad)[0], s_gpu[bad][0], s_ref[bad][0], bad.sum(), bad.size)
    rel = err / np.maximum(s_ref, 1e-300)
    return float(np.median(rel)), float(rel.max())


CASES = [
    # name, T, d, E, I, k, I_s, norm, dead expert
    ("s_small", 60, 64, 8, 96, 2, 32, 1, 3),        # one-workgroup dispatch, ragged tiles, an expert with no token
    ("s_ragged", 600, 256, 16, 200, 4, 128, 0, -1),  # routing kernels (T*k > 1024), I % 256 != 0
    ("s_tiles", 1100, 520, 8, 264, 2, 0, 1, -1),     # two row tiles per expert, d % 256 != 0
]


@pytest.mark.gpu
@pytest.mark.parametrize("spec", CASES, ids=[c[0] for c in CASES])
def test_gpu_saliency_and_rank_match_oracle(spec):
    import torch
    name, T, d, E, I, k, I_s, norm, dead = spec
    cid = 170 + CASES.index(spec)
    cfg, x, lg, w, s = mini_layer(name, T, d, E, I, k, I_s, norm=norm, config_id=cid)
    if dead >= 0:
        lg = lg.copy()
        lg[:, dead] = -100.0
    tgt = synth.make_target(cfg, T)
    x2, lg2 = synth.make_calibration_batch(cfg, 0, T)
    tgt2 = synth.make_target(cfg, T, batch=0)

    layer = fm.Layer(d, E, I, k, I_s, synth.BF16, norm, max_tokens=T)
    layer.set_weights(*[fm.to_device(a) if a is not None else None for a in (*w, *s)])
    # the first case makes W_down^T inside every call, the others once up front
    # (and the middle case sizes its workspace for more tokens than a batch has)
    sal = fm.Saliency(layer, T + (37 if CASES.index(spec) == 1 else 0), transpose_once=CASES.index(spec) > 0)
    say(name, "T", T, "d", d, "E", E, "I", I, "k", k, "I_s", I_s)
    dev = [fm.to_device(a) for a in (x, lg, tgt, x2, lg2, tgt2)]
    sal.add_batch(dev[0], dev[1], dev[2])
    torch.cuda.synchronize()
    s1 = sal.scores.cpu().numpy().copy()
    ref1 = oracle.channel_saliency([(x, lg, tgt)], *w, k, norm, *s)
    med, mx = check_scores(s1, ref1)
    say(name, "one batch: median rel err %.2e, max %.2e" % (med, mx))
    if dead >= 0:
        assert np.all(s1[dead] == 0.0)

    # repeated call: the same bits (fixed summation order)
    sal.scores.zero_()
    sal.add_batch(dev[0], dev[1], dev[2])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sal.scores.cpu().numpy(), s1)

    # a two-batch ranking set with scale 1/2: the mean of Eq. 2
    sal.scores.zero_()
    sal.add_batch(dev[0], dev[1], dev[2], scale=0.5)
    sal.add_batch(dev[3], dev[4], dev[5], scale=0.5)
    torch.cuda.synchronize()
    s2 = sal.scores.cpu().numpy().copy()
    ref2 = oracle.channel_saliency([(x, lg, tgt), (x2, lg2, tgt2)], *w, k, norm, *s)
    check_scores(s2, ref2)

    # Eq. 3 on the device scores: the same permutation and weights as the
    # oracle's reorder of the same fp32 scores
    wg_r, wu_r, wd_r, perm = sal.rank_reorder()
    torch.cuda.synchronize()
    og, ou, od, operm = oracle.rank_reorder(s2, *w)
    np.testing.assert_array_equal(perm.cpu().numpy(), operm)
    for a, b in ((wg_r, og), (wu_r, ou), (wd_r, od)):
        np.testing.assert_array_equal(fm.to_host(a), b)


@pytest.mark.gpu
def test_gpu_saliency_finds_planted_channels():
    """Channels whose down column is scaled up carry more of the output and
    must rank first; channels with a zero down column score exactly 0 and
    rank last."""
    import torch
    T, d, E, I, k = 512, 128, 4, 64, 2
    cfg, x, lg, w, s = mini_layer("s_planted", T, d, E, I, k, 0, norm=1, config_id=180)
    wg, wu, wd = w
    wd = synth.bf16_bits_to_f32(wd).copy()
    rng = np.random.default_rng(5)
    strong = np.stack([rng.choice(I, 4, replace=False) for _ in range(E)])
    dead = np.stack([np.setdiff1d(rng.permutation(I), strong[e])[:3] for e in range(E)])
    for e in range(E):
        wd[e][:, strong[e]] *= 8.0
        wd[e][:, dead[e]] = 0.0
    wd = synth.f32_to_bf16_bits(wd)
    tgt = synth.make_target(cfg, T)
    layer = fm.Layer(d, E, I, k, 0, synth.BF16, 1, max_tokens=T)
    layer.set_weights(*[fm.to_device(a) for a in (wg, wu, wd)])
    sal = fm.Saliency(layer, T)
    say("planted", T, d, E, I, k)
    sal.add_batch(fm.to_device(x), fm.to_device(lg), fm.to_device(tgt))
    _, _, _, perm = sal.rank_reorder()
    torch.cuda.synchronize()
    perm = perm.cpu().numpy()
    scores = sal.scores.cpu().numpy()
    for e in range(E):
        assert set(perm[e][:4]) == set(strong[e])
        assert set(perm[e][-3:]) == set(dead[e])
        assert np.all(scores[e][dead[e]] == 0.0)
