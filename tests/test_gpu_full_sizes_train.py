"""Saliency and action learning at the full size of the Qwen1.5-MoE-shaped
workload (T = 4096, d = 2048, E = 60, I = 1408, top-4, shared 5632), in the
launch configuration bench.py times, on outputs the oracle can compute on a
sub-batch:
  - a token's input and router-logit gradients depend on that token alone;
  - expert e's saliency scores and mask gradient depend only on the tokens
    routed to e (their upstream gradients depend on each token alone),
so the oracle runs on sampled tokens, or on the tokens of sampled experts,
with the full weights.  Tolerances as in the small-size tests.
"""
import functools

import numpy as np
import pytest

import oracle
from paper_2606_27866_amd import flexmoe as fm
from paper_2606_27866_amd import synth
from tests.gpu_util import BF16_TOL, check_y, say

pytestmark = pytest.mark.gpu
NAME = "qwen15_moe_a27b"


@functools.lru_cache(maxsize=1)
def inputs():
    cfg = synth.CONFIGS[NAME]
    say("generating", NAME)
    w = synth.make_expert_weights(cfg)
    s = synth.make_shared_weights(cfg)
    x, lg = synth.make_calibration_batch(cfg, 0)
    return cfg, w, s, x, lg


@functools.lru_cache(maxsize=1)
def device_layer():
    cfg, w, s, _, _ = inputs()
    layer = fm.Layer(cfg.d, cfg.E, cfg.I, cfg.top_k, cfg.I_shared, cfg.dtype, cfg.norm_topk, cfg.T)
    layer.set_weights(*[fm.to_device(a) for a in (*w, *s)])
    return layer


def sampled_experts(idx, E):
    n = np.bincount(idx.reshape(-1), minlength=E)
    order = np.argsort(n, kind="stable")
    return [int(order[-1]), int(order[len(order) // 2]), int(order[0])]   # most, median, fewest tokens


def tokens_of(idx, e):
    return np.nonzero((idx == e).any(axis=1))[0]


def test_full_size_saliency_sampled_experts():
    import torch
    cfg, w, s, x, lg = inputs()
    layer = device_layer()
    tgt = synth.make_target(cfg)
    sal = fm.Saliency(layer, cfg.T)
    say(NAME, "saliency, T", cfg.T)
    sal.add_batch(fm.to_device(x), fm.to_device(lg), fm.to_device(tgt))
    torch.cuda.synchronize()
    scores = sal.scores.cpu().numpy()
    idx, _ = oracle.route(lg, cfg.top_k, cfg.norm_topk)
    for e in sampled_experts(idx, cfg.E):
        tok = tokens_of(idx, e)
        say("expert", e, "tokens", len(tok))
        ref = oracle.channel_saliency([(x[tok], lg[tok], tgt[tok])], *w, cfg.top_k, cfg.norm_topk, *s)[e]
        err = np.abs(scores[e] - ref)
        assert np.all(err <= 3e-2 * ref + 1e-4 * ref.max()), (e, float((err / np.maximum(ref, 1e-30)).max()))


def test_full_size_action_step_sampled():
    import torch
    cfg, w, s, x, lg = inputs()
    layer = device_layer()
    ratios = synth.ACTION_RATIOS
    alpha, gumbel = synth.make_action_inputs(cfg, len(ratios))
    learner = fm.ActionLearner(layer, cfg.T, ratios)
    learner.transpose_weights()
    ad, gd = fm.to_device(alpha), fm.to_device(gumbel)
    say(NAME, "action step, T", cfg.T)
    learner.sample(ad, gd)
    xd, ld = fm.to_device(x), fm.to_device(lg)
    y = learner.forward(xd, ld)
    dy = synth.make_target(cfg, std=1e-3)    # an upstream gradient dL/dY
    dx, dl, dm = learner.backward(ld, fm.to_device(dy))
    torch.cuda.synchronize()
    keep = learner.keep.cpu().numpy()
    keep_ref, _, _ = oracle.sample_actions(ratios, cfg.I, alpha, gumbel, 1.0)
    np.testing.assert_array_equal(keep, keep_ref)
    yh = synth.bf16_bits_to_f32(fm.to_host(y)).astype(np.float64)
    dxh, dlh, dmh = dx.cpu().numpy(), dl.cpu().numpy(), dm.cpu().numpy()
    rows = np.random.default_rng(1).choice(cfg.T, 24, replace=False)
    y_ref = oracle.layer_forward(x[rows], lg[rows], *w, keep, cfg.top_k, cfg.norm_topk, *s)
    check_y(yh[rows], y_ref, BF16_TOL)
    dx_ref, dl_ref, _ = oracle.masked_backward(x[rows], lg[rows], *w, keep, cfg.top_k, cfg.norm_topk, dy[rows], *s)
    check_y(dxh[rows].astype(np.float64), dx_ref, 2e-2)
    check_y(dlh[rows].astype(np.float64), dl_ref, 2e-2)
    idx, _ = oracle.route(lg, cfg.top_k, cfg.norm_topk)
    for e in sampled_experts(idx, cfg.E):
        tok = tokens_of(idx, e)
        _, _, dm_ref = oracle.masked_backward(x[tok], lg[tok], *w, keep, cfg.top_k, cfg.norm_topk, dy[tok], *s)
        say("expert", e, "tokens", len(tok), "keep", int(keep[e]))
        check_y(dmh[e].astype(np.float64), dm_ref[e], 2e-2)
