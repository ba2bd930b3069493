"""Pins of the oracle's gradients and channel saliency (Sec. 3.1, Eq. 2).

The oracle writes the gradients of L = 1/2 sum_t ||y_t - y_target_t||^2 out
by the chain rule.  They are checked against things other than that
derivation: central finite differences of the (separately pinned) forward,
reverse-mode autodiff of an independent dense torch formulation, a 1-channel
case worked by hand, and properties the paper's saliency must have (channel
permutation equivariance, which is what makes the reorder of Eq. 3
meaningful; zero score for a channel that cannot affect the output; zero
score past the prefix of a masked expert).
"""
import math

import numpy as np
import pytest

import oracle
from tests.bruteforce import f64, random_layer, router_weights, topk_by_sort


def _loss(x, lg, wg, wu, wd, keep, k, norm, tgt, sh):
    y = oracle.layer_forward(x, lg, wg, wu, wd, keep, k, norm, *sh)
    return 0.5 * float(((y - tgt.astype(np.float64)) ** 2).sum())


CASES = [
    # T, d, E, I, k, I_s, norm, keep
    (5, 6, 3, 5, 2, 3, 1, None),
    (7, 4, 4, 6, 2, 0, 0, [6, 3, 0, 1]),
    (4, 5, 2, 4, 1, 2, 0, [2, 4]),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_grads_match_finite_differences(case):
    T, d, E, I, k, I_s, norm, keep = CASES[case]
    rng = np.random.default_rng(100 + case)
    x, lg, wg, wu, wd, sh = random_layer(rng, T, d, E, I, k, I_s)
    keep = np.array(keep if keep is not None else [I] * E, np.int32)
    tgt = rng.standard_normal((T, d)).astype(np.float32)
    L, gg, gu, gd = oracle.layer_grads(x, lg, wg, wu, wd, keep, k, norm, tgt, *sh)
    assert L == pytest.approx(_loss(x, lg, wg, wu, wd, keep, k, norm, tgt, sh), rel=1e-13)
    for W, G in ((wg, gg), (wu, gu), (wd, gd)):
        for flat in range(W.size):
            ix = np.unravel_index(flat, W.shape)
            h = np.float32(2.0 ** -13)
            Wp, Wm = W.copy(), W.copy()
            Wp[ix] = W[ix] + h
            Wm[ix] = W[ix] - h
            step = float(Wp[ix]) - float(Wm[ix])   # exact in fp64
            args = [wg, wu, wd]
            which = [wg is W, wu is W, wd is W].index(True)
            args[which] = Wp
            lp = _loss(x, lg, *args, keep, k, norm, tgt, sh)
            args[which] = Wm
            lm = _loss(x, lg, *args, keep, k, norm, tgt, sh)
            fd = (lp - lm) / step
            assert abs(fd - G[ix]) <= 2e-7 * max(1.0, abs(G[ix])), (which, ix, fd, G[ix])


def _torch_grads(x, lg, wg, wu, wd, keep, k, norm, tgt, sh):
    """Reverse-mode autodiff of a dense form of the layer: every expert on
    every token, the prefix mask by multiplication, a dense [T][E] gate."""
    import torch
    X = torch.tensor(f64(x))
    T, d = X.shape
    Wg = torch.tensor(f64(wg), requires_grad=True)
    Wu = torch.tensor(f64(wu), requires_grad=True)
    Wd = torch.tensor(f64(wd), requires_grad=True)
    E, I, _ = Wg.shape
    idx = topk_by_sort(lg, k)
    w = router_weights(lg, idx, norm)
    G = np.zeros((T, E))
    G[np.repeat(np.arange(T), k), idx.reshape(-1)] = w.reshape(-1)
    G = torch.tensor(G)
    Y = torch.zeros((T, d), dtype=torch.float64)
    for e in range(E):
        m = (torch.arange(I) < int(keep[e])).double()
        H = torch.nn.functional.silu(X @ Wg[e].T) * (X @ Wu[e].T) * m
        Y = Y + G[:, e:e + 1] * (H @ Wd[e].T)
    if sh[0] is not None:
        Sg, Su, Sd = (torch.tensor(f64(a)) for a in sh)
        Y = Y + (torch.nn.functional.silu(X @ Sg.T) * (X @ Su.T)) @ Sd.T
    L = 0.5 * ((Y - torch.tensor(f64(tgt))) ** 2).sum()
    L.backward()
    return float(L.detach()), Wg.grad.numpy(), Wu.grad.numpy(), Wd.grad.numpy()


@pytest.mark.parametrize("seed", range(4))
def test_grads_and_saliency_match_autodiff(seed):
    rng = np.random.default_rng(200 + seed)
    T, d, E, I, k, I_s = [(9, 8, 4, 7, 2, 5), (12, 6, 6, 9, 3, 0), (3, 10, 5, 4, 4, 6), (16, 8, 8, 8, 2, 8)][seed]
    norm = seed % 2
    x, lg, wg, wu, wd, sh = random_layer(rng, T, d, E, I, k, I_s, bf16=seed >= 2)
    keep = rng.integers(0, I + 1, size=E).astype(np.int32) if seed == 1 else np.full(E, I, np.int32)
    tgt = rng.standard_normal((T, d)).astype(np.float32)
    L, gg, gu, gd = oracle.layer_grads(x, lg, wg, wu, wd, keep, k, norm, tgt, *sh)
    Lt, tg, tu, td = _torch_grads(x, lg, wg, wu, wd, keep, k, norm, tgt, sh)
    assert L == pytest.approx(Lt, rel=1e-12)
    for a, b in ((gg, tg), (gu, tu), (gd, td)):
        np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)
    # Eq. 2 as a sum of squares over the channel's group, from the autodiff gradients
    s = oracle.channel_saliency_from_grads(wg, wu, wd, gg, gu, gd)
    Wg, Wu, Wd = f64(wg), f64(wu), f64(wd)
    want = ((Wg * tg) ** 2).sum(2) + ((Wu * tu) ** 2).sum(2) + ((Wd * td) ** 2).sum(1)
    np.testing.assert_allclose(s, want, rtol=1e-10, atol=1e-14)


def test_single_channel_worked_by_hand():
    # one token, one expert, one channel, d = 1: every quantity by hand
    x, wg, wu, wd, tgt = 0.5, 2.0, -1.5, 0.75, 0.25
    g, u = wg * x, wu * x                       # 1, -0.75
    sg = 1.0 / (1.0 + math.exp(-g))
    silu, dsilu = g * sg, sg * (1.0 + g * (1.0 - sg))
    h = silu * u
    y = wd * h
    dy = y - tgt
    g_wd, dh = dy * h, wd * dy
    g_wg, g_wu = dh * u * dsilu * x, dh * silu * x
    f = lambda v: np.array(v, np.float32)
    L, gg, gu, gd = oracle.layer_grads(f([[x]]), f([[0.0]]), f([[[wg]]]), f([[[wu]]]), f([[[wd]]]),
                                       np.array([1], np.int32), 1, 1, f([[tgt]]))
    assert L == pytest.approx(0.5 * dy * dy, rel=1e-14)
    assert gg[0, 0, 0] == pytest.approx(g_wg, rel=1e-14)
    assert gu[0, 0, 0] == pytest.approx(g_wu, rel=1e-14)
    assert gd[0, 0, 0] == pytest.approx(g_wd, rel=1e-14)
    s = oracle.channel_saliency_from_grads(f([[[wg]]]), f([[[wu]]]), f([[[wd]]]), gg, gu, gd)
    assert s[0, 0] == pytest.approx((wg * g_wg) ** 2 + (wu * g_wu) ** 2 + (wd * g_wd) ** 2, rel=1e-13)
    # the group's sum of squares differs from the square of its sum
    assert s[0, 0] != pytest.approx((wg * g_wg + wu * g_wu + wd * g_wd) ** 2, rel=1e-3)


def test_saliency_is_channel_permutation_equivariant():
    # reordering an expert's hidden channels (Eq. 3) leaves the layer unchanged,
    # so each channel's score moves with it
    rng = np.random.default_rng(7)
    T, d, E, I, k = 24, 8, 4, 12, 2
    x, lg, wg, wu, wd, sh = random_layer(rng, T, d, E, I, k, 6)
    batches = [(x, lg, rng.standard_normal((T, d)).astype(np.float32))]
    s = oracle.channel_saliency(batches, wg, wu, wd, k, 1, *sh)
    pi = np.stack([rng.permutation(I) for _ in range(E)])
    wg_p = np.stack([wg[e][pi[e]] for e in range(E)])
    wu_p = np.stack([wu[e][pi[e]] for e in range(E)])
    wd_p = np.stack([wd[e][:, pi[e]] for e in range(E)])
    s_p = oracle.channel_saliency(batches, wg_p, wu_p, wd_p, k, 1, *sh)
    np.testing.assert_allclose(s_p, np.stack([s[e][pi[e]] for e in range(E)]), rtol=1e-9, atol=1e-15)
    # and the rank of Eq. 3 from these scores puts the permuted channels back
    # in the same order (scores are distinct here)
    _, _, _, perm = oracle.rank_reorder(s.astype(np.float32), wg, wu, wd)
    _, _, _, perm_p = oracle.rank_reorder(s_p.astype(np.float32), wg_p, wu_p, wd_p)
    np.testing.assert_array_equal(np.stack([pi[e][perm_p[e]] for e in range(E)]), perm)


def test_saliency_zero_cases():
    rng = np.random.default_rng(11)
    T, d, E, I, k = 10, 6, 5, 7, 2
    x, lg, wg, wu, wd, sh = random_layer(rng, T, d, E, I, k, 0)
    lg[:, 4] = -30.0          # expert 4 receives no token
    wd[1][:, 3] = 0.0         # channel 3 of expert 1 cannot reach the output
    tgt = rng.standard_normal((T, d)).astype(np.float32)
    s = oracle.channel_saliency([(x, lg, tgt)], wg, wu, wd, k, 0)
    assert np.all(s[4] == 0.0)
    assert s[1, 3] == 0.0
    assert np.all(s[:4][np.arange(4) != 4] >= 0.0)
    # a masked expert: channels past its prefix take no part and get no gradient
    keep = np.array([7, 3, 0, 5, 7], np.int32)
    _, gg, gu, gd = oracle.layer_grads(x, lg, wg, wu, wd, keep, k, 0, tgt)
    sm = oracle.channel_saliency_from_grads(wg, wu, wd, gg, gu, gd)
    for e in range(E):
        assert np.all(sm[e, keep[e]:] == 0.0)
    # the ranking set average is the mean of the per-batch scores
    b2 = (x[::-1].copy(), lg[::-1].copy(), tgt * 0.5)
    s2 = oracle.channel_saliency([b2], wg, wu, wd, k, 0)
    np.testing.assert_allclose(oracle.channel_saliency([(x, lg, tgt), b2], wg, wu, wd, k, 0), (s + s2) / 2,
                               rtol=1e-14, atol=0)
