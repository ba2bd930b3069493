"""Pins of the oracle's action learning (Sec. 3.2, Eqs. 5-8).

The oracle writes the straight-through Gumbel-softmax sample, the masked
layer's backward and the action-logit gradient out by hand.  They are
checked against reverse-mode autodiff (torch, fp64) of an independent dense
formulation that builds the whole chain the paper describes -- action
logits -> soft and hard samples -> straight-through estimator -> prefix mask
mixture -> masked layer -> squared-error quality loss + load-weighted cost -
entropy -- and differentiates it with respect to the layer input, the router
logits, the mask and the action logits; against NumPy/SciPy for the sample
itself; and against central finite differences for the input gradient.
"""
import numpy as np
import pytest
from scipy.special import softmax

import oracle
from tests.bruteforce import f64, random_layer, topk_by_sort

RATIOS = (0.1, 0.4, 0.7, 1.0)


def test_sample_matches_numpy():
    rng = np.random.default_rng(3)
    E, K, I = 40, 4, 96
    alpha = rng.standard_normal((E, K)).astype(np.float32)
    g = rng.gumbel(size=(E, K)).astype(np.float32)
    # ties: equal sums in a few experts must pick the lower action index
    alpha[5] = [0.5, 0.25, 0.5, 0.0]
    g[5] = [0.0, 0.25, 0.0, 0.5]
    tau = 0.7
    keep, act, zs = oracle.sample_actions(RATIOS, I, alpha, g, tau)
    s32 = alpha + g
    np.testing.assert_array_equal(act, np.argmax(s32, axis=1))
    assert act[5] == 0
    np.testing.assert_allclose(zs, softmax((alpha.astype(np.float64) + g) / tau, axis=1), rtol=1e-13)
    widths = [int(np.ceil(r * I - 1e-9)) for r in RATIOS]
    np.testing.assert_array_equal(keep, [widths[a] for a in act])


def _torch_chain(x, lg, wg, wu, wd, sh, k, norm, ratios, alpha, gumbel, tau, dy, lam, beta):
    """Dense autodiff of Eqs. 5-8 around the masked layer.  The quality term
    is <dy, Y> (its gradient with respect to Y is exactly dy, the upstream
    gradient the oracle's backward takes)."""
    import torch
    t = lambda a: torch.tensor(f64(a))
    X = t(x).requires_grad_(True)
    L = torch.tensor(np.asarray(lg, np.float64), requires_grad=True)
    Wg, Wu, Wd = t(wg), t(wu), t(wd)
    E, I, _ = Wg.shape
    T, d = X.shape
    A = torch.tensor(np.asarray(alpha, np.float64), requires_grad=True)
    G = torch.tensor(np.asarray(gumbel, np.float64))
    zsoft = torch.softmax((A + G) / tau, dim=1)
    hard = torch.zeros_like(zsoft)
    hard[torch.arange(E), torch.tensor(np.argmax(np.asarray(alpha, np.float32) + gumbel, axis=1))] = 1.0
    zt = hard - zsoft.detach() + zsoft                       # straight-through (Eq. 6)
    widths = [int(np.ceil(r * I - 1e-9)) for r in ratios]
    pref = torch.stack([(torch.arange(I) < w).double() for w in widths])   # m(r_k) [K][I]
    M = zt @ pref                                            # [E][I]
    M.retain_grad()
    idx = topk_by_sort(lg, k)
    P = torch.softmax(L, dim=1)
    rows = torch.arange(T).repeat_interleave(k)
    w = P[rows, torch.tensor(idx.reshape(-1), dtype=torch.long)].reshape(T, k)
    if norm:
        w = w / w.sum(1, keepdim=True)
    Y = torch.zeros((T, d), dtype=torch.float64)
    for j in range(k):
        for e in range(E):
            sel = torch.tensor(idx[:, j] == e)
            if not sel.any():
                continue
            H = torch.nn.functional.silu(X[sel] @ Wg[e].T) * (X[sel] @ Wu[e].T) * M[e]
            Y = Y.index_add(0, torch.nonzero(sel)[:, 0], w[sel, j:j + 1] * (H @ Wd[e].T))
    if sh[0] is not None:
        Sg, Su, Sd = (t(a) for a in sh)
        Y = Y + (torch.nn.functional.silu(X @ Sg.T) * (X @ Su.T)) @ Sd.T
    Lq = (Y * torch.tensor(np.asarray(dy, np.float64))).sum()
    counts = np.bincount(idx.reshape(-1), minlength=E)
    q = torch.tensor(counts / (T * k))
    p = torch.softmax(A, dim=1)
    r = torch.tensor(np.asarray(ratios, np.float64))
    C = (q * (p * r).sum(1)).sum()
    Hn = (-(p * torch.log(p)).sum(1)).mean()
    (Lq + lam * C - beta * Hn).backward()
    return (Y.detach().numpy(), Lq.item(), X.grad.numpy(), L.grad.numpy(), M.grad.numpy(), A.grad.numpy(),
            C.item(), Hn.item(), counts)


CASES = [
    # T, d, E, I, k, I_s, norm, bf16
    (12, 8, 4, 10, 2, 6, 1, False),
    (20, 6, 6, 12, 3, 0, 0, False),
    (9, 16, 5, 20, 2, 8, 0, True),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_backward_and_action_grad_match_autodiff(case):
    T, d, E, I, k, I_s, norm, bf16 = CASES[case]
    rng = np.random.default_rng(40 + case)
    x, lg, wg, wu, wd, sh = random_layer(rng, T, d, E, I, k, I_s, bf16=bf16)
    alpha = rng.standard_normal((E, len(RATIOS))).astype(np.float32)
    gumbel = rng.gumbel(size=alpha.shape).astype(np.float32)
    tau, lam, beta = 0.8, 0.3, 0.05
    tgt = rng.standard_normal((T, d)).astype(np.float32)
    keep, act, zs = oracle.sample_actions(RATIOS, I, alpha, gumbel, tau)
    y = oracle.layer_forward(x, lg, wg, wu, wd, keep, k, norm, *sh)
    dy = (y - tgt).astype(np.float32)       # the quality loss's upstream gradient
    dx, dl, dm = oracle.masked_backward(x, lg, wg, wu, wd, keep, k, norm, dy, *sh)
    counts = np.bincount(topk_by_sort(lg, k).reshape(-1), minlength=E).astype(np.int32)
    da, C, H = oracle.action_grad(RATIOS, I, alpha, gumbel, tau, dm, counts, T * k, lam, beta)
    Yt, Lq, tdx, tdl, tdm, tda, tC, tH, _ = _torch_chain(x, lg, wg, wu, wd, sh, k, norm, RATIOS, alpha,
                                                          gumbel, tau, dy, lam, beta)
    np.testing.assert_allclose(y, Yt, rtol=1e-12, atol=1e-14)
    for a, b in ((dx, tdx), (dl, tdl), (dm, tdm), (da, tda)):
        np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-13 * max(1.0, np.abs(b).max()))
    assert C == pytest.approx(tC, rel=1e-13)
    assert H == pytest.approx(tH, rel=1e-13)


def test_input_gradient_matches_finite_differences():
    T, d, E, I, k, I_s = 6, 5, 3, 7, 2, 4
    rng = np.random.default_rng(9)
    x, lg, wg, wu, wd, sh = random_layer(rng, T, d, E, I, k, I_s)
    keep = np.array([7, 3, 1], np.int32)
    tgt = rng.standard_normal((T, d)).astype(np.float32)
    y0 = oracle.layer_forward(x, lg, wg, wu, wd, keep, k, 1, *sh)
    dy = (y0 - tgt).astype(np.float32)
    dx, dl, _ = oracle.masked_backward(x, lg, wg, wu, wd, keep, k, 1, dy, *sh)

    def loss_lin(xx, ll):
        # L' = <dy, y(xx, ll)>: its gradient at the base point is the oracle's
        # backward of dy exactly
        return float((oracle.layer_forward(xx, ll, wg, wu, wd, keep, k, 1, *sh) * dy).sum())

    h = np.float32(2.0 ** -12)
    for t in range(T):
        for i in range(d):
            xp, xm = x.copy(), x.copy()
            xp[t, i] += h
            xm[t, i] -= h
            fd = (loss_lin(xp, lg) - loss_lin(xm, lg)) / (float(xp[t, i]) - float(xm[t, i]))
            assert abs(fd - dx[t, i]) <= 2e-6 * max(1.0, abs(dx[t, i]))
        for e in range(E):   # small logit moves keep the top-k set
            lp, lm = lg.copy(), lg.copy()
            lp[t, e] += h
            lm[t, e] -= h
            assert (topk_by_sort(lp, k) == topk_by_sort(lg, k)).all()
            fd = (loss_lin(x, lp) - loss_lin(x, lm)) / (float(lp[t, e]) - float(lm[t, e]))
            assert abs(fd - dl[t, e]) <= 2e-6 * max(1.0, abs(dl[t, e]))


def test_action_grad_special_cases():
    E, K, I = 3, 4, 16
    alpha = np.zeros((E, K), np.float32)
    g = np.zeros((E, K), np.float32)
    dm = np.zeros((E, I))
    counts = np.array([5, 0, 3], np.int32)
    # uniform logits, no quality signal: the entropy is log K and its gradient
    # vanishes; the cost gradient pushes each loaded expert towards thinner
    # actions in proportion to its load
    da, C, H = oracle.action_grad(RATIOS, I, alpha, g, 1.0, dm, counts, 8, 1.0, 1.0)
    assert H == pytest.approx(np.log(K), rel=1e-14)
    rbar = np.mean(RATIOS)
    assert C == pytest.approx((5 / 8 + 3 / 8) * rbar, rel=1e-14)
    np.testing.assert_allclose(da[1], 0.0, atol=1e-16)
    np.testing.assert_allclose(da[0], 5 / 8 * 0.25 * (np.array(RATIOS) - rbar), rtol=1e-13)
    # a unit gradient on every channel of the mask: dz_k = K_k (the width)
    dm[:] = 1.0
    da, _, _ = oracle.action_grad(RATIOS, I, alpha, g, 2.0, dm, counts, 8, 0.0, 0.0)
    w = np.array([int(np.ceil(r * I - 1e-9)) for r in RATIOS], np.float64)
    np.testing.assert_allclose(da[2], 0.25 * (w - w.mean()) / 2.0, rtol=1e-13)
