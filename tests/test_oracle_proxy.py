"""Pins of the float64 output-head score proxy (App. D) against independent facts."""
import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import score_proxy as osp


def _case(seed, n=12, d=24, V=40, w_std=0.3):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((n, d))
    W = w_std * rng.standard_normal((V, d))
    o = rng.integers(0, V, n)
    return h, W, o


@pytest.mark.parametrize("seed,w_std", [(0, 0.3), (1, 1.5), (2, 0.01)])
def test_gamma_is_the_head_score_norm(seed, w_std):
    """gamma = ||grad_W log softmax(W h)[o]||_F^2, by float64 autograd, token by token."""
    h, W, o = _case(seed, w_std=w_std)
    got = osp.score_proxy(h, W, o)["gamma"]
    for i in range(len(o)):
        tW = torch.tensor(W, requires_grad=True)
        lp = torch.log_softmax(tW @ torch.tensor(h[i]), dim=0)[int(o[i])]
        (g,) = torch.autograd.grad(lp, tW)
        assert got[i] == pytest.approx(float((g * g).sum()), rel=1e-12)


def test_two_log_sum_exp_identity():
    """||p||^2 = exp(l2 - 2 l1) with l1 = lse(z), l2 = lse(2z); p(o) = exp(z_o - l1);
    ||e_o - p||^2 = 1 - 2 p(o) + ||p||^2."""
    h, W, o = _case(3, w_std=0.8)
    out = osp.score_proxy(h, W, o)
    z = h @ W.T
    l1 = logsumexp(z, axis=1)
    l2 = logsumexp(2 * z, axis=1)
    np.testing.assert_allclose(out["p_sq"], np.exp(l2 - 2 * l1), rtol=1e-12)
    np.testing.assert_allclose(out["logp"], z[np.arange(len(o)), o] - l1, rtol=1e-12, atol=1e-12)
    hn = (h * h).sum(axis=1)
    np.testing.assert_allclose(out["gamma"], hn * (1 - 2 * np.exp(out["logp"]) + out["p_sq"]), rtol=1e-10)


def test_special_cases():
    h, W, o = _case(4)
    V = W.shape[0]
    # a zero head: p uniform, gamma = ||h||^2 (1 - 1/V)
    out = osp.score_proxy(h, np.zeros_like(W), o)
    np.testing.assert_allclose(out["gamma"], (h * h).sum(axis=1) * (1 - 1.0 / V), rtol=1e-13)
    np.testing.assert_allclose(out["p_sq"], 1.0 / V, rtol=1e-13)
    # a nearly deterministic head that puts its mass on the target: gamma -> 0
    Wd = np.zeros_like(W)
    Wd[o[0]] = 60.0 * h[0] / np.linalg.norm(h[0])
    g = osp.score_proxy(h[:1], Wd, o[:1])["gamma"][0]
    assert 0.0 <= g < 1e-12 * (h[0] @ h[0]) + 1e-300
    # ... and on another token: ||e_o - p||^2 -> 2
    other = (o[0] + 1) % V
    g2 = osp.score_proxy(h[:1], Wd, np.array([other]))["gamma"][0]
    assert g2 == pytest.approx(2.0 * (h[0] @ h[0]), rel=1e-12)
    # a zero hidden state: gamma = 0
    assert not osp.score_proxy(np.zeros_like(h), W, o)["gamma"].any()


def test_bounds_and_chunking():
    h, W, o = _case(5, n=37, w_std=1.0)
    a = osp.score_proxy(h, W, o, chunk=5)
    b = osp.score_proxy(h, W, o, chunk=256)
    np.testing.assert_array_equal(a["gamma"], b["gamma"])
    hn = (h * h).sum(axis=1)
    # 0 <= ||e_o - p||^2 <= 2 and ||p||^2 in [1/V, 1]
    assert np.all(a["gamma"] >= 0) and np.all(a["gamma"] <= 2 * hn)
    assert np.all(a["p_sq"] >= 1.0 / W.shape[0] - 1e-15) and np.all(a["p_sq"] <= 1 + 1e-15)
