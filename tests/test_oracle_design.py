"""Pins of the float64 cutoff-design oracle (Sec. 3.3; App. E, F) against independent facts."""
import numpy as np
import pytest
from scipy.optimize import minimize

from oracle import cutoff_design as cd


def _direct_solve(w, B):
    """General-purpose solve of min sum w/xi s.t. sum xi = B, 1 >= xi_1 >= ... >= xi_T > 0,
    in the variables y = log xi (SLSQP; the exponential keeps every iterate positive)."""
    T = len(w)
    cons = [{"type": "eq", "fun": lambda y: np.exp(y).sum() - B, "jac": lambda y: np.exp(y)}]
    for t in range(T - 1):
        cons.append({"type": "ineq", "fun": lambda y, t=t: y[t] - y[t + 1]})
    res = minimize(lambda y: np.sum(w * np.exp(-y)), np.full(T, np.log(B / T)), jac=lambda y: -w * np.exp(-y),
                   bounds=[(-40.0, 0.0)] * T, constraints=cons, method="SLSQP",
                   options=dict(ftol=1e-15, maxiter=5000))
    x = np.exp(res.x)
    # SLSQP may end on a line-search message at the optimum: accept a feasible point
    assert abs(x.sum() - B) < 1e-8 and np.all(np.diff(x) <= 1e-10) and x.max() <= 1.0, res.message
    return x


@pytest.mark.parametrize("seed,T,B", [(0, 6, 2.0), (1, 8, 3.5), (2, 10, 7.0), (3, 9, 1.2), (4, 12, 11.0),
                                     (5, 7, 0.5), (6, 15, 4.0)])
def test_matches_a_direct_convex_solve(seed, T, B):
    rng = np.random.default_rng(seed)
    w = rng.gamma(0.7, 1.0, T) * rng.choice([0.05, 1.0, 20.0], T)
    xi = cd.design_xi(w, B)
    ref = _direct_solve(w, B)
    assert np.sum(w / xi) <= np.sum(w / ref) * (1 + 1e-10)
    np.testing.assert_allclose(xi, ref, rtol=1e-6)
    assert xi.sum() == pytest.approx(B, rel=1e-12)
    assert np.all(np.diff(xi) <= 0) and xi[0] <= 1.0


def test_unconstrained_closed_form():
    """Non-increasing weights and a small budget: the paper's closed form B sqrt(w)/sum sqrt(w)."""
    w = np.sort(np.random.default_rng(5).gamma(1.0, 1.0, 30))[::-1]
    B = 4.0
    xi = cd.design_xi(w, B)
    np.testing.assert_allclose(xi, B * np.sqrt(w) / np.sqrt(w).sum(), rtol=1e-14)
    assert len(cd.pav_blocks(w)) == 30


def test_pooling_of_increasing_weights():
    """Increasing weights violate monotonicity everywhere: one pooled block, xi = B/T."""
    w = np.arange(1.0, 21.0)
    assert len(cd.pav_blocks(w)) == 1
    np.testing.assert_allclose(cd.design_xi(w, 5.0), 5.0 / 20, rtol=1e-15)


def test_blockwise_closed_form():
    """Two pooled blocks: xi_m = B s_m / sum_j L_j s_j with s_m = sqrt(W_m / L_m)."""
    w = np.array([1.0, 4.0, 9.0, 0.25, 1.0])        # blocks [0..2] and [3..4]
    blocks = cd.pav_blocks(w)
    assert [(s, L) for s, L, _ in blocks] == [(0, 3), (3, 2)]
    s = np.array([np.sqrt(14.0 / 3), np.sqrt(1.25 / 2)])
    B = 2.0
    expect = B * s / (3 * s[0] + 2 * s[1])
    xi = cd.design_xi(w, B)
    np.testing.assert_allclose(xi, np.repeat(expect, [3, 2]), rtol=1e-14)


def test_saturated_prefix():
    """A dominant first weight saturates at 1; the rest shares B - 1 (App. F remark)."""
    w = np.array([1e6, 4.0, 1.0, 1.0])
    xi = cd.design_xi(w, 2.0)
    assert xi[0] == 1.0
    rest = np.sqrt(w[1:])
    np.testing.assert_allclose(xi[1:], 1.0 * rest / rest.sum(), rtol=1e-14)
    np.testing.assert_allclose(cd.design_xi(w, 10.0), 1.0)     # budget >= T: full trajectory


def test_variants():
    T = 50
    t = np.arange(T)
    np.testing.assert_allclose(cd.design_xi(np.ones(T), 5.0, cd.UNIFORM), (T - t) / T)
    assert cd.design_xi(np.ones(T), 5.0, cd.UNIFORM).sum() == pytest.approx((T + 1) / 2)  # E[H] of U{1..T}
    np.testing.assert_allclose(cd.design_xi(np.ones(T), 5.0, cd.TIME_PRIOR, lam=0.1), np.exp(-0.1 * t))
    w = np.random.default_rng(6).gamma(0.5, 1.0, T)
    h = cd.design_xi(w, 8.0, cd.HEURISTIC)
    raw = np.minimum(1.0, 8.0 * np.sqrt(w) / np.sqrt(w).sum())
    np.testing.assert_allclose(h, np.maximum(np.minimum.accumulate(raw), cd.XI_FLOOR))
    # the heuristic is feasible but never better than the optimum at the same or larger budget
    opt = cd.design_xi(w, h.sum())
    assert np.sum(w / opt) <= np.sum(w / h) * (1 + 1e-12)


def test_zero_weights():
    np.testing.assert_allclose(cd.design_xi(np.zeros(10), 4.0), 0.4)
    xi = cd.design_xi(np.array([4.0, 1.0, 0.0, 0.0]), 3.0)       # trailing zero-weight block
    assert xi[0] == 1.0 and xi[1] == 1.0 and xi.sum() == pytest.approx(3.0)
    assert np.all(np.diff(xi) <= 0)


def _dense_u(pis, succ):
    """1/2 - 1/2 || p_hat pibar_G - (1 - p_hat) pibar_B ||_1 with dense distributions."""
    pis = np.asarray(pis)
    succ = np.asarray(succ, dtype=bool)
    n = len(succ)
    p = succ.mean()
    g = pis[succ].mean(axis=0) if succ.any() else np.zeros(pis.shape[1])
    b = pis[~succ].mean(axis=0) if (~succ).any() else np.zeros(pis.shape[1])
    return 0.5 - 0.5 * np.abs(p * g - (1 - p) * b).sum()


def test_proxy_weights_full_distributions():
    """top-k = V: u_t is the dense formula over the completions alive at t; gbar is their mean."""
    rng = np.random.default_rng(7)
    P, K, V = 2, 4, 12
    lengths = np.array([5, 3, 5, 1, 2, 4, 4, 3])
    S = lengths.sum()
    logits = rng.standard_normal((S, V)) * 1.5
    pi = np.exp(logits) / np.exp(logits).sum(axis=1, keepdims=True)
    order = np.argsort(-pi, axis=1)
    ids = order.astype(np.int32)
    logp = np.log(np.take_along_axis(pi, order, axis=1))
    gamma = rng.gamma(2.0, 1.0, S)
    rewards = np.array([1, 0, 0, 1, 1, 1, 0, 1], dtype=np.float64)
    out = cd.proxy_weights(gamma, ids, logp, lengths, rewards, P, K)
    off = np.concatenate([[0], np.cumsum(lengths)])
    i = 0
    for p in range(P):
        rows = np.arange(p * K, (p + 1) * K)
        for t in range(1, lengths[rows].max() + 1):
            alive = rows[lengths[rows] >= t]
            pis = pi[off[alive] + t - 1]
            assert out["u"][i] == pytest.approx(_dense_u(pis, rewards[alive] > 0.5), abs=1e-13)
            assert out["gbar"][i] == pytest.approx(gamma[off[alive] + t - 1].mean(), rel=1e-14)
            i += 1
    assert i == len(out["w"])
    np.testing.assert_allclose(out["w"], out["gbar"] * out["u"])
    assert np.all(out["u"] >= 0) and np.all(out["u"] <= 0.5)


def test_u_is_zero_for_equal_rewards_and_bounds_the_reward_variance():
    rng = np.random.default_rng(8)
    # equal rewards: the outcome is known, u = 0 (whatever the distributions)
    lengths = np.array([3, 3, 3])
    ids = np.tile(np.arange(4, dtype=np.int32), (9, 1))
    logp = np.log(rng.dirichlet(np.ones(4), 9))
    out = cd.proxy_weights(np.ones(9), ids, logp, lengths, np.ones(3), 1, 3)
    np.testing.assert_allclose(out["u"], 0.0, atol=1e-15)
    # App. E: E[Var(R | S_t)] <= u_t.  A world of 5 states with their own next-token
    # distributions and success rates, represented exactly by completions: state s
    # contributes n1_s successes and n0_s failures that share its distribution.
    V = 6
    n1 = np.array([3, 0, 2, 5, 1])
    n0 = np.array([1, 4, 2, 0, 3])
    pis = rng.dirichlet(np.ones(V) * 0.7, 5)
    rows_pi, rewards = [], []
    for s in range(5):
        rows_pi += [pis[s]] * (n1[s] + n0[s])
        rewards += [1.0] * n1[s] + [0.0] * n0[s]
    rows_pi = np.array(rows_pi)
    K = len(rewards)
    order = np.argsort(-rows_pi, axis=1)
    out = cd.proxy_weights(np.ones(K), order.astype(np.int32),
                           np.log(np.take_along_axis(rows_pi, order, axis=1)),
                           np.ones(K, dtype=np.int64), np.array(rewards), 1, K)
    n = n1 + n0
    ps = n1 / n
    ev = np.sum(n / n.sum() * ps * (1 - ps))
    assert ev <= out["u"][0] + 1e-15
    # truncating to the top-2 entries of each distribution keeps a valid u in [0, 1/2]
    out2 = cd.proxy_weights(np.ones(K), order[:, :2].astype(np.int32),
                            np.log(np.take_along_axis(rows_pi, order[:, :2], axis=1)),
                            np.ones(K, dtype=np.int64), np.array(rewards), 1, K)
    assert 0.0 <= out2["u"][0] <= 0.5


def test_design_tables_layout():
    w = np.concatenate([np.ones(5), np.arange(1.0, 4.0)])
    xi = cd.design_tables(w, [0, 5, 8], 2.0)
    np.testing.assert_allclose(xi[:5], 0.4)
    np.testing.assert_allclose(xi[5:], 2.0 / 3)


def _common_tail_case(seed, n, k, V=60, listed=36, rest_range=(0.05, 0.5)):
    """Dense next-token distributions pi_r = pit_r + rest_r tau: pit_r on the k ids of row r's
    list (ids < `listed`), tau one tail distribution on the ids >= `listed` (outside every
    list), rest_r the row's mass outside its list."""
    rng = np.random.default_rng(seed)
    tau = rng.dirichlet(np.ones(V - listed))
    ids = np.stack([rng.choice(listed, k, replace=False) for _ in range(n)]).astype(np.int32)
    rest = rng.uniform(*rest_range, n)
    top = rng.dirichlet(np.ones(k), n) * (1.0 - rest)[:, None]
    dense = np.zeros((n, V))
    dense[np.arange(n)[:, None], ids] = top
    dense[:, listed:] = rest[:, None] * tau[None, :]
    return dense, ids, np.log(top), rest


@pytest.mark.parametrize("seed,n,k,succ", [(10, 6, 3, [1, 0, 0, 1, 1, 0]), (11, 8, 5, [1, 1, 1, 0, 1, 1, 0, 1]),
                                           (12, 5, 2, [0, 0, 1, 0, 0]), (13, 7, 4, [0, 1, 0, 1, 0, 1, 0])])
def test_topk_rest_coordinate_equals_dense_formula(seed, n, k, succ):
    """App. E with top-k lists (k < V): when the mass outside each list lies on one tail
    distribution shared by all completions and outside every list, the dense
    1/2 - 1/2 || p pibar_G - (1-p) pibar_B ||_1 equals the top-k formula with one signed
    "rest" coordinate exactly.  Rest masses 0.05..0.5 with successes holding more rest
    mass in some cases and less in others, so both signs of the rest difference occur."""
    dense, ids, logp, rest = _common_tail_case(seed, n, k)
    succ = np.array(succ, dtype=np.float64)
    out = cd.proxy_weights(np.ones(n), ids, logp, np.ones(n, dtype=np.int64), succ, 1, n)
    ref = _dense_u(dense, succ > 0.5)
    assert out["u"][0] == pytest.approx(ref, abs=1e-13)
    assert 0.0 < ref < 0.5


def test_topk_rest_coordinate_pins_sign_and_abs():
    """Mutants of the oracle's rest term fail the dense-formula pin: dropping the
    success/failure sign of each completion's rest mass, or the absolute value of the
    summed rest (flipping every sign at once leaves |rest| unchanged and is the same
    formula).  The mutants are the oracle's own source with one edit each."""
    import inspect
    import textwrap
    src = textwrap.dedent(inspect.getsource(cd.proxy_weights))
    mutants = {"no sign": ("rest += sign * max(0.0, 1.0 - mass)", "rest += max(0.0, 1.0 - mass)"),
               "no abs": ("+ abs(rest)", "+ rest")}
    cases = [(10, 6, 3, [1, 0, 0, 1, 1, 0]), (12, 5, 2, [0, 0, 1, 0, 0]), (13, 7, 4, [0, 1, 0, 1, 0, 1, 0])]
    for name, (old, new) in mutants.items():
        assert src.count(old) == 1, name
        ns = {"np": np}
        exec(src.replace(old, new), ns)
        failed = False
        for seed, n, k, succ in cases:
            dense, ids, logp, _ = _common_tail_case(seed, n, k)
            s = np.array(succ, dtype=np.float64)
            u = ns["proxy_weights"](np.ones(n), ids, logp, np.ones(n, dtype=np.int64), s, 1, n)["u"][0]
            failed |= abs(u - _dense_u(dense, s > 0.5)) > 1e-9
        assert failed, f"mutant '{name}' passes the pin"
