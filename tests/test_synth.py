"""Checks of the seeded workload generator against independent definitions."""
import dataclasses
import numpy as np
import pytest
import torch
from scipy import stats

from oracle import ppo_head
from paper_2606_29758_amd import synth


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3.0
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 0.0]   # ties to even
    mine = synth.round_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, ref)


def test_workload_is_deterministic_and_shaped():
    a = synth.make_workload("tiny")
    b = synth.make_workload("tiny")
    for k in ("lengths", "xi", "xi_off", "advantage", "target_full", "lp_noise", "hidden_bits", "w_bits"):
        assert np.array_equal(getattr(a, k), getattr(b, k)), k
    cfg = a.cfg
    assert a.lengths.min() >= 32 and a.lengths.max() <= 128
    assert a.hidden_bits.shape == (a.total_tokens, cfg.d)
    assert a.w_bits.shape == (cfg.V, cfg.d)
    assert a.target_full.min() >= 0 and a.target_full.max() < cfg.V
    assert np.array_equal(a.horizon, a.lengths.reshape(cfg.P, cfg.K).max(axis=1))


def test_advantage_is_group_mean_centred():
    wl = synth.make_workload("qwen1.5b", with_matrices=False)
    ref = ppo_head.advantages(wl.rewards, wl.cfg.K)
    assert np.array_equal(wl.advantage, ref.astype(np.float32))
    assert np.allclose(wl.advantage.reshape(-1, wl.cfg.K).sum(axis=1), 0.0, atol=1e-6)


def test_std_normalised_advantage():
    """GRPO-style advantages: each group with unequal rewards has mean 0 and population
    variance 1 (up to the 1e-6 guard); groups with equal rewards get A = 0."""
    cfg = dataclasses.replace(synth.CONFIGS["qwen1.5b"], adv_norm="std")
    wl = synth.make_workload(cfg, with_matrices=False)
    ref = ppo_head.advantages(wl.rewards, cfg.K, std_normalise=True)
    assert np.array_equal(wl.advantage, ref.astype(np.float32))
    g = ref.reshape(-1, cfg.K)
    r = wl.rewards.reshape(-1, cfg.K)
    const = (r == r[:, :1]).all(axis=1)
    assert const.any() and (~const).any()
    assert np.all(g[const] == 0)
    assert np.allclose(g[~const].mean(axis=1), 0, atol=1e-12)
    sd = r[~const].std(axis=1)
    assert np.allclose((g[~const] ** 2).mean(axis=1), (sd / (sd + 1e-6)) ** 2, rtol=1e-12)


@pytest.mark.parametrize("T", [1, 7, 64, 500])
def test_beta22_survival_closed_form(T):
    # survival of Beta(2,2) at y: 1 - 3y^2 + 2y^3; xi_t = S((t-1)/T)
    y = (np.arange(1, T + 1) - 1.0) / T
    expect = 1 - 3 * y ** 2 + 2 * y ** 3
    got = synth.beta_survival_table(2.0, 2.0, T)
    assert np.allclose(got, np.maximum(expect, 2.0 ** -60), rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("a,b", [(1.0, 3.0), (2.5, 1.0)])
def test_beta_edge_closed_forms(a, b):
    T = 200
    y = (np.arange(1, T + 1) - 1.0) / T
    expect = (1 - y) ** b if a == 1.0 else 1 - y ** a
    got = synth.beta_survival_table(a, b, T)
    assert np.allclose(got, np.maximum(expect, 2.0 ** -60), rtol=1e-10, atol=1e-15)


def test_expected_cutoff_equals_survival_sum():
    """E[H] = sum_t xi_t (the budget identity of Sec. 3.3) for H = ceil(f T), f ~ Beta."""
    a, b, T = 1.5, 4.0, 300
    xi = synth.beta_survival_table(a, b, T)
    dist = stats.beta(a, b)
    # E[ceil(fT)] by integrating ceil(fT) against the Beta density, interval by interval
    e = sum(h * (dist.cdf(h / T) - dist.cdf((h - 1) / T)) for h in range(1, T + 1))
    assert xi.sum() == pytest.approx(e, rel=1e-10)
    # and the mean of f itself bounds it: T*E[f] <= E[H] <= T*E[f] + 1
    assert T * a / (a + b) <= e <= T * a / (a + b) + 1


def test_full_trajectory_shares_data_with_7b():
    a = synth.make_workload("qwen7b", with_matrices=False)
    b = synth.make_workload("qwen7b_full", with_matrices=False)
    assert np.array_equal(a.lengths, b.lengths) and np.array_equal(a.target_full, b.target_full)
    assert np.all(b.xi == 1.0)
