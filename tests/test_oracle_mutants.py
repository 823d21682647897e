"""The oracle's pins catch plausible mistakes in it.

Each case plants one mistake in a copy of an oracle module (a dropped term, a
wrong sign, bound, index or operand, a misplaced reduction), then runs every
pin test of that module against the copy: at least one pin must fail.  The
unaltered copy must pass every pin, so a failure is the planted mistake's.
The mistakes are planted on the CPU, in the oracle only; nothing here touches
the GPU path.
"""
import inspect
import itertools
import os
import types

import pytest

import oracle
import test_oracle_design
import test_oracle_loss
import test_oracle_proxy
import test_oracle_sampler

ORACLE_DIR = os.path.dirname(os.path.abspath(oracle.__file__))

# module, the pin tests that use it and the name they know it by
TARGETS = {
    "ppo_head": [(test_oracle_loss, "ppo_head")],
    "cutoffs": [(test_oracle_sampler, "cutoffs"), (test_oracle_loss, "cutoffs")],
    "philox": [(test_oracle_sampler, "philox")],
    "score_proxy": [(test_oracle_proxy, "osp")],
    "cutoff_design": [(test_oracle_design, "cd")],
}

# (module, text as written, planted mistake, what the mistake is)
MUTANTS = [
    # LM-head + PPO loss (Sec. 3.1, Sec. 3.2, App. D)
    ("ppo_head", "lse_c = m + np.log(", "lse_c = np.log(", "lse without the row maximum"),
    ("ppo_head", "l_c = z[rows, target[s:e]] - lse_c", "l_c = z[rows, target[s:e] - 1] - lse_c",
     "target index off by one"),
    ("ppo_head", "r_c = np.exp(l_c - lp_old[s:e])", "r_c = np.exp(lp_old[s:e] - l_c)", "ratio inverted"),
    ("ppo_head", "clipped = np.clip(r_c, 1.0 - eps_low, 1.0 + eps_high)",
     "clipped = np.clip(r_c, 1.0 - eps_high, 1.0 + eps_low)", "clip bounds swapped"),
    ("ppo_head", "s_c = np.minimum(r_c * a_c, clipped * a_c)", "s_c = np.maximum(r_c * a_c, clipped * a_c)",
     "pessimistic min replaced by max"),
    ("ppo_head", "mu_c = (((a_c > 0) & (r_c <= 1.0 + eps_high))", "mu_c = (((a_c > 0) & (r_c >= 1.0 - eps_low))",
     "wrong clip branch for positive advantages"),
    ("ppo_head", "d_c = -loss_scale * c[s:e] * mu_c * r_c * a_c", "d_c = loss_scale * c[s:e] * mu_c * r_c * a_c",
     "gradient sign"),
    ("ppo_head", "d_c = -loss_scale * c[s:e] * mu_c * r_c * a_c", "d_c = -loss_scale * mu_c * r_c * a_c",
     "cutoff weight missing from the gradient"),
    ("ppo_head", "d_c = -loss_scale * c[s:e] * mu_c * r_c * a_c", "d_c = -loss_scale * c[s:e] * mu_c * a_c",
     "ratio missing from the gradient"),
    ("ppo_head", "G[rows, target[s:e]] += d_c", "G[rows, target[s:e]] -= d_c", "one-hot term sign"),
    ("ppo_head", "G[rows, target[s:e]] += d_c", "pass", "one-hot term dropped"),
    ("ppo_head", "dH[s:e] = G @ W", "dH[s:e] = -G @ W", "dH sign"),
    ("ppo_head", "dW += G.T @ h[s:e]", "dW = G.T @ h[s:e]", "dW overwritten per chunk instead of summed"),
    ("ppo_head", "loss = -loss_scale * float(np.sum(c * surr))", "loss = -loss_scale * float(np.sum(surr))",
     "cutoff weight missing from the loss"),
    ("ppo_head", "loss = -loss_scale * float(np.sum(c * surr))", "loss = loss_scale * float(np.sum(c * surr))",
     "loss sign"),
    ("ppo_head", "out[s:s + chunk] = lp[np.arange(lp.shape[0]), target[s:s + chunk]]",
     "out[s:s + chunk] = lp[np.arange(lp.shape[0]), target[s:s + chunk] - 1]", "target log-prob index"),
    ("ppo_head", "G = -delta[s:e, None] * np.exp(z - lse[s:e, None])",
     "G = delta[s:e, None] * np.exp(z - lse[s:e, None])", "selected dW rows: softmax term sign"),
    # cutoff sampling and packing (Sec. 3.2, Algorithm 1)
    ("cutoffs", "q.append(max(1, int(np.floor(float(v) * float(TWO32)))))",
     "q.append(max(1, int(np.ceil(float(v) * float(TWO32)))))", "thresholds rounded up"),
    ("cutoffs", "kept = [t for t in range(len(q)) if x < q[t]]", "kept = [t for t in range(len(q)) if x <= q[t]]",
     "inclusive threshold comparison"),
    ("cutoffs", "H[r] = min(int(lengths[r]), max(kept))", "H[r] = max(kept)", "cutoff not clipped to the length"),
    ("cutoffs", "weight[i] = token_weight(q[j + 1])", "weight[i] = token_weight(q[j])", "weight index off by one"),
    ("cutoffs", "src_row[i] = full_off[r] + j", "src_row[i] = cu[r] + j", "source row from the packed offset"),
    ("cutoffs", "seq_id[i] = r", "seq_id[i] = p", "completion id replaced by the prompt id"),
    ("cutoffs", "pmf[min(h, T_r)] += (q[h] - q[h + 1]) / float(TWO32)",
     "pmf[min(h, T_r)] += (q[h] - q[h + 1]) / float(TWO32 - 1)", "pmf normalised by 2^32 - 1"),
    ("cutoffs", "if np.any(np.diff(seg) > 0.0):", "if np.any(np.diff(seg) < 0.0):",
     "monotonicity check reversed"),
    # Philox4x32-10 (SC'11)
    ("philox", "p0 = PHILOX_M0 * c0", "p0 = PHILOX_M1 * c0", "round multiplier M0 replaced by M1"),
    ("philox", "if rnd > 0:", "if rnd >= 0:", "key bumped before the first round"),
    ("philox", "(hi1 ^ c1 ^ k0) & MASK32, lo1, (hi0 ^ c3 ^ k1) & MASK32, lo0",
     "(hi0 ^ c1 ^ k0) & MASK32, lo1, (hi1 ^ c3 ^ k1) & MASK32, lo0", "high words of the products swapped"),
    ("philox", "ctr = (r & MASK32, 0, offset & MASK32, (offset >> 32) & MASK32)",
     "ctr = (0, r & MASK32, offset & MASK32, (offset >> 32) & MASK32)", "counter words swapped"),
    # output-head score proxy (App. D)
    ("score_proxy", "diff[rows, o] += 1.0", "diff[rows, o] -= 1.0", "one-hot sign"),
    ("score_proxy", "gamma[s:s + chunk] = (hs * hs).sum(axis=1) * (diff * diff).sum(axis=1)",
     "gamma[s:s + chunk] = (diff * diff).sum(axis=1)", "||h||^2 factor dropped"),
    ("score_proxy", "psq[s:s + chunk] = (p * p).sum(axis=1)", "psq[s:s + chunk] = p.sum(axis=1)",
     "||p||^2 without the square"),
    # cutoff design (Sec. 3.3, App. E, App. F)
    ("cutoff_design", "gbar.append(sum(gamma[off[r] + t - 1] for r in alive) / n)",
     "gbar.append(sum(gamma[off[r] + t - 1] for r in alive) / K)", "gbar averaged over all K completions"),
    ("cutoff_design", "u.append(max(0.0, 0.5 - 0.5 * l1 / n))", "u.append(max(0.0, 0.5 - 0.5 * l1))",
     "u without the 1/n_t scaling"),
    ("cutoff_design", "while stack and math.sqrt(stack[-1][2] / stack[-1][1]) < math.sqrt(blk[2] / blk[1]):",
     "while stack and math.sqrt(stack[-1][2] / stack[-1][1]) > math.sqrt(blk[2] / blk[1]):",
     "pooling merges the wrong way"),
    ("cutoff_design", "xi = np.minimum(1.0, budget * root / root.sum())",
     "xi = np.minimum(1.0, budget * w / w.sum())", "heuristic proportional to w, not sqrt(w)"),
    ("cutoff_design", "acc += blocks[m][1] * score[m]", "acc += score[m]", "block lengths dropped from the budget"),
    ("cutoff_design", "if kappa * score[m] <= 1.0:", "if kappa * score[m] < 0.5:", "cap test wrong"),
    ("cutoff_design", "return (T - t) / T", "return (T - t - 1) / T", "uniform variant off by one"),
]


# pin tests that plant mistakes of their own in the oracle's source text (read from the file)
SELF_MUTATING = {"test_topk_rest_coordinate_pins_sign_and_abs"}


def _param_sets(fn):
    """The keyword sets pytest would call `fn` with (its parametrize marks, crossed)."""
    axes = []
    for mark in getattr(fn, "pytestmark", []):
        if mark.name != "parametrize":
            continue
        names, values = mark.args[0], mark.args[1]
        names = [n.strip() for n in names.split(",")] if isinstance(names, str) else list(names)
        axes.append([dict(zip(names, v if len(names) > 1 else (v,))) for v in values])
    for combo in itertools.product(*axes) if axes else [()]:
        kw = {}
        for part in combo:
            kw.update(part)
        yield kw


def _failing_pin(module_name, mod):
    """Runs every pin test of the oracle module with `mod` in its place; returns the first
    failing test's name, or None if all pass."""
    for test_mod, attr in TARGETS[module_name]:
        orig = getattr(test_mod, attr)
        setattr(test_mod, attr, mod)
        try:
            for name in sorted(n for n in vars(test_mod) if n.startswith("test_") and n not in SELF_MUTATING):
                fn = getattr(test_mod, name)
                for kw in _param_sets(fn):
                    mp = pytest.MonkeyPatch()
                    try:
                        if "monkeypatch" in inspect.signature(fn).parameters:
                            kw = dict(kw, monkeypatch=mp)
                        fn(**kw)
                    except Exception:
                        return f"{test_mod.__name__}.{name}"
                    finally:
                        mp.undo()
        finally:
            setattr(test_mod, attr, orig)
    return None


def _load(module_name, old=None, new=None):
    with open(os.path.join(ORACLE_DIR, module_name + ".py")) as f:
        src = f.read()
    if old is not None:
        assert src.count(old) == 1, f"{module_name}: the text to alter must occur exactly once: {old!r}"
        src = src.replace(old, new)
    mod = types.ModuleType(f"oracle.{module_name}")
    mod.__package__ = "oracle"
    mod.__file__ = os.path.join(ORACLE_DIR, module_name + ".py")
    exec(compile(src, f"<oracle {module_name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("module_name", sorted(TARGETS))
def test_unaltered_copies_pass_every_pin(module_name):
    assert _failing_pin(module_name, _load(module_name)) is None


@pytest.mark.parametrize("module_name,old,new,what", MUTANTS, ids=[m[3] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(module_name, old, new, what):
    assert _failing_pin(module_name, _load(module_name, old, new)) is not None, f"no pin catches: {what}"
