"""Mutation tests of the oracle's pins (CPU only).  Each case copies one oracle
function's source, applies one plausible slip (a max for a min, swapped clip
bounds, a dropped normalisation or sign, a mean or variance divided by the
wrong count, a dropped epsilon), runs the mutant through the committed pins of
that function, and requires at least one pin to reject it.  The unmutated
functions pass every pin."""
import inspect

import pytest

import oracle.advantage as oracle_advantage
import oracle.grpo as oracle_grpo
import test_oracle_grpo as grpo_pins
import test_oracle_rollout as rollout_pins


def _mutant(fn, old, new):
    src = inspect.getsource(fn)
    assert src.count(old) == 1, old
    ns = dict(fn.__globals__)
    exec(compile(src.replace(old, new), inspect.getsourcefile(fn), "exec"), ns)
    return ns[fn.__name__]


def _rejected(pins):
    for pin in pins:
        try:
            pin()
        except Exception:   # a failed assertion, or an error the slip causes
            return True
    return False


SURROGATE_PINS = [grpo_pins.test_clip_quadrants_by_hand, grpo_pins.test_decoupled_clip_upper_bound] + \
    [lambda e=e: grpo_pins.test_matches_piecewise_form(e) for e in [(0.2, 0.2), (0.2, 0.28), (0.1, 0.5)]] + \
    [grpo_pins.test_ratio_one_closed_forms, grpo_pins.test_equal_lengths_make_modes_agree,
     grpo_pins.test_keep_mask_is_the_subset]

SURROGATE_SLIPS = {
    "max_instead_of_min": ("min(unclipped, clipped)", "max(unclipped, clipped)"),
    "clip_bounds_swapped": ("min(max(rho, 1.0 - eps_lo), 1.0 + eps_hi)", "min(max(rho, 1.0 - eps_hi), 1.0 + eps_lo)"),
    "no_clip": ("clipped = min(max(rho, 1.0 - eps_lo), 1.0 + eps_hi) * a", "clipped = rho * a"),
    "seq_mean_not_normalised": ("seq_total += seq_sum / L", "seq_total += seq_sum"),
    "token_mean_over_sequences": ('total / n_tok if mode == "token"', 'total / n_seq if mode == "token"'),
    "loss_sign": ("return -agg,", "return agg,"),
    "ratio_inverted": ("math.exp(new_lp[s, t] - old_lp[s, t])", "math.exp(old_lp[s, t] - new_lp[s, t])"),
}

ADVANTAGE_PINS = [rollout_pins.test_advantage_worked_examples] + \
    [lambda d=d: rollout_pins.test_advantage_invariants(d) for d in (0, 1)] + \
    [rollout_pins.test_advantage_constant_groups_and_bernoulli, rollout_pins.test_advantage_permutation_equivariant]

ADVANTAGE_SLIPS = {
    "variance_ignores_ddof": ("/ (g - ddof)", "/ g"),
    "mean_divided_by_g_minus_ddof": ("mu = sum(float(v) for v in r) / g", "mu = sum(float(v) for v in r) / (g - ddof)"),
    "deviation_not_squared": ("(float(v) - mu) ** 2", "abs(float(v) - mu)"),
    "centred_with_plus": ("(float(v) - mu) / (sigma + eps)", "(float(v) + mu) / (sigma + eps)"),
    "epsilon_dropped": ("(sigma + eps)", "(sigma + 0.0)"),
}


def test_unmutated_oracle_passes_every_pin():
    assert not _rejected(SURROGATE_PINS)
    assert not _rejected(ADVANTAGE_PINS)


@pytest.mark.parametrize("name", sorted(SURROGATE_SLIPS))
def test_surrogate_slip_is_rejected(name, monkeypatch):
    bad = _mutant(oracle_grpo.clipped_surrogate, *SURROGATE_SLIPS[name])
    monkeypatch.setattr(grpo_pins, "clipped_surrogate", bad)
    assert _rejected(SURROGATE_PINS), name


@pytest.mark.parametrize("name", sorted(ADVANTAGE_SLIPS))
def test_advantage_slip_is_rejected(name, monkeypatch):
    bad = _mutant(oracle_advantage.group_advantage, *ADVANTAGE_SLIPS[name])
    monkeypatch.setattr(rollout_pins, "group_advantage", bad)
    monkeypatch.setattr(grpo_pins, "group_advantage", bad)
    assert _rejected(ADVANTAGE_PINS), name
