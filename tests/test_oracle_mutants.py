"""Mutation tests of the oracle's pins (CPU only).  Each case copies one oracle
function's source, applies one plausible slip (a max for a min, swapped clip
bounds, a dropped normalisation or sign, a mean or variance divided by the
wrong count, a dropped epsilon), runs the mutant through the committed pins of
that function, and requires at least one pin to reject it.  The unmutated
functions pass every pin.  Covered: the clipped surrogate, the group-relative
advantage, the controller's straggler statistics, dual and posterior update
and neighbourhood choice, the sampler's noise, uniform mapping, bit layout,
temperature, forced EOS, log-probability and tie rule, and the teacher-forced
log-probabilities of the loss forward."""
import importlib
import inspect

import pytest

import oracle.advantage as oracle_advantage
import oracle.grpo as oracle_grpo
import oracle.philox as oracle_philox
import oracle.sagc as oracle_sagc
import oracle.sampling as oracle_sampling
import test_oracle_grpo as grpo_pins
import test_oracle_philox as philox_pins
import test_oracle_rollout as rollout_pins
import test_oracle_sagc as sagc_pins
from oracle.model import OracleModel
from workload import make_inputs, make_weights

# the package re-exports the function `rollout` under the submodule's name
oracle_rollout = importlib.import_module("oracle.rollout")


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


SAGC_PINS = [sagc_pins.test_group_stats_worked_examples, sagc_pins.test_group_stats_match_numpy,
             sagc_pins.test_dual_and_posterior_worked_example, sagc_pins.test_choice_rules,
             sagc_pins.test_initial_size_state] + \
    [lambda s=s: sagc_pins.test_closed_loop_separates_arms(s) for s in (0, 1)] + \
    [lambda z=z: sagc_pins.test_initial_size_is_uniform_over_the_admitted_sizes(z) for z in ((4, 8, 16), (2, 4))]

SAGC_SLIPS = {
    "stats_even_median_upper": ("group_stats", "(seg[g // 2 - 1] + seg[g // 2]) / 2.0", "float(seg[g // 2])"),
    "stats_tau_inclusive": ("group_stats", "1.0 if R > tau else 0.0", "1.0 if R >= tau else 0.0"),
    "stats_max_is_first": ("group_stats", "lmax = seg[-1]", "lmax = seg[0]"),
    "stats_unsorted": ("group_stats", "seg = sorted(int(v) for v in lengths[off:off + g])",
                       "seg = [int(v) for v in lengths[off:off + g]]"),
    "dual_step_sign": ("sagc_step", "st.lam + cfg.eta * (s_bar - cfg.delta)", "st.lam - cfg.eta * (s_bar - cfg.delta)"),
    "dual_not_projected": ("sagc_step", "max(0.0, st.lam + cfg.eta * (s_bar - cfg.delta))",
                           "(st.lam + cfg.eta * (s_bar - cfg.delta))"),
    "posterior_counts_swapped": ("sagc_step", "cfg.gamma * st.alpha[i] + s_bar", "cfg.gamma * st.alpha[i] + (1.0 - s_bar)"),
    "posterior_not_discounted": ("sagc_step", "st.beta[i] = cfg.gamma * st.beta[i]", "st.beta[i] = st.beta[i]"),
    "choice_ties_to_larger": ("sagc_choose", "scores[i] > scores[best]", "scores[i] >= scores[best]"),
    "choice_penalty_sign": ("sagc_choose", "- lam * samples[i]", "+ lam * samples[i]"),
    "choice_whole_range": ("sagc_choose", "(g_index - 1, g_index, g_index + 1)", "range(k)"),
    "init_never_largest": ("sagc_init", "int(u53(w[0]) * k)", "int(u53(w[0]) * (k - 1))"),
    "init_rounded": ("sagc_init", "int(u53(w[0]) * k)", "int(round(u53(w[0]) * (k - 1)))"),
    "init_low_half_only": ("sagc_init", "int(u53(w[0]) * k)", "int(u53(w[0] & 0xFFFFFFFF) * k)"),
}


def test_unmutated_oracle_passes_every_pin():
    assert not _rejected(SURROGATE_PINS)
    assert not _rejected(ADVANTAGE_PINS)
    assert not _rejected(SAGC_PINS)


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


@pytest.mark.parametrize("name", sorted(SAGC_SLIPS))
def test_controller_slip_is_rejected(name, monkeypatch):
    fn_name, old, new = SAGC_SLIPS[name]
    bad = _mutant(getattr(oracle_sagc, fn_name), old, new)
    monkeypatch.setattr(oracle_sagc, fn_name, bad)
    assert _rejected(SAGC_PINS), name


def _tiny():
    return OracleModel(grpo_pins.TINY.shape, make_weights(grpo_pins.TINY.shape, 0)), make_inputs(grpo_pins.TINY, 0)


SAMPLING_PINS = [philox_pins.test_gumbel_bits_layout, philox_pins.test_uniform_mapping_endpoints_and_exactness,
                 philox_pins.test_sample_token_forced_eos_and_logprob, philox_pins.test_sample_token_tie_goes_to_lowest_id,
                 lambda: grpo_pins.test_recompute_equals_rollout_logprobs(_tiny(), 0.7)] + \
    [lambda T=T: philox_pins.test_sample_token_frequencies_match_softmax(T) for T in (1.0, 0.7)] + \
    [lambda T=T: philox_pins.test_gumbel_max_frequencies_match_softmax(T) for T in (1.0, 0.7)]

# (module, function, old text, new text)
SAMPLING_SLIPS = {
    "noise_sign": (oracle_philox, "gumbel_noise", "return -np.log(-np.log(u))", "return np.log(-np.log(u))"),
    "uniform_reaches_one": (oracle_philox, "uniforms_from_bits", "((2.0 * k + 1.0) * 2.0 ** -24)",
                            "((k + 1.0) * 2.0 ** -23)"),
    "high_half_lost": (oracle_philox, "gumbel_uniform_bits", "halves[:, 1::2] = w >> _S32",
                       "halves[:, 1::2] = w & _M32"),
    "temperature_multiplies": (oracle_sampling, "sample_token", "z.astype(np.float32) / np.float32(temperature)",
                               "z.astype(np.float32) * np.float32(temperature)"),
    "logprob_ignores_temperature": (oracle_sampling, "sample_token", "zt = z / float(temperature)", "zt = z"),
    "forced_eos_one_late": (oracle_sampling, "sample_token", "t == int(forced_len) - 1", "t == int(forced_len)"),
    "eos_not_masked": (oracle_sampling, "sample_token", "score[eos_id] = -np.inf", "score[eos_id] = score[eos_id]"),
    "logprob_unnormalised": (oracle_sampling, "sample_token", "float(zt[y] - lse)", "float(zt[y])"),
    "ties_to_highest_id": (oracle_sampling, "sample_token", "int(np.argmax(score))",
                           "int(len(score) - 1 - np.argmax(score[::-1]))"),
}


@pytest.mark.parametrize("name", sorted(SAMPLING_SLIPS))
def test_sampling_slip_is_rejected(name, monkeypatch):
    mod, fn_name, old, new = SAMPLING_SLIPS[name]
    bad = _mutant(getattr(mod, fn_name), old, new)
    monkeypatch.setattr(mod, fn_name, bad)
    # every module that imported the function by name
    for m in (oracle_sampling, oracle_rollout, philox_pins, grpo_pins):
        if getattr(m, fn_name, None) is not None and m is not mod:
            monkeypatch.setattr(m, fn_name, bad)
    assert _rejected(SAMPLING_PINS), name


def test_unmutated_sampler_passes_every_pin():
    assert not _rejected(SAMPLING_PINS)


RECOMPUTE_PINS = [lambda T=T: grpo_pins.test_recompute_equals_rollout_logprobs(_tiny(), T) for T in (1.0, 0.7)]

RECOMPUTE_SLIPS = {
    "logits_row_one_late": ("zt = z[Lp - 1 + t] / float(temperature)", "zt = z[min(Lp + t, len(z) - 1)] / float(temperature)"),
    "temperature_dropped": ("zt = z[Lp - 1 + t] / float(temperature)", "zt = z[Lp - 1 + t]"),
    "unnormalised": ("out[s, t] = zt[y[t]] - logsumexp(zt)", "out[s, t] = zt[y[t]]"),
}


@pytest.mark.parametrize("name", sorted(RECOMPUTE_SLIPS))
def test_recompute_slip_is_rejected(name, monkeypatch):
    bad = _mutant(oracle_grpo.teacher_forced_logprobs, *RECOMPUTE_SLIPS[name])
    monkeypatch.setattr(grpo_pins, "teacher_forced_logprobs", bad)
    assert _rejected(RECOMPUTE_PINS), name


def test_unmutated_recompute_passes_its_pins():
    assert not _rejected(RECOMPUTE_PINS)
