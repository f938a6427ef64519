"""The oracle's pins catch plausible mistakes (CPU only).  Each case plants
one mistake in an oracle function -- a swapped pair of bounds, a dropped
term, a wrong sign, an index off by one, rows misaligned with their tokens,
the other variance estimator, eps inside the square root, a rounding
instead of a floor, a window one slot too wide, steps counted one too many,
a dropped tail bin, the AsymRE offset's sign flipped or its loss
normalised per token instead of per sequence, the draw counter's words swapped, a packed window
shifted by one token -- by wrapping it under the name a pin test calls it by, then
runs pins of that function and requires at least one of them to fail.  The
oracle itself is untouched; the mistakes live in this file only."""

import numpy as np
import pytest

import oracle.buffer as ob_mod
import oracle.philox as philox_mod
import test_oracle_advantage as t_adv
import test_oracle_buffer as t_buf
import test_oracle_grad as t_grad
import test_oracle_logprob as t_lp
import test_oracle_loss as t_loss
import test_oracle_loss_variants as t_var
import test_oracle_philox as t_ph


def _some_pin_fails(pins):
    failed = []
    for pin in pins:
        try:
            pin()
        except AssertionError:
            failed.append(pin)
    return failed


def _mutations(golden_dir):
    from oracle.advantage import group_advantage
    from oracle.grad import logprob_backward
    from oracle.logprob import entropy, logprob
    from oracle.loss import asymre_coef, asymre_loss, grpo_loss, grpo_seq_loss

    def swapped_bounds(*a, eps_low=0.2, eps_high=0.2):
        return grpo_loss(*a, eps_low=eps_high, eps_high=eps_low)

    def flipped_gradient(*a, **k):
        loss, d, st = grpo_loss(*a, **k)
        return loss, -d, st

    def lengths_dropped(logp, old, seq, adv, lens, n_seq, **k):
        return grpo_loss(logp, old, seq, adv, np.ones_like(np.asarray(lens)), n_seq, **k)

    def target_off_by_one(h, W, y, *a, **k):
        return logprob(h, W, (np.asarray(y) + 1) % np.asarray(W).shape[0], *a, **k)

    def backward_sign(*a, **k):
        dh, dW = logprob_backward(*a, **k)
        return -dh, -dW

    def rows_misaligned(h, *a, **k):
        return logprob_backward(np.roll(np.asarray(h), 1, axis=0), *a, **k)

    def entropy_sign(h, W, *a, **k):
        return -entropy(h, W, *a, **k)

    def other_std(rewards, group_off, ddof=1, eps=1e-6):
        return group_advantage(rewards, group_off, ddof=1 - ddof, eps=eps)

    def seq_bounds_swapped(*a, eps_low=0.2, eps_high=0.2):
        return grpo_seq_loss(*a, eps_low=eps_high, eps_high=eps_low)

    real_uniform = philox_mod.uniform_index

    def rounded_index(x, n):
        return min(int(round(int(x) * int(n) / 2**64)), int(n) - 1)

    real_retained = ob_mod.retained_set

    def window_too_wide(rewards, n_fresh, n_pos_keep):
        return real_retained(rewards, int(n_fresh) + 1, n_pos_keep)

    def eps_inside_the_root(rewards, group_off, ddof=1, eps=1e-6):
        # A = (r - mean) / sqrt(var + eps) instead of / (std + eps)
        out = []
        for g in range(len(group_off) - 1):
            r = [float(x) for x in rewards[group_off[g]:group_off[g + 1]]]
            base = group_advantage(r, [0, len(r)], ddof=ddof, eps=0.0)
            n = len(r)
            if n - ddof <= 0 or all(v == 0.0 for v in base):
                out += [0.0] * n
                continue
            m = sum(r) / n
            var = sum((v - m) ** 2 for v in r) / (n - ddof)
            out += [(v - m) / (var + eps) ** 0.5 for v in r]
        return out

    real_since = ob_mod.steps_since_last_use

    def since_off_by_one(batches):
        return [[v if v < 0 else v + 1 for v in b] for b in real_since(batches)]

    real_hist = ob_mod.histogram

    def offset_sign_flipped(rewards, group_off, delta_v=-0.1):
        return asymre_coef(rewards, group_off, -delta_v)

    def asymre_normalised_per_token(logp, seq, coef, n_seq):
        # divides by the number of valid tokens instead of the sequences
        n_tok = int(np.sum(np.asarray(seq) >= 0))
        return asymre_loss(logp, seq, coef, max(n_tok, 1))

    real_block = philox_mod.draw_block

    def counter_words_swapped(seed, step, j):
        return real_block(seed, j, step)

    real_gather = ob_mod.gather

    def window_off_by_one(*a, **k):
        if k.get("layout", a[8] if len(a) > 8 else None) == ob_mod.LAYOUT_PACKED:
            k = dict(k, token_begin=k.get("token_begin", 0) + 1)
        return real_gather(*a, **k)

    def tail_bin_dropped(values, n_bins, lo=0):
        return real_hist([v for v in values if v - lo < n_bins], n_bins, lo)

    return [
        ("token clip bounds swapped", t_loss, "grpo_loss", swapped_bounds,
         [lambda: t_loss.test_asymmetric_clip_range(1.0, 1.25, True, 1.25),
          lambda: t_loss.test_asymmetric_clip_range(-1.0, 0.75, False, -0.9)]),
        ("gradient sign flipped", t_loss, "grpo_loss", flipped_gradient,
         [t_loss.test_finite_differences_away_from_kinks, t_loss.test_on_policy_identity]),
        ("per-sequence token mean dropped", t_loss, "grpo_loss", lengths_dropped,
         [t_loss.test_on_policy_identity]),
        ("target index off by one", t_lp, "logprob", target_off_by_one,
         [t_lp.test_pure_python_brute_force_tiny, t_lp.test_against_scipy_logsumexp]),
        ("backward sign flipped", t_grad, "logprob_backward", backward_sign,
         [t_grad.test_finite_differences_of_the_whole_path]),
        ("hidden rows misaligned with their tokens", t_grad, "logprob_backward",
         rows_misaligned, [t_grad.test_finite_differences_of_the_whole_path]),
        ("entropy sign flipped", t_lp, "entropy", entropy_sign,
         [t_lp.test_entropy_of_uniform_logits_is_log_v]),
        ("population instead of sample spread", t_adv, "group_advantage", other_std,
         [lambda: t_adv.test_binary_rewards_closed_form(4), t_adv.test_population_std_closed_form]),
        ("sequence clip bounds swapped", t_var, "grpo_seq_loss", seq_bounds_swapped,
         [t_var.test_seq_ratio_asymmetric_clip_range]),
        ("index rounded instead of floored", philox_mod, "uniform_index", rounded_index,
         [lambda: t_ph.test_uniform_index_is_floor_of_scaled_word(3),
          lambda: t_ph.test_uniform_index_is_floor_of_scaled_word(1000)]),
        ("retention window one slot too wide", ob_mod, "retained_set", window_too_wide,
         [lambda: t_buf.test_paper_worked_example_positive_bias(golden_dir),
          t_buf.test_retain_brute_force_definition]),
        ("eps inside the square root", t_adv, "group_advantage", eps_inside_the_root,
         [lambda: t_adv.test_one_outlier_closed_form(8, 0.1, 3)]),
        ("steps since last use off by one", ob_mod, "steps_since_last_use", since_off_by_one,
         [lambda: t_buf.test_steps_since_last_use_paper_example(golden_dir),
          t_buf.test_steps_since_last_use_brute_force]),
        ("histogram tail bin dropped", ob_mod, "histogram", tail_bin_dropped,
         [t_buf.test_histogram_bins_by_hand]),
        ("AsymRE offset sign flipped", t_var, "asymre_coef", offset_sign_flipped,
         [t_var.test_asymre_coef_group_sum_fixes_the_sign_of_delta_v]),
        ("AsymRE normalised per token", t_var, "asymre_loss", asymre_normalised_per_token,
         [t_var.test_asymre_gradient_is_constant_per_sequence_and_matches_finite_differences,
          t_var.test_asymre_shift_identity_and_masking]),
        ("draw counter words swapped", philox_mod, "draw_block", counter_words_swapped,
         [t_ph.test_draw_block_counter_layout]),
        ("packed window shifted by one token", ob_mod, "gather", window_off_by_one,
         [t_buf.test_gather_packed_windows_tile_the_stream]),
    ]


CASES = ["token clip bounds swapped", "gradient sign flipped", "per-sequence token mean dropped",
         "target index off by one", "backward sign flipped",
         "hidden rows misaligned with their tokens", "entropy sign flipped",
         "population instead of sample spread", "sequence clip bounds swapped",
         "index rounded instead of floored", "retention window one slot too wide",
         "eps inside the square root", "steps since last use off by one",
         "histogram tail bin dropped", "AsymRE offset sign flipped",
         "AsymRE normalised per token", "draw counter words swapped",
         "packed window shifted by one token"]


@pytest.mark.parametrize("name", CASES)
def test_pins_catch_a_planted_mistake(name, golden_dir, monkeypatch):
    muts = {m[0]: m for m in _mutations(golden_dir)}
    assert set(muts) == set(CASES)
    _, where, attr, wrong, pins = muts[name]
    # the pins pass on the oracle as it is ...
    assert not _some_pin_fails(pins), name
    # ... and at least one fails with the mistake planted
    monkeypatch.setattr(where, attr, wrong)
    assert _some_pin_fails(pins), f"no pin caught: {name}"
