"""Plant plausible mistakes in the oracle (on the CPU) and check that the pins catch each.

A mistake that no pin catches would mean the oracle is only checked against
itself there.  Each mutation wraps an oracle function with a wrong variant and
runs the pin tests of test_oracle_pins; at least one must fail.
"""
import numpy as np
import pytest

import oracle
import oracle.beam as ob
from oracle.beam import NEG_INF
from tests import test_oracle_pins as pins

PINS = [
    pins.test_projection_matches_scalar_loop,
    pins.test_log_softmax_rows_sum_to_one,
    pins.test_lmbr_row_single_path_closed_form,
    pins.test_hand_worked_example,
    pins.test_top_k_total_order,
    pins.test_k1_is_greedy_search,
    lambda: pins.test_exhaustive_argmax(4, 3, 16, 30),
    pins.test_finished_entries_keep_rescorable_scores,
    pins.test_lambda_zero_is_plain_nmt_beam_search,
    pins.test_first_step_expands_only_slot_zero,
    pins.test_beam_invariants_small_config,
    pins.test_forced_eos_bias_enters_before_softmax,
    lambda: pins.test_exhaustive_argmax_length_normalised(4, 3, 16, 30),
    pins.test_length_normalised_order_hand_example,
    pins.test_per_sentence_steps_match_exhaustive_search,
    lambda: pins.test_constraints_match_exhaustive_search((0, 1, 3)),
    lambda: pins.test_eos_backup_stack(False),
    pins.test_early_pruning_hand_example,
    lambda: pins.test_early_pruning_admissible_for_monotone_scores(4, 3, 16, 36),
]


def _drop_theta0(orig):
    return lambda self, h, V, th: orig(self, h, V, th) - th[0]


def _history_off_by_one(orig):
    return lambda self, h, V, th: orig(self, tuple(h)[:-1], V, th)


def _unigram_only(orig):
    return lambda self, h, V, th: orig(self, (), V, th)


def _rolled_weights(orig):
    return lambda W, h, bias=None: orig(np.roll(np.asarray(W), 1, axis=0), h, bias)


def _transposed_hidden(orig):
    return lambda W, h, bias=None: orig(W, np.asarray(h)[:, ::-1], bias)


def _no_normaliser(orig):
    return lambda x: np.asarray(x, dtype=np.float64) - np.max(x, axis=-1, keepdims=True)


def _negated_lambda(orig):
    def init(self, V, K, lam, *a, **kw):
        orig(self, V, K, -lam, *a, **kw)
    return init


def _all_slots_live(orig):
    def reset(self):
        orig(self)
        self.q[:] = 0.0
    return reset


def _eos_not_masked(orig):
    def step(self, logits, eos_bias=None, allowed=None):
        rec = orig(self, logits, eos_bias, allowed)
        for b in range(self.B):
            for j in range(self.K):
                if rec.token[b, j] == self.eos and np.isfinite(rec.qhat[b, j]):
                    self.q[b, j] = rec.qhat[b, j]
        return rec
    return step


def _ascending_ties_reversed(orig):
    def topk(scores, k):
        s = np.asarray(scores, dtype=np.float64)
        n = s.shape[0]
        order = np.lexsort((-np.arange(n), -s))
        return order[:k]
    return topk


def _finish_drops_live(orig):
    def finished(self, b):
        return list(self.F[b])
    return finished


def _length_off_by_one(orig):
    def rank(self, e):
        t, j, score = e
        return (-(score / (t + 1) if self.length_norm else score), t, j)
    return rank


def _constraint_ignored(orig):
    def step(self, logits, eos_bias=None, allowed=None):
        return orig(self, logits, eos_bias, None)
    return step


def _steps_ignored(orig):
    def init(self, *a, **kw):
        kw.pop("steps", None)
        orig(self, *a, **kw)
    return init


def _backup_wrong_parent(orig):
    def best(self, b):
        h = orig(self, b)
        if h is not None and not self.finished(b) and self.finish == "eos_backup":
            return ob.Hypothesis(self.traceback(b, h.t, h.j), h.score, h.t, h.j)
        return h
    return best


def _prune_sign_flipped(orig):
    def prune(self, b, t, fbest):
        for j in range(self.K):
            if self.q[b, j] > NEG_INF and self._value((t, j, self.q[b, j])) > fbest - self.prune:
                self.q[b, j] = NEG_INF
    return prune


def _prune_late(orig):
    def prune(self, b, t, fbest):
        earlier = [self._value(e) for e in self.F[b] if e[0] < t]
        orig(self, b, t, max(earlier) if earlier else NEG_INF)
    return prune


def _prune_raw_values(orig):
    def prune(self, b, t, fbest):
        for j in range(self.K):
            if self.q[b, j] > NEG_INF and self.q[b, j] < fbest - self.prune:
                self.q[b, j] = NEG_INF
    return prune


MUTATIONS = {
    "drop_theta0": (ob.Posteriors, "lmbr_row", _drop_theta0),
    "history_off_by_one": (ob.Posteriors, "lmbr_row", _history_off_by_one),
    "unigram_only": (ob.Posteriors, "lmbr_row", _unigram_only),
    "rolled_weights": (ob, "project", _rolled_weights),
    "transposed_hidden": (ob, "project", _transposed_hidden),
    "no_normaliser": (ob, "log_softmax", _no_normaliser),
    "negated_lambda": (ob.Decoder, "__init__", _negated_lambda),
    "all_slots_live": (ob.Decoder, "reset", _all_slots_live),
    "eos_not_masked": (ob.Decoder, "step", _eos_not_masked),
    "ties_reversed": (ob, "top_k_total_order", _ascending_ties_reversed),
    "finish_drops_live": (ob.Decoder, "finished", _finish_drops_live),
    "length_off_by_one": (ob.Decoder, "_rank", _length_off_by_one),
    "constraint_ignored": (ob.Decoder, "step", _constraint_ignored),
    "steps_ignored": (ob.Decoder, "__init__", _steps_ignored),
    "backup_wrong_parent": (ob.Decoder, "best", _backup_wrong_parent),
    "prune_sign_flipped": (ob.Decoder, "_prune", _prune_sign_flipped),
    "prune_late": (ob.Decoder, "_prune", _prune_late),
    "prune_raw_values": (ob.Decoder, "_prune", _prune_raw_values),
}


@pytest.mark.slow
@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name, monkeypatch):
    owner, attr, make = MUTATIONS[name]
    bad = make(getattr(owner, attr))
    monkeypatch.setattr(owner, attr, bad)
    if owner is ob and hasattr(oracle, attr):             # names re-exported by the package
        monkeypatch.setattr(oracle, attr, bad)
    caught = []
    for pin in PINS:
        try:
            pin()
        except Exception:                              # any failing pin counts
            caught.append(getattr(pin, "__name__", "lambda"))
            break
    assert caught, f"no pin failed with the planted mistake {name!r}"
