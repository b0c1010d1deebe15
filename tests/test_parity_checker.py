"""The GPU parity checker itself (tests/gpu_util.check_selection), on the CPU.

A selection made by the oracle's own TopB passes; plausible kernel mistakes
planted into a copy of it -- a wrong candidate at a near-tie boundary, a
candidate outside the top K, a repeated pick, a wrong score, a dropped slot,
swapped slots, a NaN -- are each rejected.
"""
import numpy as np
import pytest

import synth
from oracle.beam import Decoder, Posteriors, synthetic_logits
from tests import gpu_util as G


@pytest.fixture(scope="module")
def step_record():
    cfg = synth.get_config("tiny").replace(V=400, H=32, T=4, paths=8, path_len=6)
    W64 = synth.bf16_to_f32(synth.make_weights(cfg)).astype(np.float64)
    dec = Decoder(cfg.V, cfg.K, cfg.lam, cfg.theta, [Posteriors(*synth.posteriors(cfg, 0))], keep_cand=True)
    for _ in range(3):
        rec = dec.step(synthetic_logits(cfg, [0], dec, W64))
    return rec


def _sel(rec):
    return rec.parent[0].copy(), rec.token[0].copy(), rec.qhat[0].copy()


def test_oracle_selection_passes(step_record):
    G.compare_step(step_record, 0, *_sel(step_record))


def _near_tie(rec, delta):
    """A copy of the step whose K-th candidate has a rival delta below it,
    outside the selections."""
    cand = rec.cand[0].copy()
    p, t, q = _sel(rec)
    K, V = cand.shape
    flat = cand.ravel()
    order = np.lexsort((np.arange(flat.size), -flat))
    rival = order[K]                                  # the (K+1)-th candidate
    flat[rival] = flat[order[K - 1]] - delta
    top = np.sort(flat)[::-1][:K + 1]
    return cand, top, rival, p, t, q


def test_rejects_pick_outside_top_k_at_a_near_tie(step_record):
    """The hole of a check that only compares sets at decisive gaps: the GPU
    takes a candidate far below the K-th while the K/K+1 gap is tiny."""
    cand, top, rival, p, t, q = _near_tie(step_record, 5e-4)
    K, V = cand.shape
    flat = cand.ravel()
    order = np.lexsort((np.arange(flat.size), -flat))
    far = order[K + 5]
    p[K - 1], t[K - 1], q[K - 1] = far // V, far % V, flat[far]
    with pytest.raises(AssertionError):
        G.check_selection(cand, top, p, t, q)
    # taking the near-tied rival instead is a valid TopB
    p[K - 1], t[K - 1], q[K - 1] = rival // V, rival % V, flat[rival]
    G.check_selection(cand, top, p, t, q)


@pytest.mark.parametrize("mistake", ["repeat", "score", "dead", "swap_far", "nan", "range"])
def test_rejects_planted_mistakes(step_record, mistake):
    rec = step_record
    cand, top = rec.cand[0], rec.top[0]
    p, t, q = _sel(rec)
    K = len(p)
    if mistake == "repeat":
        p[1], t[1] = p[0], t[0]
    elif mistake == "score":
        q[2] += 2e-3
    elif mistake == "dead":
        q[K - 1] = float("-inf")
    elif mistake == "swap_far":                      # best slot swapped with the worst
        assert top[0] - top[K - 1] > G.GAP
        p[[0, K - 1]], t[[0, K - 1]], q[[0, K - 1]] = p[[K - 1, 0]], t[[K - 1, 0]], q[[K - 1, 0]]
    elif mistake == "nan":
        q[0] = float("nan")
    elif mistake == "range":
        t[0] = cand.shape[1]
    with pytest.raises(AssertionError):
        G.check_selection(cand, top, p, t, q)
