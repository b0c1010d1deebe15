"""Pins of the fp64 oracle against closed forms, special cases and brute force.

No GPU.  Each test checks the oracle against something other than itself:
hand-derived values (tests/golden), textbook routines written here from their
definitions (plain beam search, greedy search, exhaustive search, a scalar
scorer of whole sequences), and invariants the paper states.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth
from oracle.beam import Decoder, Posteriors, decode_synthetic, synthetic_logits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
NEG_INF = float("-inf")


def tiny_cfg(index, V, H, T, K, paths=6, path_len=4, lam=1.0, theta=synth.THETA, B=1):
    return synth.Config(f"t{index}", index, B=B, K=K, V=V, H=H, T=T, lam=lam, theta=theta,
                        paths=paths, path_len=path_len, zipf_a=1.1)


def tables_for(cfg, sentences):
    return [Posteriors(*synth.posteriors(cfg, s)) for s in sentences]


# --------------------------------------------------------------------------
# A scalar scorer of a whole hypothesis, written from Eq. 1 and Eq. 2
# --------------------------------------------------------------------------
def scalar_logits(cfg, s, hist, W64):
    h = synth.bf16_to_f32(synth.hidden_state(cfg, s, hist)).astype(np.float64)
    return [math.fsum(float(W64[v, i]) * float(h[i]) for i in range(cfg.H)) for v in range(cfg.V)]


def sequence_score(cfg, s, seq, W64, ngrams, lam=None, form="baseline", eos_bias=None):
    """sum_t [log P_NMT(y_t | y_<t) + lam * (theta0 + sum_n theta_n P(y_{t-n+1..t}))]."""
    lam = cfg.lam if lam is None else lam
    total = []
    for t in range(1, len(seq) + 1):
        x = scalar_logits(cfg, s, seq[:t - 1], W64)
        if eos_bias is not None:
            x[1] += eos_bias(t, s)
        m = max(x)
        lse = m + math.log(math.fsum(math.exp(v - m) for v in x))
        lp = x[seq[t - 1]] - lse
        L = cfg.theta[0] + sum(cfg.theta[n] * ngrams.get(tuple(seq[t - n:t]), 0.0)
                               for n in range(1, 5) if t >= n)
        total.append(lp + lam * L if form == "baseline" else L + lam * lp)
    return math.fsum(total)


# --------------------------------------------------------------------------
# Eq. 1 building blocks
# --------------------------------------------------------------------------
def test_projection_matches_scalar_loop():
    cfg = tiny_cfg(20, V=7, H=8, T=1, K=2)
    W64 = synth.bf16_to_f32(synth.make_weights(cfg)).astype(np.float64)
    h = synth.bf16_to_f32(synth.hidden_state(cfg, 0, (3, 4))).astype(np.float64)
    x = oracle.project(W64, h[None, :])[0]
    ref = [math.fsum(W64[v, i] * h[i] for i in range(cfg.H)) for v in range(cfg.V)]
    assert np.allclose(x, ref, rtol=0, atol=1e-13)
    bias = np.arange(cfg.V, dtype=np.float64)
    assert np.allclose(oracle.project(W64, h[None, :], bias)[0], np.array(ref) + bias, atol=1e-13)


def test_log_softmax_rows_sum_to_one():
    rng = np.random.default_rng(3)
    for scale in [1.0, 30.0, 300.0]:
        x = rng.standard_normal((16, 4000)) * scale
        lp = oracle.log_softmax(x)
        s = np.array([math.fsum(np.exp(r)) for r in lp])
        assert np.all(np.abs(s - 1.0) < 1e-12)
    # against a math.fsum log-sum-exp on short rows
    for row in [[0.0, 0.0, 0.0, 0.0], [1.0, -2.0, 3.5], [1000.0, 999.0, -1000.0]]:
        m = max(row)
        lse = m + math.log(math.fsum(math.exp(v - m) for v in row))
        assert np.allclose(oracle.log_softmax(np.array(row)), [v - lse for v in row], atol=1e-12)
    assert np.allclose(oracle.log_softmax(np.zeros(4)), -math.log(4), atol=1e-15)


# --------------------------------------------------------------------------
# Eq. 2: the LMBR term
# --------------------------------------------------------------------------
def test_lmbr_row_single_path_closed_form():
    g = json.load(open(os.path.join(GOLDEN, "single_path_L.json")))
    path = np.array([g["path"]], dtype=np.int32)
    tabs = Posteriors(*synth.posteriors_from_paths(path, np.array([1.0])))
    assert all(p == 1.0 for p in tabs.p.values())
    V, theta, word = g["V"], g["theta"], g["path"]
    for t, expect in enumerate(g["on_path"], start=1):
        row = tabs.lmbr_row(tuple(word[:t - 1]), V, theta)
        assert abs(row[word[t - 1]] - expect) < 1e-12
        for y in range(V):
            if y == word[t - 1]:
                continue
            want = g["unigram_only"] if y in word else g["off_path"]
            assert abs(row[y] - want) < 1e-12


def test_lmbr_row_matches_ngram_definition():
    cfg = synth.get_config("tiny")
    order, toks, post = synth.posteriors(cfg, 0)
    tab = Posteriors(order, toks, post)
    d = synth.ngram_dict(order, toks, post)
    paths, _ = synth.make_lattice(cfg, 0)
    hists = [(), tuple(paths[0, :1]), tuple(paths[1, :2]), tuple(paths[2, :5]), (999, 998, 997)]
    for h in hists:
        row = tab.lmbr_row(h, cfg.V, cfg.theta)
        for y in range(cfg.V):
            seq = tuple(h) + (y,)
            want = cfg.theta[0] + sum(cfg.theta[n] * d.get(seq[len(seq) - n:], 0.0)
                                      for n in range(1, 5) if len(seq) >= n)
            assert abs(row[y] - want) < 1e-12


# --------------------------------------------------------------------------
# Algorithm 1 against a hand-derived example
# --------------------------------------------------------------------------
def test_hand_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    order = [len(u) for u, _ in g["ngrams"]]
    toks = [list(u) + [-1] * (4 - len(u)) for u, _ in g["ngrams"]]
    post = np.array([p for _, p in g["ngrams"]], dtype=np.float32)
    tab = Posteriors(np.array(order), np.array(toks), post)
    dec = Decoder(g["V"], g["K"], g["lambda"], g["theta"], [tab], eos=g["eos"])
    for want in g["steps"]:
        rec = dec.step(np.zeros((g["K"], g["V"])))
        assert rec.parent[0].tolist() == want["parent"]
        assert rec.token[0].tolist() == want["token"]
        assert np.allclose(rec.qhat[0], want["qhat"], atol=g["tol"], rtol=0)
    best = dec.best(0)
    assert list(best.tokens) == g["best"]["tokens"]
    assert (best.t, best.j) == (g["best"]["t"], g["best"]["j"])
    assert abs(best.score - g["best"]["score"]) < g["tol"]


def test_top_k_total_order():
    s = np.array([1.0, 3.0, 3.0, -np.inf, 2.0, 3.0, -np.inf])
    assert oracle.top_k_total_order(s, 4).tolist() == [1, 2, 5, 4]
    assert oracle.top_k_total_order(s, 7).tolist() == [1, 2, 5, 4, 0, 3, 6]
    allneg = np.full(5, -np.inf)
    assert oracle.top_k_total_order(allneg, 3).tolist() == [0, 1, 2]


# --------------------------------------------------------------------------
# Special cases the paper states, and brute force
# --------------------------------------------------------------------------
def plain_beam(cfg, s, W64, K, T, eos=1):
    """Textbook left-to-right beam search on log P_NMT only (note 1 after Algorithm 1)."""
    slots = [((), 0.0)] + [None] * (K - 1)
    finished = []
    for t in range(1, T + 1):
        cands = []
        for k, sl in enumerate(slots):
            if sl is None:
                continue
            hist, sc = sl
            x = scalar_logits(cfg, s, hist, W64)
            m = max(x)
            lse = m + math.log(math.fsum(math.exp(v - m) for v in x))
            for y in range(cfg.V):
                cands.append((sc + (x[y] - lse), k * cfg.V + y, hist + (y,)))
        cands.sort(key=lambda c: (-c[0], c[1]))
        slots = []
        for j, (sc, _, h) in enumerate(cands[:K]):
            if h[-1] == eos:
                finished.append((sc, t, j, h))
                slots.append(None)
            else:
                slots.append((h, sc))
        slots += [None] * (K - len(slots))
    for j, sl in enumerate(slots):
        if sl is not None:
            finished.append((sl[1], T, j, sl[0]))
    return min(finished, key=lambda e: (-e[0], e[1], e[2]))


def test_lambda_zero_is_plain_nmt_beam_search():
    cfg = tiny_cfg(21, V=9, H=16, T=5, K=3, paths=8, path_len=5)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    for s in range(3):
        dec = decode_synthetic(cfg, [s], W, tables_for(cfg, [s]), lam=0.0)
        best = dec.best(0)
        sc, t, j, h = plain_beam(cfg, s, W64, cfg.K, cfg.T)
        assert best.tokens == h and (best.t, best.j) == (t, j)
        assert abs(best.score - sc) < 1e-9


def test_k1_is_greedy_search():
    cfg = synth.get_config("tiny")
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    order, toks, post = synth.posteriors(cfg, 0)
    d = synth.ngram_dict(order, toks, post)
    dec = decode_synthetic(cfg, [0], W, [Posteriors(order, toks, post)], K=1)
    hist, total = (), 0.0
    for t in range(1, cfg.T + 1):
        x = np.array(scalar_logits(cfg, 0, hist, W64))
        m = x.max()
        lp = x - (m + math.log(math.fsum(np.exp(x - m))))
        inc = [lp[y] + cfg.lam * (cfg.theta[0] + sum(
            cfg.theta[n] * d.get((hist + (y,))[-n:], 0.0) for n in range(1, 5) if t >= n))
            for y in range(cfg.V)]
        y = int(np.argmax(inc))                        # first maximum: lowest word id
        hist, total = hist + (y,), total + inc[y]
        if y == 1:
            break
    best = dec.best(0)
    assert best.tokens == hist
    assert abs(best.score - total) < 1e-9


@pytest.mark.parametrize("V,T,K,index", [(4, 3, 16, 30), (3, 4, 27, 31), (4, 3, 16, 32)])
def test_exhaustive_argmax(V, T, K, index):
    """With K >= V^(T-1) nothing is pruned before the last step, so the beam's
    best equals the argmax of Eq. 2 over every finishable sequence."""
    cfg = tiny_cfg(index, V=V, H=16, T=T, K=K, paths=5, path_len=3)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    order, toks, post = synth.posteriors(cfg, 0)
    d = synth.ngram_dict(order, toks, post)
    dec = decode_synthetic(cfg, [0], W, [Posteriors(order, toks, post)])
    best = dec.best(0)
    seqs = []
    for n in range(1, T + 1):
        for body in itertools.product([v for v in range(V) if v != 1], repeat=n - 1):
            for last in range(V):
                if last == 1 or n == T:
                    seqs.append(body + (last,))
    scored = sorted(((sequence_score(cfg, 0, q, W64, d), q) for q in seqs), key=lambda e: -e[0])
    assert abs(best.score - scored[0][0]) < 1e-9
    assert scored[0][0] - scored[1][0] > 1e-9          # unique argmax in these cases
    assert best.tokens == scored[0][1]


def test_finished_entries_keep_rescorable_scores():
    """F entries are recorded before masking and never change (Algorithm 1's EOS
    loop); re-scoring each traced-back sequence from scratch gives its score."""
    cfg = synth.get_config("tiny").replace(T=10)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    order, toks, post = synth.posteriors(cfg, 0)
    d = synth.ngram_dict(order, toks, post)
    dec = Decoder(cfg.V, cfg.K, cfg.lam, cfg.theta, [Posteriors(order, toks, post)])
    W64d = W64
    snapshots = []
    for t in range(1, cfg.T + 1):
        dec.step(synthetic_logits(cfg, [0], dec, W64d))
        snapshots.append(list(dec.F[0]))
    for a, b in zip(snapshots, snapshots[1:]):
        assert b[:len(a)] == a                         # entries never change
    F = dec.finished(0)
    assert len(F) >= cfg.K
    for t, j, sc in F:
        seq = dec.traceback(0, t, j)
        assert len(seq) == t
        assert abs(sequence_score(cfg, 0, seq, W64, d) - sc) < 1e-9


def test_forced_eos_bias_enters_before_softmax():
    cfg = synth.get_config("base").replace(V=50, H=16, B=2, T=6, eos_boost_from=3,
                                           paths=10, path_len=6)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    dec = decode_synthetic(cfg, [0, 1], W, tables_for(cfg, [0, 1]))
    for b, s in enumerate([0, 1]):
        d = dec.tables[b].p
        for t, j, sc in dec.finished(b):
            seq = dec.traceback(b, t, j)
            want = sequence_score(cfg, s, seq, W64, d, eos_bias=lambda tt, ss: synth.eos_bias(cfg, tt, ss))
            assert abs(want - sc) < 1e-9
    # the boosted odd sentence finishes early with EOS
    assert any(dec.records[t].token[1].tolist().count(1) > 0 for t in range(2, cfg.T))
    # masking stops every EOS hypothesis: no live history and no F entry
    # contains EOS anywhere but at its end
    for b in range(2):
        for j in range(cfg.K):
            if dec.q[b, j] > NEG_INF:
                assert 1 not in dec.hist[b][j]
        for t, j, _ in dec.finished(b):
            assert 1 not in dec.traceback(b, t, j)[:-1]


def test_sentence_batching_is_invariant():
    """Section 3.1 and Section 4.4: batching sentences does not change any
    sentence's translation, in any order."""
    cfg = synth.get_config("tiny").replace(B=4, V=300, H=32, T=8, paths=12, path_len=8)
    W = synth.make_weights(cfg)
    sents = [0, 1, 2, 3]
    together = decode_synthetic(cfg, sents, W, tables_for(cfg, sents))
    perm = [2, 0, 3, 1]
    permuted = decode_synthetic(cfg, perm, W, tables_for(cfg, perm))
    for b, s in enumerate(sents):
        alone = decode_synthetic(cfg, [s], W, tables_for(cfg, [s])).best(0)
        a = together.best(b)
        p = permuted.best(perm.index(s))
        assert a.tokens == alone.tokens == p.tokens
        assert abs(a.score - alone.score) < 1e-12 and abs(p.score - alone.score) < 1e-12
        for ra, rs in zip(together.records, decode_synthetic(cfg, [s], W, tables_for(cfg, [s])).records):
            assert ra.parent[b].tolist() == rs.parent[0].tolist()
            assert ra.token[b].tolist() == rs.token[0].tolist()


def test_empty_table_is_word_penalty():
    """With no posteriors every row of L is theta0 (Section 2): selections equal
    the lambda = 0 search and each F score moves by lambda * theta0 * length."""
    cfg = synth.get_config("tiny").replace(B=2, V=200, H=32, T=8)
    W = synth.make_weights(cfg)
    empty = decode_synthetic(cfg, [0, 1], W, [Posteriors(), Posteriors()])
    nmt = decode_synthetic(cfg, [0, 1], W, [Posteriors(), Posteriors()], lam=0.0)
    for ra, rb in zip(empty.records, nmt.records):
        assert np.array_equal(ra.parent, rb.parent) and np.array_equal(ra.token, rb.token)
    for b in range(2):
        fa, fb = empty.finished(b), nmt.finished(b)
        assert [(t, j) for t, j, _ in fa] == [(t, j) for t, j, _ in fb]
        for (t, j, sa), (_, _, sb) in zip(fa, fb):
            assert abs(sa - (sb + cfg.lam * cfg.theta[0] * t)) < 1e-9


def test_lambda_placement_equivalence():
    """Reading A1: Eq. 2 weights the NMT term by lambda_p; scaling every score by
    1/lambda_p gives log P + (1/lambda_p) L, so selections are identical."""
    cfg = synth.get_config("tiny").replace(B=2, T=10)
    W = synth.make_weights(cfg)
    lam_p = 0.5
    paper = decode_synthetic(cfg, [0, 1], W, tables_for(cfg, [0, 1]), lam=lam_p, form="paper")
    ours = decode_synthetic(cfg, [0, 1], W, tables_for(cfg, [0, 1]), lam=1.0 / lam_p)
    for ra, rb in zip(paper.records, ours.records):
        assert np.array_equal(ra.parent, rb.parent) and np.array_equal(ra.token, rb.token)
        fin = np.isfinite(rb.qhat)
        assert np.allclose(ra.qhat[fin], lam_p * rb.qhat[fin], rtol=1e-12, atol=1e-12)
    for b in range(2):
        assert paper.best(b).tokens == ours.best(b).tokens


def test_beam_invariants_small_config():
    """Live slots hold distinct histories (q_0 reading A4) and slot scores are
    non-increasing in the slot index (TopB order)."""
    cfg = synth.get_config("tiny").replace(B=2, V=500, T=10)
    W = synth.make_weights(cfg)
    dec = Decoder(cfg.V, cfg.K, cfg.lam, cfg.theta, tables_for(cfg, [0, 1]))
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    for t in range(cfg.T):
        rec = dec.step(synthetic_logits(cfg, [0, 1], dec, W64))
        for b in range(2):
            assert np.all(np.diff(rec.qhat[b]) <= 0)
            live = [dec.hist[b][j] for j in range(cfg.K) if dec.q[b, j] > NEG_INF]
            assert len(set(live)) == len(live)
            assert all(len(h) == t + 1 for h in dec.hist[b])
            assert rec.gap_k()[b] >= 0


def test_first_step_expands_only_slot_zero():
    cfg = synth.get_config("tiny")
    W = synth.make_weights(cfg)
    dec = decode_synthetic(cfg, [0], W, tables_for(cfg, [0]), T=1)
    rec = dec.records[0]
    assert rec.parent[0].tolist() == [0] * cfg.K
    assert len(set(rec.token[0].tolist())) == cfg.K


# --------------------------------------------------------------------------
# Decode options (Section 3: optional length normalisation, constraints before
# TopB, the backoff stack of note 5; Section 3.1: per-sentence T)
# --------------------------------------------------------------------------
def _finishable(V, T, allowed=None, eos=1):
    """Every sequence the decoder can finish: EOS-terminated ones of length <= T
    and length-T ones without EOS, over the allowed words."""
    words = [v for v in range(V) if allowed is None or allowed[v]]
    body_words = [v for v in words if v != eos]
    out = []
    for n in range(1, T + 1):
        for body in itertools.product(body_words, repeat=n - 1):
            for last in words:
                if last == eos or n == T:
                    out.append(body + (last,))
    return out


@pytest.mark.parametrize("V,T,K,index", [(4, 3, 16, 30), (3, 4, 27, 31), (4, 3, 16, 32)])
def test_exhaustive_argmax_length_normalised(V, T, K, index):
    """With nothing pruned, GetBestHypothesis with length normalisation is the
    argmax of score / length over every finishable sequence (A8)."""
    cfg = tiny_cfg(index, V=V, H=16, T=T, K=K, paths=5, path_len=3)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    order, toks, post = synth.posteriors(cfg, 0)
    d = synth.ngram_dict(order, toks, post)
    best = decode_synthetic(cfg, [0], W, [Posteriors(order, toks, post)], length_norm=True).best(0)
    scored = sorted(((sequence_score(cfg, 0, q, W64, d), q) for q in _finishable(V, T)),
                    key=lambda e: -e[0] / len(e[1]))
    top, second = scored[0], scored[1]
    assert top[0] / len(top[1]) - second[0] / len(second[1]) > 1e-9
    assert best.tokens == top[1]
    assert abs(best.score - top[0]) < 1e-9
    plain = decode_synthetic(cfg, [0], W, [Posteriors(order, toks, post)]).best(0)
    assert plain.score >= best.score - 1e-12          # the raw-score winner is the plain best


def test_per_sentence_steps_match_exhaustive_search():
    """Sentences with their own T_s (A20): each sentence's best equals the
    argmax over the sequences finishable within its own T_s, and the sentence
    has no live slot after step T_s."""
    V, T, K = 3, 4, 27
    cfg = tiny_cfg(33, V=V, H=16, T=T, K=K, paths=5, path_len=3, B=2)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    steps = [2, 4]
    tabs = tables_for(cfg, [0, 1])
    dec = decode_synthetic(cfg, [0, 1], W, tabs, steps=steps)
    assert np.all(dec.q[0] == NEG_INF)
    for s in (0, 1):
        d = synth.ngram_dict(*synth.posteriors(cfg, s))
        scored = sorted(((sequence_score(cfg, s, q, W64, d), q) for q in _finishable(V, steps[s])),
                        key=lambda e: -e[0])
        best = dec.best(s)
        assert scored[0][0] - scored[1][0] > 1e-9
        assert best.tokens == scored[0][1]
        assert abs(best.score - scored[0][0]) < 1e-9
        assert best.t <= steps[s]


@pytest.mark.parametrize("allowed_words", [(0, 1, 3), (0, 2, 3)])
def test_constraints_match_exhaustive_search(allowed_words):
    """A constraint applied before TopB (A21) restricts the search to the
    allowed words; the log-softmax stays over all V (so the scores are those
    of the unconstrained model).  The second case forbids EOS itself."""
    V, T, K = 4, 3, 16
    cfg = tiny_cfg(34, V=V, H=16, T=T, K=K, paths=5, path_len=3)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    order, toks, post = synth.posteriors(cfg, 0)
    d = synth.ngram_dict(order, toks, post)
    allowed = np.zeros((1, V), dtype=bool)
    allowed[0, list(allowed_words)] = True
    best = decode_synthetic(cfg, [0], W, [Posteriors(order, toks, post)], allowed=allowed).best(0)
    scored = sorted(((sequence_score(cfg, 0, q, W64, d), q) for q in _finishable(V, T, allowed[0])),
                    key=lambda e: -e[0])
    assert scored[0][0] - scored[1][0] > 1e-9
    assert best.tokens == scored[0][1]
    assert abs(best.score - scored[0][0]) < 1e-9
    assert all(allowed[0, w] for w in best.tokens)


@pytest.mark.parametrize("length_norm", [False, True])
def test_eos_backup_stack(length_norm):
    """Section 3, note 5 (A22): with EOS pushed far down it never survives TopB,
    F stays empty, and the result is the best EOS candidate of any live slot
    at any step.  The candidates are re-scored from scratch by the scalar
    scorer along the beam's own trajectory."""
    cfg = tiny_cfg(35, V=6, H=16, T=5, K=3, paths=6, path_len=4).replace(eos_boost=-30.0, eos_boost_from=1)
    s = 1                                               # the EOS bias applies to odd sentences
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    order, toks, post = synth.posteriors(cfg, s)
    d = synth.ngram_dict(order, toks, post)
    dec = decode_synthetic(cfg, [s], W, [Posteriors(order, toks, post)], finish="eos_backup",
                           length_norm=length_norm)
    assert dec.F[0] == [] and dec.finished(0) == []
    ebias = lambda t, ss: synth.eos_bias(cfg, t, ss)
    cands = []
    for t in range(1, cfg.T + 1):
        for k in range(cfg.K):
            if t == 1 and k > 0:
                continue                                # only slot 0 is live at the first step (A4)
            hist = dec.traceback(0, t - 1, k)
            if t > 1 and dec.records[t - 2].qhat[0, k] == NEG_INF:
                continue
            seq = hist + (1,)
            cands.append((sequence_score(cfg, s, seq, W64, d, eos_bias=ebias), t, k, seq))
    key = (lambda c: (-c[0] / c[1], c[1], c[2])) if length_norm else (lambda c: (-c[0], c[1], c[2]))
    want = min(cands, key=key)
    best = dec.best(0)
    assert best.tokens == want[3]
    assert (best.t, best.j) == (want[1], want[2])
    assert abs(best.score - want[0]) < 1e-9


def test_length_normalised_order_hand_example():
    """A8 by hand: a 1-word hypothesis scoring -3 loses to a 2-word one scoring
    -5 per word count (-3/1 < -5/2), but wins on raw score; ties on the
    normalised score go to the earlier step."""
    entries = [(1, 0, -3.0), (2, 1, -5.0), (4, 0, -10.0)]
    norm = Decoder(4, 2, 1.0, synth.THETA, [None], length_norm=True)
    raw = Decoder(4, 2, 1.0, synth.THETA, [None])
    assert min(entries, key=norm._rank) == (2, 1, -5.0)        # -2.5 beats -3 and -2.5 (tie: t=2 < 4)
    assert min(entries, key=raw._rank) == (1, 0, -3.0)


def _prob_log(p):
    return NEG_INF if p is None else math.log(p)


def test_early_pruning_hand_example():
    """A23 by hand (tests/golden/early_pruning.json): pure NMT scores whose
    values are logs of probability products; which slots a width drops right
    after the EOS push of their step, with raw and with per-word values."""
    g = json.load(open(os.path.join(GOLDEN, "early_pruning.json")))
    tol = g["tol"]

    def close(a, b):
        return (a == NEG_INF and b == NEG_INF) or abs(a - b) < tol

    for case in g["cases"]:
        dec = Decoder(g["V"], g["K"], g["lambda"], g["theta"], [None], eos=g["eos"],
                      prune=case["prune"], length_norm=case["length_norm"])
        for probs, want in zip(g["step_probs"], case["steps"]):
            rec = dec.step(np.log(np.tile(np.array(probs, dtype=np.float64), (g["K"], 1))))
            assert rec.parent[0].tolist() == want["parent"]
            assert rec.token[0].tolist() == want["token"]
            assert all(close(a, _prob_log(p)) for a, p in zip(rec.qhat[0], want["qhat_prob"]))
            assert all(close(a, _prob_log(p)) for a, p in zip(dec.q[0], want["q_after_prob"])), \
                (case["prune"], rec.t, dec.q[0])
            fb = math.log(want["fbest_prob"]) / (want["fbest_t"] if case["length_norm"] else 1)
            assert close(rec.fbest[0], fb)
        best = dec.best(0)
        assert list(best.tokens) == case["best"]["tokens"]
        assert (best.t, best.j) == (case["best"]["t"], case["best"]["j"])
        assert close(best.score, math.log(case["best"]["prob"]))


@pytest.mark.parametrize("V,T,K,index", [(4, 3, 16, 36), (3, 4, 27, 37)])
def test_early_pruning_admissible_for_monotone_scores(V, T, K, index):
    """With lambda = 0 every step adds a log-probability <= 0, so no extension
    of a hypothesis below a finished one can overtake it: width-0 pruning (A23)
    with nothing lost to the beam (K >= V^(T-1)) still returns the exhaustive
    argmax, while it does drop live slots."""
    cfg = tiny_cfg(index, V=V, H=16, T=T, K=K, paths=5, path_len=3, lam=0.0)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    order, toks, post = synth.posteriors(cfg, 0)
    d = synth.ngram_dict(order, toks, post)
    dec = Decoder(cfg.V, K, cfg.lam, cfg.theta, [Posteriors(order, toks, post)], prune=0.0)
    dropped = 0
    for t in range(1, T + 1):
        rec = dec.step(synthetic_logits(cfg, [0], dec, W64))
        live_unpruned = np.sum((rec.qhat[0] > NEG_INF) & (rec.token[0] != dec.eos))
        dropped += int(live_unpruned - np.sum(dec.q[0] > NEG_INF))
    assert dropped > 0
    scored = sorted(((sequence_score(cfg, 0, q, W64, d), q) for q in _finishable(V, T)), key=lambda e: -e[0])
    assert scored[0][0] - scored[1][0] > 1e-9
    best = dec.best(0)
    assert best.tokens == scored[0][1]
    assert abs(best.score - scored[0][0]) < 1e-9


# --------------------------------------------------------------------------
# Steering: the oracle following another decoder's choices
# --------------------------------------------------------------------------
def test_forced_own_selections_reproduce_the_decode():
    """Forcing the oracle's own TopB selections changes nothing: every record,
    every F entry and the best hypothesis are identical."""
    cfg = synth.get_config("tiny").replace(B=2, V=200, H=32, T=8, paths=8, path_len=6)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    a = Decoder(cfg.V, cfg.K, cfg.lam, cfg.theta, tables_for(cfg, [0, 1]))
    b = Decoder(cfg.V, cfg.K, cfg.lam, cfg.theta, tables_for(cfg, [0, 1]), keep_cand=True)
    for t in range(1, cfg.T + 1):
        ra = a.step(synthetic_logits(cfg, [0, 1], a, W64))
        rb = b.step(synthetic_logits(cfg, [0, 1], b, W64), force=(ra.parent, ra.token))
        for f in ("parent", "token", "qhat", "top", "inc"):
            assert np.array_equal(getattr(ra, f), getattr(rb, f)), f
        # the kept candidates are the scores TopB ranked: its best K+1, in order
        for s in range(2):
            flat = np.sort(rb.cand[s].ravel())[::-1][:cfg.K + 1]
            assert np.array_equal(flat, rb.top[s])
            assert np.array_equal(rb.cand[s][rb.parent[s], rb.token[s]], rb.qhat[s])
    assert all(r.cand is None for r in b.records[:-1])      # only the latest step keeps them
    for s in range(2):
        assert a.finished(s) == b.finished(s)
        assert a.best(s) == b.best(s)


def test_forced_other_selections_rescore():
    """Forcing choices TopB would not make (each step the candidates ranked
    2..K+1 instead of 1..K): the hypotheses the oracle then holds are scored
    by its own arithmetic, and every F entry re-scores from scratch with the
    scalar scorer to its recorded score."""
    cfg = synth.get_config("tiny").replace(V=60, H=16, T=7, paths=6, path_len=5)
    W = synth.make_weights(cfg)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    order, toks, post = synth.posteriors(cfg, 0)
    d = synth.ngram_dict(order, toks, post)
    dec = Decoder(cfg.V, cfg.K, cfg.lam, cfg.theta, [Posteriors(order, toks, post)], keep_cand=True)
    probe = Decoder(cfg.V, cfg.K, cfg.lam, cfg.theta, [Posteriors(order, toks, post)], keep_cand=True)
    for t in range(1, cfg.T + 1):
        # rank the candidates of the steered state with the oracle's own order
        probe.q, probe.hist, probe.F, probe.t = dec.q.copy(), [list(h) for h in dec.hist], [[]], dec.t
        probe.records = []
        x = synthetic_logits(cfg, [0], dec, W64)
        r = probe.step(x)
        flat = r.cand[0].ravel()
        order_idx = np.lexsort((np.arange(flat.size), -flat))
        pick = order_idx[1:cfg.K + 1]
        if not np.all(np.isfinite(flat[pick])):
            pick = order_idx[:cfg.K]
        rec = dec.step(x, force=(pick[None, :] // cfg.V, pick[None, :] % cfg.V))
        assert np.array_equal(rec.qhat[0], flat[pick])
    F = dec.finished(0)
    assert F
    for t, j, sc in F:
        seq = dec.traceback(0, t, j)
        assert abs(sequence_score(cfg, 0, seq, W64, d) - sc) < 1e-9
