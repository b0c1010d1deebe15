"""fp64 CPU oracle for batched beam decoding with LMBR n-gram posteriors.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or run
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` use it.  It shares no code with the HIP library; its only
inputs are the seeded workload arrays of ``synth``.

What it follows (Iglesias et al., "Accelerating NMT Batched Beam Decoding with
LMBR Posteriors for Deployment", NAACL-HLT 2018):

* Eq. 1: the NMT score of a hypothesis is the sum of per-step log-probabilities;
  the per-step distribution is a softmax over the V logits of the model.
* Eq. 2: LMBR decoding adds, per generated word y_t, the term
  L = theta0 + sum_{n=1..4} theta_n * P_LMBR(n-gram ending in y_t), read from
  n-gram posteriors of an evidence space.
* Algorithm 1 (DecodeNMT) with the sentence-batching changes of Section 3.1:
  per step, score B x V candidates, add the running scores, keep the top B
  (per sentence), realign the state by backpointer, push EOS candidates to the
  finished set F and mask them, and at the end trace back the best entry of F.

Readings where the paper is silent or garbled (each is exercised by a test):
  A1  score = log P_NMT + lambda * L (the paper puts its weight on the NMT
      term; selections are identical with lambda = 1/lambda_paper, see
      ``Decoder(form="paper")``).
  A2  order n covers the last n words (n = 1..4); its history is n-1 words.
  A3  orders needing more history than exists contribute nothing.
  A4  q_0 = (0, -inf, ..., -inf): only slot 0 is live at the first step.
  A5  top-K order: score descending, then flat index k*V + y ascending.
  A6  a -inf candidate that is EOS is never added to F.
  A7  slots still live after the last step join F with their score.
  A8  optional length normalisation in GetBestHypothesis: F is ranked by
      score / t, a hypothesis of step t holding t words (EOS included).
  A9  F order: score descending, then step ascending, then slot ascending.
  A10 an F entry keeps the score it had when pushed.
  A16 the forced-EOS bias is added to the EOS logit before the log-softmax.
  A19 top-K, then realign, then EOS masking (the order Algorithm 1 prints).
  A20 a per-sentence T_s (Section 3.1, item 4): after step T_s the sentence's
      live slots finish (under A7) and the sentence stops.
  A21 a constraint is a set of allowed words per sentence; the others are set
      to -inf among the candidates before TopB (Section 3, note 2), after the
      log-softmax, which stays over all V words.
  A22 the backoff of Section 3, note 5: every finite EOS candidate of a live
      slot that TopB does not keep is recorded (step t, parent slot k, score);
      with this finish mode only EOS hypotheses finish, and when F is empty
      GetBestHypothesis returns the best recorded one (same order as F).
  A23 early pruning (Section 4.3 runs the deployed systems with an early
      pruning width of 0.01, after the methods it cites; the paper gives no
      procedure): per sentence, the best finished value so far (score, or
      score per word under A8) is tracked; after a step's EOS push every live
      slot whose value is below that best minus a width delta is dropped
      (neither expanded nor finished).  delta is in the score's natural-log
      units; the paper's 0.01 is read as a probability ratio, delta = ln 100.
Parity against the paper's own numbers is unpinned: the paper prints no worked
example; the pins are closed forms, special cases and brute force.
"""
from .beam import (Decoder, Posteriors, StepRecord, log_softmax, project,
                   top_k_total_order, NEG_INF)

__all__ = ["Decoder", "Posteriors", "StepRecord", "log_softmax", "project",
           "top_k_total_order", "NEG_INF"]
