"""Plain fp64 oracle of Algorithm 1 (DecodeNMT) with sentence batching.

Test infrastructure only (see the package docstring): written for a reader to
check against the paper by eye, not for speed.  Every array here is float64;
the model inputs (bf16 hidden states and weights, fp32 posteriors) are widened
exactly before use.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

NEG_INF = float("-inf")


# --------------------------------------------------------------------------
# f_NMT's output layer and Eq. 1's per-step log-probabilities
# --------------------------------------------------------------------------
def project(W: np.ndarray, h: np.ndarray, bias: Optional[np.ndarray] = None) -> np.ndarray:
    """Logits of the model's output layer: x[m, v] = sum_i h[m, i] * W[v, i] + bias[v].

    W is [V, H], h is [M, H]; the result is the B x V score matrix P_t of
    Algorithm 1 before normalisation (Section 3: f_NMT returns log-probabilities
    for every word of the vocabulary given each live hypothesis)."""
    x = np.asarray(h, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T
    if bias is not None:
        x = x + np.asarray(bias, dtype=np.float64)[None, :]
    return x


def log_softmax(x: np.ndarray) -> np.ndarray:
    """log P_NMT(y | history) for every y: x - logsumexp(x) along the last axis (Eq. 1)."""
    x = np.asarray(x, dtype=np.float64)
    m = np.max(x, axis=-1, keepdims=True)
    return x - (m + np.log(np.sum(np.exp(x - m), axis=-1, keepdims=True)))


# --------------------------------------------------------------------------
# The LMBR term of Eq. 2
# --------------------------------------------------------------------------
class Posteriors:
    """n-gram posteriors P_LMBR(u | evidence) of one sentence (Eq. 2).

    Built from a list of (order, tokens, posterior): ``prob`` is the plain
    n-gram -> posterior map; ``successors`` indexes it by history so that a
    whole row of the matrix L (Section 2: one row per n-gram history, one
    column per vocabulary word) is formed with a few vector adds."""

    def __init__(self, order=None, tokens=None, post=None):
        self.p: Dict[Tuple[int, ...], float] = {}
        self.successors: Dict[Tuple[int, ...], Tuple[np.ndarray, np.ndarray]] = {}
        if order is None:
            return
        lists: Dict[Tuple[int, ...], Tuple[list, list]] = {}
        for n, t, p in zip(np.asarray(order).tolist(), np.asarray(tokens).tolist(),
                           np.asarray(post, dtype=np.float32).tolist()):
            gram = tuple(int(w) for w in t[:n])
            if gram in self.p:
                raise ValueError(f"duplicate n-gram {gram}")
            self.p[gram] = float(p)
            hist, word = gram[:-1], gram[-1]
            lists.setdefault(hist, ([], []))
            lists[hist][0].append(word)
            lists[hist][1].append(float(p))
        for hist, (ws, ps) in lists.items():
            self.successors[hist] = (np.asarray(ws, dtype=np.int64),
                                     np.asarray(ps, dtype=np.float64))

    def prob(self, gram: Sequence[int]) -> float:
        """P_LMBR of one n-gram; 0 when the evidence space does not contain it."""
        return self.p.get(tuple(gram), 0.0)

    def lmbr_row(self, hist: Sequence[int], V: int, theta: Sequence[float]) -> np.ndarray:
        """L(h, y) for every word y after history h (Eq. 2's overbraced term).

        L(h, y) = theta0 + sum_{n=1..4} theta_n * P_LMBR(last n-1 words of h, y).
        An order whose history is longer than h contributes nothing (A3)."""
        row = np.full(V, float(theta[0]), dtype=np.float64)
        for n in range(1, 5):
            if len(hist) < n - 1:
                continue
            ctx = tuple(hist[len(hist) - (n - 1):]) if n > 1 else ()
            hit = self.successors.get(ctx)
            if hit is None:
                continue
            words, probs = hit
            row[words] += float(theta[n]) * probs
        return row


# --------------------------------------------------------------------------
# TopB (Algorithm 1) with a total order
# --------------------------------------------------------------------------
def top_k_total_order(scores: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k best entries: score descending, then index ascending (A5).

    -inf entries rank after every finite one, among themselves by index."""
    scores = np.asarray(scores, dtype=np.float64)
    n = scores.shape[0]
    if k >= n:
        cand = np.arange(n)
    else:
        kth = np.partition(scores, n - k)[n - k]          # k-th largest value
        cand = np.nonzero(scores >= kth)[0]               # keeps every tie
    order = np.lexsort((cand, -scores[cand]))
    return cand[order][:k]


# --------------------------------------------------------------------------
# Algorithm 1 with sentence batching
# --------------------------------------------------------------------------
@dataclasses.dataclass
class StepRecord:
    """What one step of Algorithm 1 produced, per sentence b and slot j."""
    t: int                    # 1-based step
    parent: np.ndarray        # [B, K] backpointer b_t (row of the parent slot)
    token: np.ndarray         # [B, K] word y_t
    qhat: np.ndarray          # [B, K] cumulative score before EOS masking
    top: np.ndarray           # [B, K+1] best candidate scores, descending
    inc: np.ndarray           # [B, K] score added at this step (lp + lambda * L)
    fbest: Optional[np.ndarray] = None   # [B] best finished value so far (early pruning, A23)
    cand: Optional[np.ndarray] = None    # [B, K, V] every candidate score q + lp + lam*L
                                         # (-inf for dead slots and masked words); kept by
                                         # Decoder(keep_cand=True) for the latest step only

    def gap_k(self) -> np.ndarray:
        """Per sentence: K-th minus (K+1)-th best candidate score."""
        K = self.parent.shape[1]
        a, b = self.top[:, K - 1], self.top[:, K]
        out = np.zeros_like(a)                       # no finite K-th candidate: no gap
        fin = np.isfinite(a)
        out[fin] = a[fin] - b[fin]                    # b = -inf gives +inf
        return out


@dataclasses.dataclass
class Hypothesis:
    tokens: Tuple[int, ...]   # y_1 .. y_t, EOS included when it ended on EOS
    score: float
    t: int                    # step of the F entry
    j: int                    # slot of the F entry


class Decoder:
    """DecodeNMT(x, L) of Algorithm 1 for a batch of sentences (Section 3.1).

    ``form="baseline"``: candidate = q + log P_NMT + lam * L.
    ``form="paper"``:    candidate = q + L + lam * log P_NMT (Eq. 2 as printed).

    Options (the optional parts Section 3 and 3.1 name):
    ``length_norm``: GetBestHypothesis ranks by score / length (A8).
    ``finish="at_T"``: slots still live after the last step are finished (A7);
    ``finish="eos_backup"``: only EOS hypotheses finish, and when none survived
    TopB the best EOS candidate that did not survive is returned (A22).
    ``steps``: a per-sentence number of steps T_s (A20).
    ``step(..., allowed=...)``: a constraint mask applied to the candidates
    before TopB (A21).
    ``prune``: early pruning width delta >= 0 (A23): after a step's EOS push,
    live slots whose value (score, or score per word) is below the best
    finished value so far minus delta are dropped.
    ``keep_cand``: the latest StepRecord also holds every candidate score of
    the step (older records drop theirs, so memory stays at one step).
    ``step(..., force=...)``: the slots' (parent, word) are taken from the
    caller instead of TopB (to follow another decoder's choices); the scores,
    F, realignment and masking are the oracle's own, and ``top`` still lists
    the oracle's own best candidates."""

    def __init__(self, V: int, K: int, lam: float, theta: Sequence[float],
                 tables: Sequence[Optional[Posteriors]], eos: int = 1,
                 form: str = "baseline", length_norm: bool = False, finish: str = "at_T",
                 steps: Optional[Sequence[int]] = None, prune: Optional[float] = None,
                 keep_cand: bool = False):
        if form not in ("baseline", "paper"):
            raise ValueError(form)
        if finish not in ("at_T", "eos_backup"):
            raise ValueError(finish)
        self.V, self.K, self.lam = int(V), int(K), float(lam)
        self.theta = tuple(float(x) for x in theta)
        self.tables = list(tables)
        self.B = len(self.tables)
        self.eos = int(eos)
        self.form = form
        self.length_norm = bool(length_norm)
        self.finish = finish
        self.steps = None if steps is None else [int(x) for x in steps]
        if self.steps is not None and len(self.steps) != self.B:
            raise ValueError("steps needs one entry per sentence")
        if prune is not None and not prune >= 0:
            raise ValueError("prune must be >= 0")
        self.prune = None if prune is None else float(prune)
        self.keep_cand = bool(keep_cand)
        self.reset()

    def reset(self):
        B, K = self.B, self.K
        self.t = 0
        self.q = np.full((B, K), NEG_INF)                 # q_0 = (0, -inf, ...), A4
        self.q[:, 0] = 0.0
        self.hist: List[List[Tuple[int, ...]]] = [[()] * K for _ in range(B)]
        self.F: List[List[Tuple[int, int, float]]] = [[] for _ in range(B)]
        # EOS candidates of live slots that TopB did not keep: (step, parent slot, score)
        self.backup: List[List[Tuple[int, int, float]]] = [[] for _ in range(B)]
        self.records: List[StepRecord] = []

    # -- one iteration of the loop body of Algorithm 1 ----------------------
    def step(self, logits: np.ndarray, eos_bias: Optional[np.ndarray] = None,
             allowed: Optional[np.ndarray] = None,
             force: Optional[Tuple[np.ndarray, np.ndarray]] = None) -> StepRecord:
        """Consume P_t's logits ([B*K, V], row b*K + k) and advance one step.

        ``allowed`` (bool [B, V]) masks candidates out before TopB (A21).
        ``force`` = (parent, word), int [B, K] each: the selections of the
        step, in slot order, instead of the oracle's TopB."""
        B, K, V = self.B, self.K, self.V
        t = self.t + 1
        x = np.array(logits, dtype=np.float64).reshape(B, K, V)
        if eos_bias is not None:                          # A16: before the softmax
            x[:, :, self.eos] += np.asarray(eos_bias, dtype=np.float64)[:, None]
        lp = log_softmax(x)

        parent = np.zeros((B, K), dtype=np.int64)
        token = np.zeros((B, K), dtype=np.int64)
        qhat = np.full((B, K), NEG_INF)
        inc = np.full((B, K), NEG_INF)
        ntop = min(K + 1, K * V)
        top = np.full((B, K + 1), NEG_INF)
        fbest = np.full(B, NEG_INF)
        all_cand = np.full((B, K, V), NEG_INF) if self.keep_cand else None
        for b in range(B):
            cand = np.full((K, V), NEG_INF)
            step_inc = np.full((K, V), NEG_INF)
            for k in range(K):
                if self.q[b, k] == NEG_INF:               # dead slot: no expansions
                    continue
                table = self.tables[b]
                if table is None:
                    L = np.full(V, self.theta[0])
                else:
                    L = table.lmbr_row(self.hist[b][k], V, self.theta)
                if self.form == "baseline":
                    step_inc[k] = lp[b, k] + self.lam * L
                else:
                    step_inc[k] = L + self.lam * lp[b, k]
                cand[k] = self.q[b, k] + step_inc[k]     # P_t + q'_{t-1}
            if allowed is not None:                       # constraint before TopB (A21)
                cand[:, ~np.asarray(allowed[b], dtype=bool)] = NEG_INF
            if all_cand is not None:
                all_cand[b] = cand
            flat = cand.reshape(-1)
            sel = top_k_total_order(flat, ntop)           # TopB
            top[b, :ntop] = flat[sel]
            sel = sel[:K]
            if force is not None:                         # another decoder's choices
                sel = (np.asarray(force[0][b], dtype=np.int64) * V +
                       np.asarray(force[1][b], dtype=np.int64))
            if self.finish == "eos_backup":               # EOS candidates TopB dropped (A22)
                kept = set(int(i) for i in sel)
                for k in range(K):
                    c = cand[k, self.eos]
                    if c > NEG_INF and k * V + self.eos not in kept:
                        self.backup[b].append((t, k, float(c)))
            parent[b] = sel // V
            token[b] = sel % V
            qhat[b] = flat[sel]
            inc[b] = step_inc.reshape(-1)[sel]
            # realign the histories with the survivors (GetMatrixByRows(S_t, b_t))
            self.hist[b] = [self.hist[b][int(parent[b, j])] + (int(token[b, j]),)
                            for j in range(K)]
            # EOS candidates go to F with their score, then are masked (A6, A10)
            for j in range(K):
                if token[b, j] == self.eos and qhat[b, j] > NEG_INF:
                    self.F[b].append((t, j, float(qhat[b, j])))
                    self.q[b, j] = NEG_INF
                else:
                    self.q[b, j] = qhat[b, j]
            # early pruning (A23): drop the live slots that fall more than
            # prune below the best finished hypothesis so far
            if self.F[b]:
                fbest[b] = max(self._value(e) for e in self.F[b])
            if self.prune is not None:
                self._prune(b, t, fbest[b])
            # the sentence's last step (A20): its live slots finish now (A7), or
            # simply stop (A22)
            if self.steps is not None and t == self.steps[b]:
                for j in range(K):
                    if self.q[b, j] > NEG_INF:
                        if self.finish == "at_T":
                            self.F[b].append((t, j, float(self.q[b, j])))
                        self.q[b, j] = NEG_INF
        rec = StepRecord(t, parent, token, qhat, top, inc, fbest, all_cand)
        if self.records:
            self.records[-1].cand = None                  # one step of candidates at a time
        self.records.append(rec)
        self.t = t
        return rec

    def _prune(self, b: int, t: int, fbest: float):
        """Early pruning (A23) of sentence b after step t's EOS push: a live
        slot whose value is below fbest - prune is dropped."""
        for j in range(self.K):
            if self.q[b, j] > NEG_INF and self._value((t, j, self.q[b, j])) < fbest - self.prune:
                self.q[b, j] = NEG_INF

    # -- end of decoding ----------------------------------------------------
    def finished(self, b: int) -> List[Tuple[int, int, float]]:
        """F_b after the last step: pushed EOS entries plus, with finish="at_T",
        the slots still live (A7)."""
        out = list(self.F[b])
        if self.finish == "at_T":
            for j in range(self.K):
                if self.q[b, j] > NEG_INF:
                    out.append((self.t, j, float(self.q[b, j])))
        return out

    def _value(self, e: Tuple[int, int, float]) -> float:
        """What GetBestHypothesis maximises for an entry (t, j, score): the
        score, or the score per word (A8); a hypothesis of step t holds t words."""
        t, _, score = e
        return score / t if self.length_norm else score

    def _rank(self, e: Tuple[int, int, float]) -> Tuple[float, int, int]:
        """Sort key of an entry (t, j, score): best first (A8, A9)."""
        t, j, _ = e
        return (-self._value(e), t, j)

    def traceback(self, b: int, t: int, j: int) -> Tuple[int, ...]:
        """Follow the backpointers b and words y from (t, j) to the start."""
        out = []
        while t >= 1:
            rec = self.records[t - 1]
            out.append(int(rec.token[b, j]))
            j = int(rec.parent[b, j])
            t -= 1
        return tuple(reversed(out))

    def best(self, b: int) -> Optional[Hypothesis]:
        """GetBestHypothesis(F_b, b, y) (A8, A9); with finish="eos_backup" and
        no finished hypothesis, the best non-surviving EOS candidate (A22),
        whose slot is the parent it would have extended."""
        F = self.finished(b)
        if F:
            t, j, score = min(F, key=self._rank)
            return Hypothesis(self.traceback(b, t, j), score, t, j)
        if self.finish == "eos_backup" and self.backup[b]:
            t, k, score = min(self.backup[b], key=self._rank)
            return Hypothesis(self.traceback(b, t - 1, k) + (self.eos,), score, t, k)
        return None


# --------------------------------------------------------------------------
# The synthetic workload: decode with the hashed stand-in model
# --------------------------------------------------------------------------
def synthetic_logits(cfg, sentences: Sequence[int], dec: Decoder, W64: np.ndarray,
                     bias: Optional[np.ndarray] = None) -> np.ndarray:
    """Logits [B*K, V] of the stand-in model for every live slot (dead rows are 0)."""
    import synth
    B, K, V = dec.B, dec.K, dec.V
    rows, hh = [], []
    for b, s in enumerate(sentences):
        for k in range(K):
            if dec.q[b, k] > NEG_INF:
                rows.append(b * K + k)
                hh.append(synth.history_hash(cfg, s, dec.hist[b][k]))
    out = np.zeros((B * K, V), dtype=np.float64)
    if rows:
        h = synth.bf16_to_f32(synth.hidden_from_hashes(np.asarray(hh, dtype=np.uint64), cfg.H))
        out[rows] = project(W64, h.astype(np.float64), bias)
    return out


def decode_synthetic(cfg, sentences: Sequence[int], W_bits: np.ndarray,
                     tables: Sequence[Optional[Posteriors]], T: Optional[int] = None,
                     lam: Optional[float] = None, form: str = "baseline",
                     K: Optional[int] = None, allowed: Optional[np.ndarray] = None,
                     **options) -> Decoder:
    """Run T steps of Algorithm 1 on the synthetic model for the given sentences.

    ``allowed`` (bool [len(sentences), V]) is the constraint of every step;
    ``options`` go to the Decoder (length_norm, finish, steps, prune)."""
    import synth
    T = cfg.T if T is None else T
    K = cfg.K if K is None else K
    dec = Decoder(cfg.V, K, cfg.lam if lam is None else lam, cfg.theta, tables, form=form, **options)
    W64 = synth.bf16_to_f32(W_bits).astype(np.float64)
    for t in range(1, T + 1):
        x = synthetic_logits(cfg, sentences, dec, W64)
        bias = np.array([synth.eos_bias(cfg, t, s) for s in sentences], dtype=np.float64)
        dec.step(x, bias if np.any(bias != 0) else None, allowed)
    return dec
