"""Helpers shared by the GPU parity tests: drive the HIP library through its
C ABI on seeded inputs, and compare with the oracle on the same inputs."""
import functools
import json
import math
import os
import sys

import numpy as np

import synth
from oracle.beam import NEG_INF, Decoder, Posteriors, log_softmax, project

SCORE_TOL = 1e-3      # scores of selected hypotheses (the contract's absolute bound)
GAP = 1e-3            # selections must match where the oracle's gap exceeds this


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=8)
def weights(cfg):
    return synth.make_weights(cfg)


@functools.lru_cache(maxsize=4096)
def posteriors(cfg, s):
    return synth.posteriors(cfg, s)


def pack_ctx(hist):
    c = 0
    for y in hist[-3:]:
        c = ((c << 21) | (y + 1)) & ((1 << 63) - 1)
    return c


def as_i64(u):
    u = int(u) & ((1 << 64) - 1)
    return u - (1 << 64) if u >= (1 << 63) else u


class GpuDecoder:
    """A context, a projection, the posterior tables and a beam state on cuda:0."""

    def __init__(self, cfg, K=None, T_max=None, lam=None, tables=None, W=None, path="two_pass", dense=False):
        import torch
        import paper_1804_11324_amd as P
        self.P, self.torch = P, torch
        self.cfg = cfg
        self.K = cfg.K if K is None else K
        self.T_max = cfg.T if T_max is None else T_max
        lam = cfg.lam if lam is None else lam
        self.ccfg = P.make_config(cfg.B, self.K, cfg.V, cfg.H, self.T_max, 1, lam, cfg.theta,
                                  cfg.load_factor)
        self.ctx = P.lmbr_create(self.ccfg)
        Wb = weights(cfg) if W is None else W
        self.W = torch.from_numpy(np.ascontiguousarray(Wb).view(np.int16)).cuda()
        P.lmbr_set_projection(self.ctx, self.W, 0)
        if dense:                                 # tables in the paper's dense arrangement of L
            P.lmbr_set_lmbr_layout(self.ctx, P.LMBR_L_DENSE)
        for s in range(cfg.B):
            o, t, p = posteriors(cfg, s) if tables is None else tables[s]
            P.lmbr_load_posteriors(self.ctx, s, o, t, p)
        self.st = P.BeamState(self.ccfg)
        P.lmbr_state_init(self.ctx, self.st, cfg.seed)
        M = cfg.B * self.K
        self.M = M
        self.hidden = torch.empty((M, cfg.H), dtype=torch.int16, device="cuda")
        self.parent = torch.empty(M, dtype=torch.int32, device="cuda")
        self.token = torch.empty(M, dtype=torch.int32, device="cuda")
        self.score = torch.empty(M, dtype=torch.float64, device="cuda")
        # "two_pass": lmbr_beam_step on the default step path (projection into
        # the context's logits workspace, then the score pass);
        # "fused": lmbr_beam_step on the fused path (one kernel, logits on chip);
        # "logits": lmbr_project into a caller buffer, then lmbr_beam_step_logits
        assert path in ("two_pass", "fused", "logits")
        self.path = path
        if path == "fused":
            P.lmbr_set_step_path(self.ctx, P.LMBR_STEP_FUSED)
        if path == "logits":
            self.ld = (cfg.V + 63) // 64 * 64
            self.logits = torch.empty((M, self.ld), dtype=torch.float32, device="cuda")

    def step(self, eos_bias=None):
        """One step with the built-in stand-in model; returns (parent, token, score) [B, K]."""
        P, torch = self.P, self.torch
        P.lmbr_synth_hidden(self.ctx, self.st, self.hidden)
        eb = None if eos_bias is None else torch.from_numpy(np.asarray(eos_bias, np.float32)).cuda()
        if self.path in ("two_pass", "fused"):
            P.lmbr_beam_step(self.ctx, self.st, self.hidden, eb, self.parent, self.token, self.score)
        else:
            P.lmbr_project(self.ctx, self.hidden, self.logits, self.ld)
            P.lmbr_beam_step_logits(self.ctx, self.st, self.logits, self.ld, eb, self.parent, self.token,
                                    self.score)
        torch.cuda.synchronize()
        B, K = self.cfg.B, self.K
        return (self.parent.cpu().numpy().reshape(B, K), self.token.cpu().numpy().reshape(B, K),
                self.score.cpu().numpy().reshape(B, K))

    def inject(self, dec: Decoder, sentences):
        """Overwrite the GPU state of `sentences` with the oracle's (rows of dec in order)."""
        torch = self.torch
        K = self.K
        q = self.st.q.cpu().numpy()
        ctx = self.st.ctx.cpu().numpy()
        hh = self.st.hhash.cpu().numpy()
        ln = self.st.len.cpu().numpy()
        for b, s in enumerate(sentences):
            for k in range(K):
                row = s * K + k
                hist = dec.hist[b][k]
                q[row] = dec.q[b, k]
                ctx[row] = pack_ctx(hist)
                hh[row] = as_i64(synth.history_hash(self.cfg, s, hist))
                ln[row] = len(hist)
        self.st.q.copy_(torch.from_numpy(q))
        self.st.ctx.copy_(torch.from_numpy(ctx))
        self.st.hhash.copy_(torch.from_numpy(hh))
        self.st.len.copy_(torch.from_numpy(ln))
        self.st.t = dec.t
        self.P.lmbr_state_probe(self.ctx, self.st)
        torch.cuda.synchronize()

    def close(self):
        self.ctx.close()


def oracle_for(cfg, sentences, K=None, lam=None):
    tabs = [Posteriors(*posteriors(cfg, s)) for s in sentences]
    return Decoder(cfg.V, cfg.K if K is None else K, cfg.lam if lam is None else lam, cfg.theta, tabs,
                   keep_cand=True)


def oracle_logits(cfg, sentences, dec, W64):
    """Stand-in model logits for the oracle's live slots ([B*K, V], dead rows 0)."""
    B, K = len(sentences), dec.K
    rows, hh = [], []
    for b, s in enumerate(sentences):
        for k in range(K):
            if dec.q[b, k] > NEG_INF:
                rows.append(b * K + k)
                hh.append(synth.history_hash(cfg, s, dec.hist[b][k]))
    x = np.zeros((B * K, cfg.V))
    if rows:
        h = synth.bf16_to_f32(synth.hidden_from_hashes(np.array(hh, dtype=np.uint64), cfg.H))
        x[rows] = project(W64, h.astype(np.float64))
    return x


def check_selection(cand, top, gp, gt, gs, tag=""):
    """The GPU's K selections of one sentence-step are a valid TopB of the
    oracle's candidates (Algorithm 1, TopB, under the contract's 1e-3 bound).

    cand: the oracle's fp64 candidate scores [K, V] (-inf: dead row or masked
    word); top: the oracle's best K+1 scores, descending; gp/gt/gs: the GPU's
    parents, words and fp64 scores per slot.  Checks, for every slot:
      * the (parent, word) pairs are distinct;
      * as many slots are finite as the oracle has (min(K, finite candidates)),
        and the finite ones come first;
      * a finite slot's score is within SCORE_TOL of the oracle's score of the
        same candidate, which is at least the oracle's K-th score - GAP;
      * no candidate the GPU left out beats one it kept by more than GAP, and
        the kept ones are in order up to GAP (so wherever the oracle's gaps
        exceed GAP the set and the slot order are the oracle's exactly)."""
    K, V = cand.shape
    pairs = [(int(p), int(t)) for p, t in zip(gp, gt)]
    assert len(set(pairs)) == K, f"{tag}: repeated selections {pairs}"
    assert all(0 <= p < K and 0 <= t < V for p, t in pairs), f"{tag}: selection out of range {pairs}"
    fin_g = np.isfinite(gs)
    n_fin_o = int(np.isfinite(top[:K]).sum())
    assert int(fin_g.sum()) == n_fin_o, f"{tag}: {int(fin_g.sum())} finite slots, oracle has {n_fin_o}"
    assert np.all(fin_g[:n_fin_o]), f"{tag}: finite slots must come first: {gs}"
    assert not np.any(np.isnan(gs)), f"{tag}: NaN score {gs}"
    kth = top[K - 1]
    oc = np.array([cand[p, t] for p, t in pairs])
    for j in range(n_fin_o):
        assert np.isfinite(oc[j]), f"{tag}: slot {j} {pairs[j]} is -inf for the oracle"
        assert abs(gs[j] - oc[j]) <= SCORE_TOL, f"{tag}: slot {j} {pairs[j]} score {gs[j]} vs oracle {oc[j]}"
        assert oc[j] >= kth - GAP, f"{tag}: slot {j} {pairs[j]} oracle score {oc[j]} below the K-th {kth}"
        if j > 0:
            assert oc[j] <= oc[j - 1] + GAP, f"{tag}: slots {j - 1},{j} out of order: {oc[j - 1]} {oc[j]}"
    if n_fin_o:
        rest = cand.copy()
        for p, t in pairs[:n_fin_o]:
            rest[p, t] = NEG_INF
        worst = oc[:n_fin_o].min()
        assert rest.max() <= worst + GAP, \
            f"{tag}: left out a candidate at {rest.max()} while keeping one at {worst}"
    return oc


def compare_step(rec, b, gp, gt, gs, tag=""):
    """Check one sentence's GPU selections against an oracle StepRecord made
    from the same state (the oracle's own TopB, with keep_cand).

    Every slot is checked by check_selection against the oracle's full
    candidate scores; in addition, the slots the oracle's own selections fix
    (neighbouring gaps above GAP) must hold its exact (parent, word), and the
    -inf fill of surplus slots must match.  Returns the number of slots
    compared exactly."""
    assert rec.cand is not None, "compare_step needs Decoder(keep_cand=True)"
    K = rec.parent.shape[1]
    top = rec.top[b]
    check_selection(rec.cand[b], top, gp, gt, gs, tag)
    op, ot, oq = rec.parent[b], rec.token[b], rec.qhat[b]

    def gap(a, c):
        if a == NEG_INF:
            return 0.0
        return np.inf if c == NEG_INF else a - c

    n_exact = 0
    if gap(top[K - 1], top[K]) > GAP:
        so = sorted((int(p), int(t)) for p, t, q in zip(op, ot, oq) if q > NEG_INF)
        sg = sorted((int(p), int(t)) for p, t, q in zip(gp, gt, gs) if q > NEG_INF)
        assert so == sg, f"{tag}: selected set differs: oracle {so} gpu {sg}"
    for j in range(K):
        left = np.inf if j == 0 else gap(top[j - 1], top[j])
        right = gap(top[j], top[j + 1])
        if oq[j] == NEG_INF:
            # the -inf slots follow from the finite ones: exact parents/tokens
            assert gs[j] == NEG_INF, f"{tag}: slot {j} should be dead"
            if gap(top[K - 1], top[K]) > GAP or top[K - 1] == NEG_INF:
                assert (gp[j], gt[j]) == (op[j], ot[j]), f"{tag}: dead slot {j} {(gp[j], gt[j])} vs {(op[j], ot[j])}"
                n_exact += 1
            continue
        if left > GAP and right > GAP:
            assert (gp[j], gt[j]) == (op[j], ot[j]), \
                f"{tag}: slot {j}: oracle {(op[j], ot[j], oq[j])} gpu {(gp[j], gt[j], gs[j])}"
            assert abs(gs[j] - oq[j]) <= SCORE_TOL, f"{tag}: slot {j} score {gs[j]} vs {oq[j]}"
            n_exact += 1
    return n_exact


def rescore(cfg, s, seq, W64, table, lam=None):
    """Score of a whole hypothesis of sentence s from scratch (Eq. 1 plus
    lambda times Eq. 2's L, summed over its words), one prefix at a time with
    the oracle's projection, log-softmax and L row; the forced-EOS bias of the
    workload enters each step's logits as in the decode."""
    lam = cfg.lam if lam is None else lam
    parts = []
    for t in range(1, len(seq) + 1):
        hist = tuple(seq[:t - 1])
        h = synth.bf16_to_f32(synth.hidden_state(cfg, s, hist)).astype(np.float64)
        x = project(W64, h[None, :])[0]
        x[1] += synth.eos_bias(cfg, t, s)
        lp = log_softmax(x)
        L = table.lmbr_row(hist, cfg.V, cfg.theta)
        y = seq[t - 1]
        parts.append(lp[y] + lam * L[y])
    return math.fsum(parts)


def first_divergence(a, b):
    """1-based position of the first differing token (None when equal)."""
    if tuple(a) == tuple(b):
        return None
    n = min(len(a), len(b))
    return next((i for i in range(n) if a[i] != b[i]), n) + 1


def write_record(name, rec):
    """Append a parity record (JSON) under $LMBR_PARITY_RECORD, if set."""
    d = os.environ.get("LMBR_PARITY_RECORD")
    if not d:
        return
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, f"{name}.json"), "w") as f:
        json.dump(rec, f, indent=1, sort_keys=True)
