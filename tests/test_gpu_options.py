"""Parity of the decode options with the fp64 oracle, through the C ABI.

The options are the optional parts of Section 3: GetBestHypothesis with
length normalisation, the stack of EOS candidates that did not survive TopB
(returned when no hypothesis finishes), per-sentence decode lengths, a
constraint that masks candidates before TopB, and the early pruning of
Section 4.3.  Inputs are seeded and shared
with the oracle; the tolerances are those of the other parity tests (scores
within 1e-3; selections exact wherever the oracle's gaps exceed 1e-3).
"""
import math

import numpy as np
import pytest

import synth
from oracle.beam import NEG_INF, Decoder, Posteriors, decode_synthetic
from tests import gpu_util as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible to torch")
    import paper_1804_11324_amd as P
    P.lib()
    return torch


def _cfg(index, **kw):
    """Sixteen sentences over a ragged 3001-word vocabulary (twelve 256-column
    tiles, the last one partial)."""
    base = dict(B=16, K=4, V=3001, H=128, T=16, lam=1.0, theta=synth.THETA, paths=30,
                path_len=12, zipf_a=1.1)
    base.update(kw)
    return synth.Config(f"opt{index}", index, **base)


def allowed_words(cfg, seed, frac=0.3):
    """bool [B, V]: a random fraction of the words (EOS included) per sentence;
    sentence 1 allows two words and EOS (fewer candidates than slots at the
    first step), sentence 2 a single word and no EOS."""
    rng = np.random.default_rng(seed)
    a = rng.random((cfg.B, cfg.V)) < frac
    a[:, 1] = True
    if cfg.B > 2:
        a[1] = False
        a[1, [5, 17, 1]] = True
        a[2] = False
        a[2, 9] = True
    return a


def pack_bits(allowed):
    """bool [B, V] -> uint32 [B, ceil(V/32)]: bit v % 32 of word v // 32."""
    B, V = allowed.shape
    W = (V + 31) // 32
    pad = np.zeros((B, W * 32), dtype=bool)
    pad[:, :V] = allowed
    return np.packbits(pad, axis=1, bitorder="little").view("<u4").reshape(B, W)


def set_options(g, length_norm=False, finish="at_T", steps=None, allowed=None, prune=None):
    P, torch = g.P, g.torch
    fin = P.LMBR_FINISH_EOS_BACKUP if finish == "eos_backup" else P.LMBR_FINISH_AT_T
    P.lmbr_set_decode_options(g.ctx, int(length_norm), fin, prune)
    P.lmbr_set_sentence_steps(g.ctx, steps)
    if allowed is not None:
        g.allowed = torch.from_numpy(pack_bits(allowed).view(np.int32)).cuda()
        P.lmbr_set_constraints(g.ctx, g.allowed)
    else:
        P.lmbr_set_constraints(g.ctx, None)
    P.lmbr_state_init(g.ctx, g.st, g.cfg.seed)


def read_record(g):
    """The per-sentence record: best finished value, and the backup's (score, step, slot)."""
    raw = g.st.sent.cpu().numpy().reshape(-1, 3)
    ints = raw[:, 2].copy().view(np.int32).reshape(-1, 2)
    return raw[:, 0].copy(), raw[:, 1].copy(), ints[:, 0], ints[:, 1]


def traceback(g, T):
    torch, P = g.torch, g.P
    B = g.cfg.B
    toks = torch.empty((B, g.T_max), dtype=torch.int32, device="cuda")
    lens = torch.empty(B, dtype=torch.int32, device="cuda")
    scs = torch.empty(B, dtype=torch.float64, device="cuda")
    step = torch.empty(B, dtype=torch.int32, device="cuda")
    slot = torch.empty(B, dtype=torch.int32, device="cuda")
    P.lmbr_traceback(g.ctx, g.st, toks, lens, scs, step, slot)
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in (toks, lens, scs, step, slot)]


def rank_value(dec, e):
    t, _, score = e
    return score / t if dec.length_norm else score


def decisive_choice(dec, entries):
    """The best of `entries` is separated from the runner-up by more than the gap."""
    if len(entries) < 2:
        return True
    v = sorted((rank_value(dec, e) for e in entries), reverse=True)
    return v[0] - v[1] > G.GAP


def prune_margin(dec, b):
    """Smallest distance of a live slot's value to the pruning threshold over
    the decode (inf without pruning)."""
    if dec.prune is None:
        return np.inf
    m = np.inf
    for r in dec.records:
        thr = r.fbest[b] - dec.prune
        if thr == NEG_INF:
            continue
        for j in range(dec.K):
            if r.qhat[b, j] > NEG_INF and r.token[b, j] != dec.eos:
                m = min(m, abs(dec._value((r.t, j, r.qhat[b, j])) - thr))
    return m


def check_decode(dec, cfg, outs, sents, record, tag):
    toks, lens, scs, step, slot = outs
    fbest, bk_score, bk_step, bk_slot = record
    clean = agree = 0
    for b, s in enumerate(sents):
        best = dec.best(b)
        gaps = [r.gap_k()[b] for r in dec.records if np.isfinite(r.top[b, cfg.K - 1])]
        steady = (not gaps or min(gaps) > G.GAP) and prune_margin(dec, b) > G.GAP
        F = dec.finished(b)
        pool = F if F else (dec.backup[b] if dec.finish == "eos_backup" else [])
        gpu_seq = tuple(int(x) for x in toks[s, :lens[s]])
        if best is None:
            agree += lens[s] == 0
            if steady:
                clean += 1
                assert lens[s] == 0 and scs[s] == NEG_INF, f"{tag} s={s}: gpu found {gpu_seq}"
            continue
        same = gpu_seq == best.tokens
        agree += same
        if steady and decisive_choice(dec, pool):
            clean += 1
            assert same, f"{tag} s={s}: gpu {gpu_seq} oracle {best.tokens}"
            assert abs(scs[s] - best.score) <= G.SCORE_TOL, f"{tag} s={s}: score {scs[s]} vs {best.score}"
            assert (step[s] + 1, slot[s]) == (best.t, best.j), \
                f"{tag} s={s}: entry {(step[s] + 1, slot[s])} vs {(best.t, best.j)}"
        # the backup record itself, also where F made it unused
        if dec.finish == "eos_backup" and steady:
            if not dec.backup[b]:
                assert bk_step[s] == 0, f"{tag} s={s}: gpu backup {bk_step[s]} but the oracle has none"
            elif decisive_choice(dec, dec.backup[b]):
                t, k, c = min(dec.backup[b], key=dec._rank)
                assert (bk_step[s], bk_slot[s]) == (t, k), f"{tag} s={s}: backup {(bk_step[s], bk_slot[s])} vs {(t, k)}"
                assert abs(bk_score[s] - c) <= G.SCORE_TOL
        if dec.prune is not None and steady:
            want = dec.records[-1].fbest[b]
            assert (fbest[s] == NEG_INF) == (want == NEG_INF), f"{tag} s={s}: best finished {fbest[s]} vs {want}"
            if want > NEG_INF:
                assert abs(fbest[s] - want) <= G.SCORE_TOL
    G.log(f"  {tag}: agreement {agree}/{len(sents)}, decisive {clean}")
    return clean


OPTION_CASES = {
    "length_norm": dict(length_norm=True),
    "eos_backup": dict(finish="eos_backup"),
    "eos_backup_norm": dict(finish="eos_backup", length_norm=True),
    "steps": dict(steps=True),
    "steps_backup": dict(steps=True, finish="eos_backup"),
    "constrained": dict(allowed=True),
    "prune": dict(prune=math.log(100.0)),
    "prune_norm_backup": dict(prune=0.1, length_norm=True, finish="eos_backup", eos=(4.0, 3)),
    "all": dict(steps=True, finish="eos_backup", length_norm=True, allowed=True, prune=0.1, eos=(4.0, 3)),
}


@pytest.mark.parametrize("path", ["two_pass", "fused", "logits"])
@pytest.mark.parametrize("name", list(OPTION_CASES))
def test_option_decode_parity(torch_cuda, name, path):
    """A whole decode under each option, step by step through the C ABI, then
    GetBestHypothesis.  Odd sentences get a large negative EOS bias so that
    their EOS candidates never survive TopB (F stays empty for them), or,
    where early pruning needs finished hypotheses, a positive one from step 3."""
    opt = dict(OPTION_CASES[name])
    index = 60 + list(OPTION_CASES).index(name)
    boost, start = opt.pop("eos", (-30.0, 1))
    cfg = _cfg(index, eos_boost=boost, eos_boost_from=start)
    rng = np.random.default_rng(cfg.seed)
    steps = rng.integers(1, cfg.T + 1, size=cfg.B).astype(np.int32) if opt.pop("steps", False) else None
    allowed = allowed_words(cfg, cfg.seed + 1) if opt.pop("allowed", False) else None
    G.log(f"options {name} ({path}): B={cfg.B} K={cfg.K} V={cfg.V} T={cfg.T} steps={steps} "
          f"constraint={allowed is not None} {opt}")
    g = G.GpuDecoder(cfg, path=path)
    set_options(g, steps=steps, allowed=allowed, **opt)
    bias = synth.eos_bias_table(cfg)
    for t in range(cfg.T):
        g.step(bias[t])
    outs = traceback(g, cfg.T)
    record = read_record(g)
    sents = list(range(cfg.B))
    dec = decode_synthetic(cfg, sents, G.weights(cfg), [Posteriors(*G.posteriors(cfg, s)) for s in sents],
                           allowed=allowed, steps=None if steps is None else steps.tolist(), **opt)
    clean = check_decode(dec, cfg, outs, sents, record, f"{name}/{path}")
    assert clean >= cfg.B // 2, "too few decisive sentences for a meaningful comparison"
    g.close()


@pytest.mark.parametrize("path", ["two_pass", "fused", "logits"])
def test_constraint_step_parity(torch_cuda, path):
    """Every step of a constrained decode against the oracle's step from the
    same state (the GPU state is reset to the oracle's after each step):
    masked words never selected, the -inf slots filled in flat order when a
    sentence has fewer allowed candidates than slots."""
    cfg = _cfg(70, T=8)
    allowed = allowed_words(cfg, 71)
    sents = list(range(cfg.B))
    G.log(f"constraint steps ({path}): B={cfg.B} K={cfg.K} V={cfg.V} T={cfg.T}")
    g = G.GpuDecoder(cfg, path=path)
    set_options(g, allowed=allowed)
    dec = Decoder(cfg.V, cfg.K, cfg.lam, cfg.theta, [Posteriors(*G.posteriors(cfg, s)) for s in sents],
                  keep_cand=True)
    W64 = synth.bf16_to_f32(G.weights(cfg)).astype(np.float64)
    n_exact = 0
    for t in range(1, cfg.T + 1):
        gp, gt, gs = g.step()
        rec = dec.step(G.oracle_logits(cfg, sents, dec, W64), None, allowed)
        for b in sents:
            n_exact += G.compare_step(rec, b, gp[b], gt[b], gs[b], tag=f"t={t} s={b}")
            fin = gs[b] > NEG_INF
            assert allowed[b, gt[b][fin]].all(), f"t={t} s={b}: a disallowed word was selected"
        g.inject(dec, sents)
    G.log(f"  {n_exact}/{cfg.T * cfg.B * cfg.K} slots compared exactly")
    assert n_exact >= 0.9 * cfg.T * cfg.B * cfg.K
    g.close()


def test_option_arguments_validated(torch_cuda):
    import paper_1804_11324_amd as P
    cfg = _cfg(72, T=4)
    g = G.GpuDecoder(cfg)
    with pytest.raises(P.LmbrError) as e:
        P.lmbr_set_decode_options(g.ctx, 0, 7)
    assert e.value.code == -1
    with pytest.raises(P.LmbrError) as e:
        P.lmbr_set_decode_options(g.ctx, 2, 0)
    assert e.value.code == -1
    with pytest.raises(P.LmbrError) as e:
        P.lmbr_set_sentence_steps(g.ctx, np.full(cfg.B, cfg.T + 1, dtype=np.int32))
    assert e.value.code == -1
    with pytest.raises(P.LmbrError) as e:
        P.lmbr_set_sentence_steps(g.ctx, np.zeros(cfg.B, dtype=np.int32))
    assert e.value.code == -1
    with pytest.raises(P.LmbrError) as e:
        P.lmbr_set_decode_options(g.ctx, 0, 0, -1.0)
    assert e.value.code == -1
    with pytest.raises(P.LmbrError) as e:
        P.lmbr_set_decode_options(g.ctx, 0, 0, float("nan"))
    assert e.value.code == -1
    for bad in (-1, 2):
        with pytest.raises(P.LmbrError) as e:
            P.lmbr_set_step_path(g.ctx, bad)
        assert e.value.code == -1
    # the backup stack and early pruning need the per-sentence record
    keep = g.st.c.sent
    for args in [(0, P.LMBR_FINISH_EOS_BACKUP, None), (0, P.LMBR_FINISH_AT_T, 2.0)]:
        P.lmbr_set_decode_options(g.ctx, *args)
        g.st.c.sent = None
        with pytest.raises(P.LmbrError) as e:
            P.lmbr_state_init(g.ctx, g.st, cfg.seed)
        assert e.value.code == -1
        g.st.c.sent = keep
    P.lmbr_state_init(g.ctx, g.st, cfg.seed)
    fbest, score, step, slot = read_record(g)
    assert np.all(fbest == NEG_INF) and np.all(score == NEG_INF)
    assert np.all(step == 0) and np.all(slot == -1)
    # without the options the record is optional
    P.lmbr_set_decode_options(g.ctx, 0, P.LMBR_FINISH_AT_T, None)
    g.st.c.sent = None
    P.lmbr_state_init(g.ctx, g.st, cfg.seed)
    g.st.c.sent = keep
    g.close()


def test_compaction_frees_blocks(torch_cuda):
    """Live-row compaction: half of 64 sentences end after step 2 (their 256
    rows die), so from step 3 on the fused kernel projects one 256-row block
    instead of two, and the two-pass step's projection only the live rows
    (lmbr_projected_rows).  The decode must still match the oracle, on every
    path (the logits path scores every live row of the caller's logits)."""
    cfg = _cfg(80, B=64, K=8, T=6)
    steps = np.array([2] * 32 + [6] * 32, dtype=np.int32)
    sents = list(range(cfg.B))
    dec = decode_synthetic(cfg, sents, G.weights(cfg), [Posteriors(*G.posteriors(cfg, s)) for s in sents],
                           steps=steps.tolist())
    for path in ("two_pass", "fused", "logits"):
        G.log(f"compaction ({path}): B={cfg.B} K={cfg.K} V={cfg.V} T={cfg.T}, sentences 0..31 end at step 2")
        g = G.GpuDecoder(cfg, path=path)
        set_options(g, steps=steps)
        for t in range(cfg.T):
            live = int(g.torch.isfinite(g.st.q).sum().item())
            g.step()
            if path == "two_pass":
                # the default step projects the live rows only, listed first:
                # row blocks past them are skipped
                assert g.P.lmbr_projected_rows(g.ctx) == live
            if t == 1:
                live = int(g.torch.isfinite(g.st.q).sum().item())
                assert live <= 256, f"{live} live rows after the short sentences ended"
        outs = traceback(g, cfg.T)
        clean = check_decode(dec, cfg, outs, sents, read_record(g), f"compaction/{path}")
        assert clean >= cfg.B // 2
        g.close()


def test_projection_strips_follow_live_blocks(torch_cuda):
    """Shorter projection strips when fewer row blocks are live than the grid
    was cut for: 256 sentences of 8 beams over 16384 words make 8 row blocks
    of 256 rows, cut into strips of two column tiles.  The first step has one
    live block (one slot per sentence) and, after 160 sentences end at step 1,
    three blocks stay live: the live blocks then take one-tile strips over the
    grid.  The default step must equal, bit for bit, the step from logits
    projected in full (lmbr_project, no live-row map), and the decode must
    match the oracle on its decisive sentences."""
    cfg = _cfg(81, B=256, K=8, V=16384, H=64, T=4, paths=20)
    steps = np.array([1] * 160 + [4] * 96, dtype=np.int32)
    sents = list(range(cfg.B))
    dec = decode_synthetic(cfg, sents, G.weights(cfg), [Posteriors(*G.posteriors(cfg, s)) for s in sents],
                           steps=steps.tolist())
    hist = {}
    for path in ("two_pass", "logits"):
        G.log(f"projection strips ({path}): B={cfg.B} K={cfg.K} V={cfg.V}, sentences 0..159 end at step 1")
        g = G.GpuDecoder(cfg, path=path)
        set_options(g, steps=steps)
        for t in range(cfg.T):
            live = int(g.torch.isfinite(g.st.q).sum().item())
            g.step()
            if path == "two_pass":
                assert g.P.lmbr_projected_rows(g.ctx) == live
            if t == 1:
                assert int(g.torch.isfinite(g.st.q).sum().item()) <= 96 * cfg.K
        outs = traceback(g, cfg.T)
        if path == "two_pass":
            clean = check_decode(dec, cfg, outs, sents, read_record(g), "strips")
            assert clean >= cfg.B // 4
        hist[path] = [x.cpu().numpy() for x in (g.st.bp, g.st.tok, g.st.qhist)] + outs
        g.close()
    for a, b in zip(hist["two_pass"], hist["logits"]):
        assert np.array_equal(a, b), "the live-row projection differs from the full projection"


def test_beam_past_the_live_row_map(torch_cuda):
    """A beam of more than 16384 rows (1100 sentences x 16 beams): the default
    step projects every row without a live-row listing (each workgroup's scan
    would cost more than it saves), and the score pass still skips the dead
    rows.  The decode must equal, bit for bit, the decode from logits
    projected by lmbr_project, and match the oracle on sampled sentences."""
    cfg = _cfg(82, B=1100, K=16, V=1000, H=64, T=4, paths=8, path_len=10)
    steps = np.full(cfg.B, cfg.T, dtype=np.int32)
    sents = [0, 259, 555, 1036, 1099]        # the first four decisive (all gaps above 1e-3), the last row block
    W = G.weights(cfg)
    dec = decode_synthetic(cfg, sents, W, [Posteriors(*G.posteriors(cfg, s)) for s in sents])
    hist = {}
    for path in ("two_pass", "logits"):
        G.log(f"beam past the live-row map ({path}): B={cfg.B} K={cfg.K} (M={cfg.B * cfg.K}) V={cfg.V} T={cfg.T}")
        g = G.GpuDecoder(cfg, path=path, W=W)
        set_options(g, steps=steps)
        for t in range(cfg.T):
            g.step()
            if path == "two_pass":
                assert g.P.lmbr_projected_rows(g.ctx) == g.M    # every row projected
        outs = traceback(g, cfg.T)
        if path == "two_pass":
            clean = check_decode(dec, cfg, outs, sents, read_record(g), "past the map")
            assert clean >= 4
        hist[path] = [x.cpu().numpy() for x in (g.st.bp, g.st.tok, g.st.qhist)] + outs
        g.close()
    for a, b in zip(hist["two_pass"], hist["logits"]):
        assert np.array_equal(a, b), "the default step differs from the step from projected logits"
