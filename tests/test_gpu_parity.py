"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Marked gpu: needs an MI355X and the built liblmbr.so.  Every comparison uses
the same seeded inputs on both sides (synth); nothing expected comes from the
HIP path.  Tolerances: selected scores within 1e-3 absolute; selections exact
wherever the oracle's gap between the K-th and (K+1)-th candidate exceeds
1e-3 (and slot order wherever neighbouring gaps exceed it); integer outputs of
the stand-in state generator and of the bookkeeping bit-exact.
"""
import json
import math
import os

import numpy as np
import pytest

import synth
from oracle.beam import NEG_INF, Decoder, Posteriors, decode_synthetic, project
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible to torch")
    import paper_1804_11324_amd as P
    P.lib()
    return torch


# --------------------------------------------------------------------------
# a0: stand-in decoder state
# --------------------------------------------------------------------------
def test_synth_hidden_bit_exact(torch_cuda):
    torch = torch_cuda
    cfg = synth.get_config("small").replace(B=64, K=16)
    G.log("synth_hidden: M=1024 H=512")
    g = G.GpuDecoder(cfg.replace(V=256, paths=4, path_len=3), K=16, T_max=2)
    rng = np.random.default_rng(5)
    hh = rng.integers(-2 ** 63, 2 ** 63 - 1, size=g.M, dtype=np.int64)
    g.st.hhash.copy_(torch.from_numpy(hh))
    g.P.lmbr_synth_hidden(g.ctx, g.st, g.hidden)
    torch.cuda.synchronize()
    got = g.hidden.cpu().numpy().view(np.uint16)
    want = synth.hidden_from_hashes(hh.view(np.uint64), cfg.H)
    assert np.array_equal(got, want)
    # the initial hash of state_init follows hh_0(s)
    g.P.lmbr_state_init(g.ctx, g.st, cfg.seed)
    torch.cuda.synchronize()
    h0 = g.st.hhash.cpu().numpy().view(np.uint64).reshape(cfg.B, 16)
    for s in [0, 1, 63]:
        assert all(int(x) == synth.initial_hash(cfg, s) for x in h0[s])
    g.close()


# --------------------------------------------------------------------------
# a1: projection
# --------------------------------------------------------------------------
@pytest.mark.parametrize("M,V,H", [(4, 1000, 64), (1, 37, 64), (63, 1001, 128), (64, 32000, 512),
                                   (65, 4099, 192), (256, 32000, 512), (300, 777, 256),
                                   (768, 32000, 1024), (2048, 64000, 1024)])
def test_projection_matches_fp64(torch_cuda, M, V, H):
    torch = torch_cuda
    import paper_1804_11324_amd as P
    G.log(f"projection M={M} V={V} H={H}")
    cfg = synth.Config("p", 7, B=M, K=1, V=V, H=H, T=1, lam=1.0, theta=synth.THETA, paths=1,
                       path_len=1, zipf_a=1.1)
    W = synth.make_weights(cfg)
    hid = synth.hidden_from_hashes(np.arange(M, dtype=np.uint64) * np.uint64(1000003), H)
    bias = np.random.default_rng(M).standard_normal(V).astype(np.float32)
    ctx = P.lmbr_create(P.make_config(M, 1, V, H, 1))
    Wd = torch.from_numpy(W.view(np.int16)).cuda()
    bd = torch.from_numpy(bias).cuda()
    P.lmbr_set_projection(ctx, Wd, 0, bd)
    ld = (V + 3) // 4 * 4 + 4
    out = torch.full((M, ld), float("nan"), dtype=torch.float32, device="cuda")
    hd = torch.from_numpy(hid.view(np.int16)).cuda()
    P.lmbr_project(ctx, hd, out, ld)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    assert np.all(np.isnan(got[:, V:])), "wrote past column V"
    rows = np.arange(M) if M <= 256 else np.random.default_rng(1).choice(M, 256, replace=False)
    A = synth.bf16_to_f32(hid[rows]).astype(np.float64)
    W64 = synth.bf16_to_f32(W).astype(np.float64)
    ref = project(W64, A, bias.astype(np.float64))
    err = np.abs(got[rows, :V] - ref)
    bound = np.abs(A) @ np.abs(W64).T * (H * 2.0 ** -24) + 1e-6
    G.log(f"  max |err| = {err.max():.3e}")
    assert np.all(err <= bound)
    assert err.max() < 1e-4
    ctx.close()


def test_projection_hv_layout(torch_cuda):
    torch = torch_cuda
    import paper_1804_11324_amd as P
    M, V, H = 64, 1000, 128
    G.log("projection layout [H,V]")
    cfg = synth.Config("p", 8, B=M, K=1, V=V, H=H, T=1, lam=1.0, theta=synth.THETA, paths=1,
                       path_len=1, zipf_a=1.1)
    W = synth.make_weights(cfg)
    hid = synth.hidden_from_hashes(np.arange(M, dtype=np.uint64), H)
    outs = []
    for layout, arr in [(0, W), (1, np.ascontiguousarray(W.T))]:
        ctx = P.lmbr_create(P.make_config(M, 1, V, H, 1))
        Wd = torch.from_numpy(arr.view(np.int16)).cuda()
        P.lmbr_set_projection(ctx, Wd, layout)
        out = torch.empty((M, 1024), dtype=torch.float32, device="cuda")
        P.lmbr_project(ctx, torch.from_numpy(hid.view(np.int16)).cuda(), out, 1024)
        torch.cuda.synchronize()
        outs.append(out.cpu().numpy()[:, :V])
        ctx.close()
    assert np.array_equal(outs[0], outs[1])


# --------------------------------------------------------------------------
# a2-a4 on the hand-derived example
# --------------------------------------------------------------------------
def test_hand_example_on_gpu(torch_cuda):
    torch = torch_cuda
    import paper_1804_11324_amd as P
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    V, K = g["V"], g["K"]
    G.log("hand example")
    ctx = P.lmbr_create(P.make_config(1, K, V, 64, g["T"], g["eos"], g["lambda"], g["theta"]))
    order = np.array([len(u) for u, _ in g["ngrams"]])
    toks = np.array([list(u) + [-1] * (4 - len(u)) for u, _ in g["ngrams"]])
    post = np.array([p for _, p in g["ngrams"]], dtype=np.float32)
    P.lmbr_load_posteriors(ctx, 0, order, toks, post)
    st = P.BeamState(ctx.cfg)
    P.lmbr_state_init(ctx, st, 0)
    logits = torch.zeros((K, 64), dtype=torch.float32, device="cuda")
    par = torch.empty(K, dtype=torch.int32, device="cuda")
    tok = torch.empty(K, dtype=torch.int32, device="cuda")
    sc = torch.empty(K, dtype=torch.float64, device="cuda")
    for want in g["steps"]:
        P.lmbr_beam_step_logits(ctx, st, logits, 64, None, par, tok, sc)
        torch.cuda.synchronize()
        assert par.cpu().tolist() == want["parent"]
        assert tok.cpu().tolist() == want["token"]
        assert np.allclose(sc.cpu().numpy(), want["qhat"], atol=g["tol"], rtol=0)
    T = g["T"]
    toks_o = torch.empty((1, T), dtype=torch.int32, device="cuda")
    len_o = torch.empty(1, dtype=torch.int32, device="cuda")
    sc_o = torch.empty(1, dtype=torch.float64, device="cuda")
    step_o = torch.empty(1, dtype=torch.int32, device="cuda")
    slot_o = torch.empty(1, dtype=torch.int32, device="cuda")
    P.lmbr_traceback(ctx, st, toks_o, len_o, sc_o, step_o, slot_o)
    torch.cuda.synchronize()
    n = int(len_o.item())
    assert toks_o.cpu().numpy()[0, :n].tolist() == g["best"]["tokens"]
    assert np.all(toks_o.cpu().numpy()[0, n:] == -1)
    assert abs(sc_o.item() - g["best"]["score"]) < g["tol"]
    assert (step_o.item() + 1, slot_o.item()) == (g["best"]["t"], g["best"]["j"])
    ctx.close()


# --------------------------------------------------------------------------
# a0-a4: step parity on identical states (oracle state injected every step)
# --------------------------------------------------------------------------
STEP_CASES = {
    # name: (sentences checked by the oracle, steps)
    "tiny": (None, 10),
    "small": (None, 64),
    "base": ([0, 1, 2, 3, 30, 31, 62, 63], 100),
    "big": ([0, 5, 63], 60),
    "large": ([0, 77, 255], 32),
}


# (workload, path): every workload through the default step (projection into
# the context's logits workspace, then the score pass) and through the fused
# projection + score kernel; several also through logits in a caller buffer
STEP_PATHS = ([(n, "two_pass") for n in STEP_CASES] + [(n, "fused") for n in STEP_CASES] +
              [("tiny", "logits"), ("small", "logits"), ("base", "logits"), ("large", "logits")])


@pytest.mark.parametrize("name,path", STEP_PATHS)
def test_step_parity(torch_cuda, name, path):
    cfg = synth.get_config(name)
    sents, T = STEP_CASES[name]
    sents = list(range(cfg.B)) if sents is None else sents
    G.log(f"step parity {name} ({path}): B={cfg.B} K={cfg.K} V={cfg.V} H={cfg.H}, oracle on {sents}, T={T}")
    g = G.GpuDecoder(cfg, path=path)
    dec = G.oracle_for(cfg, sents)
    W64 = synth.bf16_to_f32(G.weights(cfg)).astype(np.float64)
    bias_tab = synth.eos_bias_table(cfg)
    n_exact = n_slots = 0
    for t in range(1, T + 1):
        gp, gt, gs = g.step(bias_tab[t - 1] if cfg.eos_boost else None)
        x = G.oracle_logits(cfg, sents, dec, W64)
        ob = np.array([synth.eos_bias(cfg, t, s) for s in sents])
        rec = dec.step(x, ob if np.any(ob) else None)
        for b, s in enumerate(sents):
            n_exact += G.compare_step(rec, b, gp[s], gt[s], gs[s], tag=f"{name} t={t} s={s}")
            n_slots += cfg.K
        g.inject(dec, sents)
    G.log(f"  {n_exact}/{n_slots} slots compared exactly")
    assert n_exact >= 0.9 * n_slots
    g.close()


@pytest.mark.parametrize("path", ["two_pass", "fused"])
def test_step_parity_ragged_strips(torch_cuda, path):
    """256 sentences at V = 59500: the score pass cuts 59 tiles of 1024
    columns (the last one 108 columns wide) into strips of six, so the last
    strip is shorter and ends inside a tile, and the dense history-free row
    ends before the tile does."""
    import dataclasses
    cfg = dataclasses.replace(synth.get_config("large"), name="large-ragged", V=59500, H=64, T=6, paths=200,
                              path_len=30)
    sents = [0, 128, 255]
    G.log(f"ragged strips ({path}): B={cfg.B} K={cfg.K} V={cfg.V} H={cfg.H}, oracle on {sents}")
    g = G.GpuDecoder(cfg, path=path)
    dec = G.oracle_for(cfg, sents)
    W64 = synth.bf16_to_f32(G.weights(cfg)).astype(np.float64)
    n_exact = n_slots = 0
    for t in range(1, cfg.T + 1):
        gp, gt, gs = g.step(None)
        x = G.oracle_logits(cfg, sents, dec, W64)
        rec = dec.step(x, None)
        for b, s in enumerate(sents):
            n_exact += G.compare_step(rec, b, gp[s], gt[s], gs[s], tag=f"ragged t={t} s={s}")
            n_slots += cfg.K
        g.inject(dec, sents)
    G.log(f"  {n_exact}/{n_slots} slots compared exactly")
    assert n_exact >= 0.9 * n_slots
    g.close()


# --------------------------------------------------------------------------
# a5: full decodes, un-injected, with the oracle following the GPU's choices
# --------------------------------------------------------------------------
# sentences checked per workload (the GPU decodes the whole batch); base
# includes odd sentences, whose forced EOS ends them after step 31
TRAJECTORY_CASES = {"tiny": [0], "small": [0, 5, 10, 15], "base": [0, 1, 30, 63],
                    "big": [0, 21, 42, 63], "large": [0, 77, 160, 255]}


def _gpu_decode(g, cfg, T, state_fn=None):
    """lmbr_decode from a fresh state: host outputs (tokens, lengths, scores)."""
    torch = g.torch
    P = g.P
    eb = torch.from_numpy(synth.eos_bias_table(cfg, T)).cuda() if cfg.eos_boost else None
    toks = np.empty((cfg.B, g.T_max), dtype=np.int32)
    lens = np.empty(cfg.B, dtype=np.int32)
    scs = np.empty(cfg.B, dtype=np.float64)
    P.lmbr_state_init(g.ctx, g.st, cfg.seed)
    P.lmbr_decode(g.ctx, g.st, T, eb, toks, lens, scs, state_fn=state_fn)
    return toks, lens, scs


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", list(TRAJECTORY_CASES))
def test_decode_trajectory_parity(torch_cuda, name):
    """A whole T-step decode on the GPU with nothing injected (Algorithm 1's
    loop, the merge's own realignment and next-step probes), read back from
    the history arrays.  The oracle then decodes the checked sentences taking
    only the GPU's discrete choices (parent, word) at each step and computing
    every score itself: each step's selections must be a valid TopB of the
    oracle's candidates (check_selection: distinct, scores within 1e-3, none
    below the oracle's K-th by more than 1e-3, none beaten by a left-out
    candidate by more than 1e-3).  GetBestHypothesis's result must re-score
    from scratch to the GPU's score and match the oracle's best entry of F.
    Separately, the oracle's own decode (TopB unsteered) gives the token
    agreement, which must be exact for sentences whose every gap exceeds
    1e-3; agreement and first-divergence steps are recorded."""
    cfg = synth.get_config(name)
    sents = TRAJECTORY_CASES[name]
    T, K = cfg.T, cfg.K
    G.log(f"trajectory {name}: B={cfg.B} K={K} V={cfg.V} H={cfg.H} T={T}, oracle on {sents}")
    g = G.GpuDecoder(cfg)
    toks, lens, scs = _gpu_decode(g, cfg, T)
    M = cfg.B * K
    bp = g.st.bp.cpu().numpy().reshape(g.T_max, cfg.B, K)
    tk = g.st.tok.cpu().numpy().reshape(g.T_max, cfg.B, K)
    qh = g.st.qhist.cpu().numpy().reshape(g.T_max, cfg.B, K)
    g.close()
    assert M == bp.shape[1] * bp.shape[2]
    tables = [Posteriors(*G.posteriors(cfg, s)) for s in sents]
    W64 = synth.bf16_to_f32(G.weights(cfg)).astype(np.float64)

    # 1. the oracle steered by the GPU's choices
    dec = Decoder(cfg.V, K, cfg.lam, cfg.theta, tables, keep_cand=True)
    n_slots = 0
    for t in range(1, T + 1):
        x = G.oracle_logits(cfg, sents, dec, W64)
        ob = np.array([synth.eos_bias(cfg, t, s) for s in sents])
        force = (bp[t - 1][sents], tk[t - 1][sents])
        rec = dec.step(x, ob if np.any(ob) else None, force=force)
        for b, s in enumerate(sents):
            G.check_selection(rec.cand[b], rec.top[b], bp[t - 1, s], tk[t - 1, s], qh[t - 1, s],
                              tag=f"{name} t={t} s={s}")
            n_slots += int(np.isfinite(qh[t - 1, s]).sum())
        if t % 16 == 0:
            G.log(f"  step {t}: {n_slots} live selections checked")
    assert n_slots > 0
    record = {"workload": name, "B": cfg.B, "K": K, "V": cfg.V, "H": cfg.H, "T": T, "sentences": sents,
              "steered_selections_checked": n_slots, "per_sentence": []}
    for b, s in enumerate(sents):
        seq = tuple(int(v) for v in toks[s, :lens[s]])
        best = dec.best(b)
        assert best is not None and len(seq) > 0, f"{name} s={s}: no hypothesis"
        assert abs(scs[s] - best.score) <= G.SCORE_TOL, f"{name} s={s}: score {scs[s]} vs oracle F {best.score}"
        F = sorted((sc for _, _, sc in dec.finished(b)), reverse=True)
        if len(F) < 2 or F[0] - F[1] > G.GAP:
            assert seq == best.tokens, f"{name} s={s}: GetBestHypothesis {seq} vs {best.tokens}"
        r = G.rescore(cfg, s, seq, W64, tables[b])
        assert abs(r - scs[s]) <= G.SCORE_TOL, f"{name} s={s}: re-scored {r} vs gpu {scs[s]}"
        record["per_sentence"].append({"sentence": s, "gpu_len": len(seq), "gpu_score": float(scs[s]),
                                       "rescored": r})
    G.log(f"  steered oracle: {n_slots} selections valid, final hypotheses re-score within {G.SCORE_TOL}")

    # 2. the oracle's own decode: token agreement
    own = Decoder(cfg.V, K, cfg.lam, cfg.theta, tables)
    for t in range(1, T + 1):
        x = G.oracle_logits(cfg, sents, own, W64)
        ob = np.array([synth.eos_bias(cfg, t, s) for s in sents])
        own.step(x, ob if np.any(ob) else None)
    agree = decisive = 0
    div = []
    for b, s in enumerate(sents):
        seq = tuple(int(v) for v in toks[s, :lens[s]])
        best = own.best(b)
        d = G.first_divergence(seq, best.tokens)
        agree += d is None
        if d is not None:
            div.append(d)
        gaps = [r.gap_k()[b] for r in own.records if np.isfinite(r.top[b, K - 1])]
        F = sorted((sc for _, _, sc in own.finished(b)), reverse=True)
        if min(gaps) > G.GAP and (len(F) < 2 or F[0] - F[1] > G.GAP):
            decisive += 1
            assert d is None, f"{name} s={s}: gpu {seq} oracle {best.tokens}"
        ps = record["per_sentence"][b]
        ps.update({"oracle_len": len(best.tokens), "oracle_score": best.score, "same_tokens": d is None,
                   "first_divergence_step": d, "min_gap": float(min(gaps))})
    record.update({"token_agreement": agree, "decisive_sentences": decisive,
                   "mean_first_divergence_step": float(np.mean(div)) if div else None})
    G.log(f"  token-sequence agreement {agree}/{len(sents)} (decisive {decisive})"
          + (f", mean first-divergence step {np.mean(div):.1f}" if div else ""))
    G.write_record(f"decode_agreement_{name}", record)


def test_decode_is_deterministic(torch_cuda):
    cfg = synth.get_config("small")
    G.log("determinism: small decode twice")
    g = G.GpuDecoder(cfg)
    a = _gpu_decode(g, cfg, cfg.T)
    qa = g.st.qhist.cpu().numpy().copy()
    b = _gpu_decode(g, cfg, cfg.T)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    assert np.array_equal(qa, g.st.qhist.cpu().numpy())
    g.close()


def _gpu_step_decode(g, cfg, T):
    """The same decode as lmbr_decode, launched step by step (stand-in state,
    lmbr_beam_step) and traced back."""
    torch = g.torch
    P = g.P
    eb = torch.from_numpy(synth.eos_bias_table(cfg, T)).cuda() if cfg.eos_boost else None
    toks = torch.empty((cfg.B, g.T_max), dtype=torch.int32, device="cuda")
    lens = torch.empty(cfg.B, dtype=torch.int32, device="cuda")
    scs = torch.empty(cfg.B, dtype=torch.float64, device="cuda")
    P.lmbr_state_init(g.ctx, g.st, cfg.seed)
    for t in range(T):
        P.lmbr_synth_hidden(g.ctx, g.st, g.hidden)
        P.lmbr_beam_step(g.ctx, g.st, g.hidden, eb[t] if eb is not None else None)
    P.lmbr_traceback(g.ctx, g.st, toks, lens, scs)
    torch.cuda.synchronize()
    return toks.cpu().numpy(), lens.cpu().numpy(), scs.cpu().numpy()


@pytest.mark.parametrize("name,path", [("small", "two_pass"), ("base", "fused"), ("big", "two_pass")])
def test_decode_graph_replays_match_steps(torch_cuda, name, path):
    """lmbr_decode captures its loop into a HIP graph at the first call and
    replays it afterwards: every replay, with eager launches and host
    synchronisations between them, equals the step-by-step decode bit for bit;
    a changed option (the step path) makes it capture again."""
    cfg = synth.get_config(name)
    T = min(cfg.T, 40)
    G.log(f"decode graph replays: {name} ({path}), T={T}")
    g = G.GpuDecoder(cfg, path=path)
    ref = _gpu_step_decode(g, cfg, T)
    for rep in range(3):
        got = _gpu_decode(g, cfg, T)
        assert all(np.array_equal(x, y) for x, y in zip(got, ref)), f"replay {rep} differs"
        again = _gpu_step_decode(g, cfg, T)            # eager work between replays
        assert all(np.array_equal(x, y) for x, y in zip(again, ref))
    other = "fused" if path == "two_pass" else "two_pass"
    g.P.lmbr_set_step_path(g.ctx, g.P.LMBR_STEP_FUSED if other == "fused" else g.P.LMBR_STEP_TWO_PASS)
    ref2 = _gpu_step_decode(g, cfg, T)
    got2 = _gpu_decode(g, cfg, T)
    assert all(np.array_equal(x, y) for x, y in zip(got2, ref2))
    g.close()


def test_decode_in_chunks_keeps_its_graphs(torch_cuda):
    """A decode run as several lmbr_decode calls of different lengths (each a
    graph of its own, kept by the context) equals the step-by-step decode bit
    for bit, on every repetition (so every graph is replayed, not only built)."""
    cfg = synth.get_config("small").replace(B=6, T=40)
    G.log("decode in chunks of 10, 7, 23 steps, three times")
    g = G.GpuDecoder(cfg)
    ref = _gpu_step_decode(g, cfg, cfg.T)
    ref_q = g.st.qhist.cpu().numpy().copy()
    toks = np.empty((cfg.B, cfg.T), np.int32)
    lens = np.empty(cfg.B, np.int32)
    scs = np.empty(cfg.B, np.float64)
    for rep in range(3):
        g.P.lmbr_state_init(g.ctx, g.st, cfg.seed)
        for T in (10, 7, 23):
            g.P.lmbr_decode(g.ctx, g.st, T, None, toks, lens, scs)
        assert g.st.t == cfg.T
        assert all(np.array_equal(x, y) for x, y in zip((toks, lens, scs), ref)), f"repetition {rep}"
        assert np.array_equal(g.st.qhist.cpu().numpy(), ref_q)
    g.close()


# --------------------------------------------------------------------------
# Edge cases: V < K (fewer finite candidates than slots), K = 1, ragged V,
# sentences that die, empty tables
# --------------------------------------------------------------------------
@pytest.mark.parametrize("V,T,K,index", [(4, 3, 16, 30), (3, 4, 16, 31), (2, 4, 3, 32), (2, 3, 1, 33)])
def test_underfull_beams_match_oracle(torch_cuda, V, T, K, index):
    cfg = synth.Config(f"x{index}", index, B=3, K=K, V=V, H=64, T=T, lam=1.0, theta=synth.THETA,
                       paths=5, path_len=3, zipf_a=1.1)
    G.log(f"underfull V={V} K={K} T={T}")
    sents = [0, 1, 2]
    if V > 2:
        g = G.GpuDecoder(cfg)
        dec = G.oracle_for(cfg, sents)
    else:                                     # no content words: empty posterior tables
        empty = (np.zeros(0, np.int32), np.zeros((0, 4), np.int32), np.zeros(0, np.float32))
        g = G.GpuDecoder(cfg, tables=[empty] * 3)
        dec = Decoder(cfg.V, K, cfg.lam, cfg.theta, [Posteriors(*empty)] * 3, keep_cand=True)
    W64 = synth.bf16_to_f32(G.weights(cfg)).astype(np.float64)
    for t in range(1, T + 1):
        gp, gt, gs = g.step()
        rec = dec.step(G.oracle_logits(cfg, sents, dec, W64))
        for b in sents:
            G.compare_step(rec, b, gp[b], gt[b], gs[b], tag=f"t={t} s={b}")
        g.inject(dec, sents)
    g.close()


@pytest.mark.parametrize("path", ["two_pass", "fused", "logits"])
def test_largest_vocabulary_and_beam(torch_cuda, path):
    """The documented maxima: V = 262144 (128 score strips of 2048 columns,
    eight 256-column tiles each) with K = 16, steps against the oracle from
    the same state, then a whole decode."""
    cfg = synth.Config("vmax", 45, B=2, K=16, V=262144, H=64, T=3, lam=1.0, theta=synth.THETA,
                       paths=40, path_len=6, zipf_a=1.1)
    G.log(f"largest V={cfg.V} K={cfg.K} ({path})")
    g = G.GpuDecoder(cfg, path=path)
    sents = [0, 1]
    dec = G.oracle_for(cfg, sents)
    W64 = synth.bf16_to_f32(G.weights(cfg)).astype(np.float64)
    n_exact = 0
    for t in range(1, cfg.T + 1):
        gp, gt, gs = g.step()
        rec = dec.step(G.oracle_logits(cfg, sents, dec, W64))
        for b in sents:
            n_exact += G.compare_step(rec, b, gp[b], gt[b], gs[b], tag=f"t={t} s={b}")
        g.inject(dec, sents)
    assert n_exact >= 0.9 * cfg.T * cfg.B * cfg.K
    g.close()


@pytest.mark.parametrize("K,V", [(1, 1001), (2, 4099), (16, 257)])
def test_odd_shapes_decode(torch_cuda, K, V):
    cfg = synth.Config(f"o{K}", 40 + K, B=5, K=K, V=V, H=128, T=12, lam=1.0, theta=synth.THETA,
                       paths=10, path_len=8, zipf_a=1.1)
    G.log(f"odd shapes K={K} V={V}")
    g = G.GpuDecoder(cfg)
    toks, lens, scs = _gpu_decode(g, cfg, cfg.T)
    sents = list(range(cfg.B))
    dec = decode_synthetic(cfg, sents, G.weights(cfg), [Posteriors(*G.posteriors(cfg, s)) for s in sents])
    for s in sents:
        best = dec.best(s)
        F = sorted((sc for _, _, sc in dec.finished(s)), reverse=True)
        gaps = [r.gap_k()[s] for r in dec.records if np.isfinite(r.top[s, K - 1])]
        if min(gaps) > G.GAP and (len(F) < 2 or F[0] - F[1] > G.GAP):
            assert tuple(toks[s, :lens[s]]) == best.tokens
            assert abs(scs[s] - best.score) < G.SCORE_TOL
    g.close()


@pytest.mark.parametrize("path", ["two_pass", "fused", "logits"])
def test_ties_zero_weights(torch_cuda, path):
    """W = 0: every logit is 0, so whole tiles tie at lambda*theta0 and only the
    posterior words stand out; ties are broken by (slot, word) index as in the
    oracle's total order.  In the fused kernel this drives the exact per-tile
    fallback (more values at the bound than candidate slots)."""
    cfg = synth.get_config("small").replace(B=4)
    G.log(f"zero weights ({path})")
    W0 = np.zeros((cfg.V, cfg.H), dtype=np.uint16)
    g = G.GpuDecoder(cfg, W=W0, path=path)
    sents = list(range(cfg.B))
    dec = G.oracle_for(cfg, sents)
    for t in range(1, 9):
        gp, gt, gs = g.step()
        rec = dec.step(np.zeros((cfg.B * cfg.K, cfg.V)))
        for b in sents:
            G.compare_step(rec, b, gp[b], gt[b], gs[b], tag=f"zero-W t={t} s={b}")
        g.inject(dec, sents)
    g.close()


@pytest.mark.parametrize("path", ["two_pass", "fused", "logits"])
def test_projection_bias_step(torch_cuda, path):
    """A projection bias b[V] is added to every row's logits before the score pass."""
    torch = torch_cuda
    cfg = synth.get_config("small").replace(B=6)
    G.log(f"projection bias ({path})")
    g = G.GpuDecoder(cfg)
    bias = np.random.default_rng(7).normal(0.0, 2.0, cfg.V).astype(np.float32)
    bias_d = torch.from_numpy(bias).cuda()
    g.P.lmbr_set_projection(g.ctx, g.W, 0, bias_d)
    sents = list(range(cfg.B))
    dec = G.oracle_for(cfg, sents)
    W64 = synth.bf16_to_f32(G.weights(cfg)).astype(np.float64)
    for t in range(1, 11):
        gp, gt, gs = g.step()
        x = G.oracle_logits(cfg, sents, dec, W64) + bias.astype(np.float64)[None, :]
        rec = dec.step(x)
        for b in sents:
            G.compare_step(rec, b, gp[b], gt[b], gs[b], tag=f"bias t={t} s={b}")
        g.inject(dec, sents)
    g.close()


def test_score_select_split(torch_cuda):
    """lmbr_score + lmbr_select is lmbr_beam_step (same kernels, bit for bit);
    a select without a score call is refused."""
    torch = torch_cuda
    import paper_1804_11324_amd as P
    cfg = synth.get_config("small").replace(B=5)
    G.log("score/select split")
    a = G.GpuDecoder(cfg)
    b = G.GpuDecoder(cfg)
    with pytest.raises(P.LmbrError) as ei:
        P.lmbr_select(b.ctx, b.st)
    assert ei.value.code == -4            # LMBR_E_STATE
    for t in range(6):
        pa, ta, sa = a.step()
        P.lmbr_synth_hidden(b.ctx, b.st, b.hidden)
        P.lmbr_score(b.ctx, b.st, b.hidden)
        P.lmbr_select(b.ctx, b.st, b.parent, b.token, b.score)
        torch.cuda.synchronize()
        assert np.array_equal(pa.ravel(), b.parent.cpu().numpy())
        assert np.array_equal(ta.ravel(), b.token.cpu().numpy())
        assert np.array_equal(sa.ravel(), b.score.cpu().numpy())
    with pytest.raises(P.LmbrError):
        P.lmbr_select(b.ctx, b.st)
    a.close()
    b.close()


def test_empty_tables_and_reload(torch_cuda):
    """No posteriors: L = theta0 everywhere; a reload replaces a table."""
    cfg = synth.get_config("tiny").replace(B=2)
    G.log("empty tables")
    empty = (np.zeros(0, np.int32), np.zeros((0, 4), np.int32), np.zeros(0, np.float32))
    g = G.GpuDecoder(cfg, tables=[empty, empty])
    sents = [0, 1]
    dec = Decoder(cfg.V, cfg.K, cfg.lam, cfg.theta, [Posteriors(), Posteriors()], keep_cand=True)
    W64 = synth.bf16_to_f32(G.weights(cfg)).astype(np.float64)
    for t in range(1, cfg.T + 1):
        gp, gt, gs = g.step()
        rec = dec.step(G.oracle_logits(cfg, sents, dec, W64))
        for b in sents:
            G.compare_step(rec, b, gp[b], gt[b], gs[b], tag=f"empty t={t} s={b}")
        g.inject(dec, sents)
    # load real tables and decode again from scratch
    for s in sents:
        g.P.lmbr_load_posteriors(g.ctx, s, *G.posteriors(cfg, s))
    toks, lens, scs = _gpu_decode(g, cfg, cfg.T)
    dec = decode_synthetic(cfg, sents, G.weights(cfg), [Posteriors(*G.posteriors(cfg, s)) for s in sents])
    for s in sents:
        assert tuple(toks[s, :lens[s]]) == dec.best(s).tokens
    g.close()


def test_gather_rows(torch_cuda):
    torch = torch_cuda
    import paper_1804_11324_amd as P
    G.log("gather rows")
    src = torch.arange(12 * 40, dtype=torch.float32, device="cuda").reshape(12, 40)
    rows = torch.tensor([3, 3, 0, 11, 7], dtype=torch.int32, device="cuda")
    dst = torch.empty((5, 40), dtype=torch.float32, device="cuda")
    P.lmbr_gather_rows(dst, src, rows, 5, 40 * 4)
    torch.cuda.synchronize()
    assert torch.equal(dst, src[rows.long()])
