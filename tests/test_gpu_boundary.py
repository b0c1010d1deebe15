"""The C ABI's boundary on the GPU: the device fault flag, a caller-provided
workspace and tables in caller memory, and the model hook of lmbr_decode (a decoder state the caller
computes and realigns by backpointer, the paper's GetMatrixByRows).

Marked gpu.  Inputs are seeded (synth); the oracle decodes the same model
independently in fp64 and follows the GPU's choices (check_selection)."""
import ctypes

import numpy as np
import pytest

import synth
from oracle.beam import Decoder, Posteriors, project
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


# --------------------------------------------------------------------------
# device fault flag (LMBR_E_DEVICE)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("bad", [float("inf"), float("nan")])
def test_nonfinite_logit_sets_device_flag(torch_cuda, bad):
    """A +inf or NaN logit of a live row (a caller's model gone wrong) makes
    that row's normaliser non-finite: the step completes, the flag reads
    LMBR_DEV_NONFINITE once, and a decode from a fresh state leaves it clear."""
    torch = torch_cuda
    import paper_1804_11324_amd as P
    cfg = synth.get_config("small").replace(B=3)
    G.log(f"device flag: logit {bad}")
    g = G.GpuDecoder(cfg, path="logits")
    g.step()
    assert P.lmbr_device_status(g.ctx) == 0
    P.lmbr_synth_hidden(g.ctx, g.st, g.hidden)
    P.lmbr_project(g.ctx, g.hidden, g.logits, g.ld)
    row = 1 * cfg.K + int(np.flatnonzero(np.isfinite(g.st.q.cpu().numpy()[cfg.K:2 * cfg.K]))[0])
    g.logits[row, 17] = bad
    P.lmbr_beam_step_logits(g.ctx, g.st, g.logits, g.ld)
    assert P.lmbr_device_status(g.ctx) == P.LMBR_DEV_NONFINITE
    assert P.lmbr_device_status(g.ctx) == 0          # read and cleared
    # the faulted step's scores are unspecified (NaN carries on in the running
    # scores, and later steps flag again); a new decode from a fresh state is clean
    P.lmbr_state_init(g.ctx, g.st, cfg.seed)
    g.step()
    g.step()
    assert P.lmbr_device_status(g.ctx) == 0
    g.close()


def test_decode_returns_device_error(torch_cuda):
    """lmbr_decode reads the flag at its end: a +inf projection bias on one
    word makes every live row's logits non-finite, and the decode returns
    LMBR_E_DEVICE (its outputs are still written)."""
    torch = torch_cuda
    import paper_1804_11324_amd as P
    cfg = synth.get_config("tiny")
    G.log("device flag through lmbr_decode")
    g = G.GpuDecoder(cfg)
    bias = torch.zeros(cfg.V, dtype=torch.float32, device="cuda")
    bias[5] = float("inf")
    P.lmbr_set_projection(g.ctx, g.W, 0, bias)
    toks = np.empty((cfg.B, cfg.T), np.int32)
    lens = np.empty(cfg.B, np.int32)
    scs = np.empty(cfg.B, np.float64)
    P.lmbr_state_init(g.ctx, g.st, cfg.seed)
    with pytest.raises(P.LmbrError) as ei:
        P.lmbr_decode(g.ctx, g.st, cfg.T, None, toks, lens, scs)
    assert ei.value.code == P.LMBR_E_DEVICE
    assert P.lmbr_device_status(g.ctx) == 0
    P.lmbr_set_projection(g.ctx, g.W, 0)              # a clean decode afterwards
    P.lmbr_state_init(g.ctx, g.st, cfg.seed)
    P.lmbr_decode(g.ctx, g.st, cfg.T, None, toks, lens, scs)
    g.close()


def test_bad_successor_range_sets_table_flag(torch_cuda):
    """A successor range outside the sentence's table (a state written by a
    caller, or restored from the wrong snapshot) is never read: the score
    pass skips it and raises LMBR_DEV_TABLE."""
    torch = torch_cuda
    import paper_1804_11324_amd as P
    cfg = synth.get_config("small").replace(B=2)
    G.log("device flag: bad successor range")
    for path in ("two_pass", "fused"):
        g = G.GpuDecoder(cfg, path=path)
        g.step()
        g.step()
        assert P.lmbr_device_status(g.ctx) == 0
        r = g.st.ranges.view(cfg.B * cfg.K, 6)
        live = int(np.flatnonzero(np.isfinite(g.st.q.cpu().numpy()))[0])
        r[live, 0] = 1 << 30                          # offset far past the table
        r[live, 1] = 4
        g.step()
        assert P.lmbr_device_status(g.ctx) & P.LMBR_DEV_TABLE
        g.close()


# --------------------------------------------------------------------------
# caller workspace
# --------------------------------------------------------------------------
def test_caller_workspace_decodes_identically(torch_cuda):
    """A context on a caller-owned workspace of lmbr_workspace_bytes(cfg) bytes
    decodes bit for bit as one that allocated its own, on both step paths."""
    torch = torch_cuda
    import paper_1804_11324_amd as P
    cfg = synth.get_config("small").replace(B=6, T=20)
    G.log("caller workspace")
    ccfg = P.make_config(cfg.B, cfg.K, cfg.V, cfg.H, cfg.T, 1, cfg.lam, cfg.theta, cfg.load_factor)
    n = P.lmbr_workspace_bytes(ccfg)
    ws = torch.full((n,), 0xAB, dtype=torch.uint8, device="cuda")   # not zeroed: the context sets what it needs
    outs = []
    for workspace in (None, ws):
        for path in (P.LMBR_STEP_TWO_PASS, P.LMBR_STEP_FUSED):
            ctx = P.lmbr_create(ccfg, workspace)
            W = torch.from_numpy(G.weights(cfg).view(np.int16)).cuda()
            P.lmbr_set_projection(ctx, W, 0)
            for s in range(cfg.B):
                P.lmbr_load_posteriors(ctx, s, *G.posteriors(cfg, s))
            P.lmbr_set_step_path(ctx, path)
            st = P.BeamState(ccfg)
            toks = np.empty((cfg.B, cfg.T), np.int32)
            lens = np.empty(cfg.B, np.int32)
            scs = np.empty(cfg.B, np.float64)
            P.lmbr_state_init(ctx, st, cfg.seed)
            P.lmbr_decode(ctx, st, cfg.T, None, toks, lens, scs)
            outs.append((toks, lens, scs, st.qhist.cpu().numpy()))
            if workspace is not None:
                assert P.lmbr_device_bytes(ctx) >= n
            ctx.close()
    for a, b in zip(outs[:2], outs[2:]):
        assert all(np.array_equal(x, y) for x, y in zip(a, b))


def test_tables_in_caller_memory(torch_cuda):
    """Posterior tables uploaded into caller-owned device memory of
    lmbr_table_bytes bytes (lmbr_load_posteriors_into) decode bit for bit as
    tables the library allocates, in the sparse and the dense layout; with a
    caller workspace too, the context then allocates nothing itself.  Too
    little memory is refused with LMBR_E_CAPACITY and changes nothing; an
    unaligned address is refused."""
    torch = torch_cuda
    import paper_1804_11324_amd as P
    cfg = synth.dense_evidence_config().replace(B=6, T=16)
    G.log(f"tables in caller memory: {cfg.name} B={cfg.B} V={cfg.V}")
    ccfg = P.make_config(cfg.B, cfg.K, cfg.V, cfg.H, cfg.T, 1, cfg.lam, cfg.theta, cfg.load_factor)
    tabs = [G.posteriors(cfg, s) for s in range(cfg.B)]
    W = torch.from_numpy(G.weights(cfg).view(np.int16)).cuda()
    for layout in (P.LMBR_L_SPARSE, P.LMBR_L_DENSE):
        outs, sizes = [], []
        for caller in (False, True):
            ws = torch.empty((P.lmbr_workspace_bytes(ccfg),), dtype=torch.uint8, device="cuda") if caller else None
            ctx = P.lmbr_create(ccfg, ws)
            P.lmbr_set_projection(ctx, W, 0)
            P.lmbr_set_lmbr_layout(ctx, layout)
            mems = []
            for s in range(cfg.B):
                if not caller:
                    P.lmbr_load_posteriors(ctx, s, *tabs[s])
                    continue
                nb = P.lmbr_table_bytes(ctx, *tabs[s])
                assert nb > 0 and nb % 256 == 0
                sizes.append(nb)
                mem = torch.empty((nb + 512,), dtype=torch.uint8, device="cuda")
                if s == 0:
                    with pytest.raises(P.LmbrError) as e:
                        P.lmbr_load_posteriors_into(ctx, s, *tabs[s], mem, nb - 256)
                    assert e.value.code == P.LMBR_E_CAPACITY
                    with pytest.raises(P.LmbrError) as e:
                        P.lmbr_load_posteriors_into(ctx, s, *tabs[s], mem[16:], nb)
                    assert e.value.code == P.LMBR_E_INVALID
                P.lmbr_load_posteriors_into(ctx, s, *tabs[s], mem, nb)
                mems.append(mem)
            if caller:
                assert P.lmbr_device_bytes(ctx) == P.lmbr_workspace_bytes(ccfg) + sum(sizes)
            st = P.BeamState(ccfg)
            toks = np.empty((cfg.B, cfg.T), np.int32)
            lens = np.empty(cfg.B, np.int32)
            scs = np.empty(cfg.B, np.float64)
            P.lmbr_state_init(ctx, st, cfg.seed)
            P.lmbr_decode(ctx, st, cfg.T, None, toks, lens, scs)
            outs.append((toks, lens, scs, st.qhist.cpu().numpy()))
            ctx.close()
            del mems, ws
        assert all(np.array_equal(x, y) for x, y in zip(*outs)), f"layout {layout}"
        G.log(f"  layout {layout}: table bytes {min(sizes)}..{max(sizes)}, decodes identical")


# --------------------------------------------------------------------------
# model hook: lmbr_state_fn + lmbr_gather_rows
# --------------------------------------------------------------------------
def test_state_fn_builtin_model_matches_null(torch_cuda):
    """A state_fn that calls the built-in stand-in itself decodes bit for bit
    as state_fn = NULL (the graph-captured loop)."""
    torch = torch_cuda
    import paper_1804_11324_amd as P
    cfg = synth.get_config("small").replace(B=5, T=24)
    G.log("state_fn: built-in stand-in through the hook")
    g = G.GpuDecoder(cfg)
    ref = _decode(g, cfg, None)
    calls = []

    def fn(t, stp, hidden, stream):
        calls.append(t)
        assert stp.contents.t == t
        return P.lib().lmbr_synth_hidden(g.ctx.handle, stp, hidden, stream)

    got = _decode(g, cfg, fn)
    assert calls == list(range(cfg.T))
    assert all(np.array_equal(x, y) for x, y in zip(ref, got))
    # a non-zero return stops the decode with that value
    with pytest.raises(P.LmbrError) as ei:
        _decode(g, cfg, lambda t, stp, hidden, stream: -4 if t == 3 else
                P.lib().lmbr_synth_hidden(g.ctx.handle, stp, hidden, stream))
    assert ei.value.code == -4 and g.st.t == 3
    g.close()


def _decode(g, cfg, fn):
    toks = np.empty((cfg.B, g.T_max), np.int32)
    lens = np.empty(cfg.B, np.int32)
    scs = np.empty(cfg.B, np.float64)
    g.P.lmbr_state_init(g.ctx, g.st, cfg.seed)
    g.P.lmbr_decode(g.ctx, g.st, cfg.T, None, toks, lens, scs, state_fn=fn)
    return toks, lens, scs


def _embeddings(cfg, tag):
    """bf16 [V, H] rows of N(0,1) stand-in embeddings (seeded, synth's generator)."""
    return synth.hidden_from_hashes(np.arange(cfg.V, dtype=np.uint64) * np.uint64(0x9E37) +
                                    np.uint64(synth.mix(cfg.seed * 31 + tag)), cfg.H)


def _two_word_hidden(E1, E2, hist):
    """Oracle side of the hooked model: bf16(E1[last word] + E2[word before]),
    each term a zero row when the history is too short (fp32 sum, then
    round-to-nearest-even to bf16)."""
    H = E1.shape[1]
    a = synth.bf16_to_f32(E1[hist[-1]]) if len(hist) >= 1 else np.zeros(H, np.float32)
    b = synth.bf16_to_f32(E2[hist[-2]]) if len(hist) >= 2 else np.zeros(H, np.float32)
    return synth.bf16_to_f32(synth.bf16_bits((a + b).astype(np.float32)))


@pytest.mark.parametrize("name", ["small", "base"])
def test_state_fn_recurrent_model_parity(torch_cuda, name):
    """A caller's model through the hook: its state per slot (the last word and
    the word before it) lives in caller buffers and is realigned each step by
    lmbr_gather_rows with the step's backpointers (GetMatrixByRows(S_t, b_t));
    its decoder state is bf16(E1[y_{t-1}] + E2[y_{t-2}]), computed with torch.
    The oracle runs the same model in numpy, follows the GPU's choices and
    checks every step's selections and the final hypotheses."""
    torch = torch_cuda
    import paper_1804_11324_amd as P
    cfg = synth.get_config(name).replace(B=8, T=30)
    sents = [0, 3, 7]
    G.log(f"state_fn: two-word model ({name}), B={cfg.B} K={cfg.K} V={cfg.V} T={cfg.T}")
    E1, E2 = _embeddings(cfg, 1), _embeddings(cfg, 2)
    g = G.GpuDecoder(cfg)
    M, K, H = cfg.B * cfg.K, cfg.K, cfg.H
    e1 = torch.from_numpy(synth.bf16_to_f32(E1)).cuda()
    e2 = torch.from_numpy(synth.bf16_to_f32(E2)).cuda()
    zero = torch.zeros((1, H), dtype=torch.float32, device="cuda")
    e1z, e2z = torch.cat([e1, zero]), torch.cat([e2, zero])     # row V: no word
    last = torch.full((M,), cfg.V, dtype=torch.int32, device="cuda")
    prev = torch.full((M,), cfg.V, dtype=torch.int32, device="cuda")
    prev_new = torch.empty_like(prev)
    base_row = (torch.arange(M, device="cuda", dtype=torch.int32) // K) * K
    hid = torch.empty((M, H), dtype=torch.bfloat16, device="cuda")
    ident = torch.arange(M, dtype=torch.int32, device="cuda")

    def fn(t, stp, hidden, stream):
        if t == 0:
            last.fill_(cfg.V)
            prev.fill_(cfg.V)
        else:
            rows = base_row + g.st.bp[(t - 1) * M:t * M]
            # the parent's last word becomes the new slot's word before last
            P.lmbr_gather_rows(prev_new, last, rows, M, 4)
            prev.copy_(prev_new)
            last.copy_(g.st.tok[(t - 1) * M:t * M])
        hid.copy_((e1z[last.long()] + e2z[prev.long()]).to(torch.bfloat16))
        return P.lib().lmbr_gather_rows(hidden, hid.data_ptr(), ident.data_ptr(), M, H * 2, stream)

    toks, lens, scs = _decode(g, cfg, fn)
    bp = g.st.bp.cpu().numpy().reshape(g.T_max, cfg.B, K)
    tk = g.st.tok.cpu().numpy().reshape(g.T_max, cfg.B, K)
    qh = g.st.qhist.cpu().numpy().reshape(g.T_max, cfg.B, K)
    g.close()

    W64 = synth.bf16_to_f32(G.weights(cfg)).astype(np.float64)
    tables = [Posteriors(*G.posteriors(cfg, s)) for s in sents]
    dec = Decoder(cfg.V, K, cfg.lam, cfg.theta, tables, keep_cand=True)
    for t in range(1, cfg.T + 1):
        x = np.zeros((len(sents) * K, cfg.V))
        for b in range(len(sents)):
            for k in range(K):
                if dec.q[b, k] > -np.inf:
                    h = _two_word_hidden(E1, E2, dec.hist[b][k]).astype(np.float64)
                    x[b * K + k] = project(W64, h[None, :])[0]
        ob = np.array([synth.eos_bias(cfg, t, s) for s in sents])
        rec = dec.step(x, ob if np.any(ob) else None, force=(bp[t - 1][sents], tk[t - 1][sents]))
        for b, s in enumerate(sents):
            G.check_selection(rec.cand[b], rec.top[b], bp[t - 1, s], tk[t - 1, s], qh[t - 1, s],
                              tag=f"{name} t={t} s={s}")
    for b, s in enumerate(sents):
        best = dec.best(b)
        assert abs(scs[s] - best.score) <= G.SCORE_TOL
        F = sorted((sc for _, _, sc in dec.finished(b)), reverse=True)
        if len(F) < 2 or F[0] - F[1] > G.GAP:
            assert tuple(int(v) for v in toks[s, :lens[s]]) == best.tokens
