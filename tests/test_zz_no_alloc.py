"""lmbr_beam_step_logits_static (allocates nothing: partials in the library's
static device scratch) against lmbr_beam_step_logits, through the C ABI.

Two calls in a row on one GPU, the second with a smaller input (a smaller
context), each compared bit for bit with the workspace entry point from the
same state; plus the capacity refusal, which launches nothing."""
import numpy as np
import pytest

import synth
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


def _twin_step(torch, P, cfg, steps_before, options=None):
    """Two identical decoders; after `steps_before` ordinary steps, one more
    step through each entry point from the same state and the same logits."""
    a = G.GpuDecoder(cfg, path="logits")
    b = G.GpuDecoder(cfg, path="logits")
    for g in (a, b):
        if options:
            P.lmbr_set_decode_options(g.ctx, **options)
            P.lmbr_state_init(g.ctx, g.st, cfg.seed)
        for _ in range(steps_before):
            g.step()
    P.lmbr_synth_hidden(a.ctx, a.st, a.hidden)
    P.lmbr_project(a.ctx, a.hidden, a.logits, a.ld)
    logits = a.logits.clone()
    P.lmbr_beam_step_logits(a.ctx, a.st, logits, a.ld, None, a.parent, a.token, a.score)
    P.lmbr_beam_step_logits_static(b.ctx, b.st, logits, a.ld, None, b.parent, b.token, b.score)
    torch.cuda.synchronize()
    for x, y in ((a.parent, b.parent), (a.token, b.token), (a.score, b.score), (a.st.q, b.st.q),
                 (a.st.ctx, b.st.ctx), (a.st.hhash, b.st.hhash), (a.st.len, b.st.len),
                 (a.st.ranges, b.st.ranges), (a.st.bp, b.st.bp), (a.st.tok, b.st.tok),
                 (a.st.qhist, b.st.qhist), (a.st.sent.view(torch.int64), b.st.sent.view(torch.int64))):
        assert torch.equal(x, y)          # bit for bit (the records pack int32 fields: compared as bits)
    assert a.st.t == b.st.t == steps_before + 1
    # and the next ordinary step continues identically from either state
    pa, ta, sa = a.step()
    pb, tb, sb = b.step()
    assert np.array_equal(pa, pb) and np.array_equal(ta, tb) and np.array_equal(sa, sb)
    a.close()
    b.close()


def test_static_step_matches_workspace_step_twice(torch_cuda):
    torch = torch_cuda
    import paper_1804_11324_amd as P
    big = synth.get_config("large").replace(B=96, H=256, paths=200, path_len=30)
    small = synth.get_config("small").replace(B=3, V=5003, H=128)
    for cfg, before in ((big, 3), (small, 5)):
        need = P.lmbr_static_scratch_bytes(P.make_config(cfg.B, cfg.K, cfg.V, cfg.H, cfg.T))
        G.log(f"static-scratch step: B={cfg.B} K={cfg.K} V={cfg.V} ({need} bytes of scratch)")
        assert 0 < need <= P._abi.LMBR_STATIC_SCRATCH_BYTES
        _twin_step(torch, P, cfg, before)
    # the backup stack's EOS column lives in the scratch too
    _twin_step(torch, P, small, 4, dict(finish=P.LMBR_FINISH_EOS_BACKUP))


def test_static_step_refuses_oversized_configs(torch_cuda):
    torch = torch_cuda
    import paper_1804_11324_amd as P
    cfg = synth.Config("nx", 95, B=2048, K=16, V=1000, H=64, T=2, lam=1.0, theta=synth.THETA,
                       paths=2, path_len=3, zipf_a=1.1)
    ccfg = P.make_config(cfg.B, cfg.K, cfg.V, cfg.H, cfg.T)
    assert P.lmbr_static_scratch_bytes(ccfg) > P._abi.LMBR_STATIC_SCRATCH_BYTES
    G.log("static-scratch step: oversized configuration refused")
    g = G.GpuDecoder(cfg, path="logits", tables=[(np.zeros(0, np.int32), np.zeros((0, 4), np.int32),
                                                  np.zeros(0, np.float32))] * cfg.B)
    before = g.st.q.clone()
    with pytest.raises(P.LmbrError) as ei:
        P.lmbr_beam_step_logits_static(g.ctx, g.st, g.logits, g.ld)
    assert ei.value.code == -2 and g.st.t == 0
    torch.cuda.synchronize()
    assert torch.equal(before, g.st.q)
    g.close()
