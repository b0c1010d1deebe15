"""Unit tests of the seeded input generator (no GPU)."""
import numpy as np
import pytest
import torch

import synth


def test_splitmix64_published_sequence():
    # SplitMix64 seeded with 0: the generator's state advances by the golden
    # gamma and each output is mix(state before the add); the first outputs of
    # the published reference generator for seed 0 are these.
    expect = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    got = [synth.mix((i * synth.GOLDEN) & synth.M64) for i in range(3)]
    assert got == expect
    vec = synth.mix_np(np.array([(i * synth.GOLDEN) & synth.M64 for i in range(3)], dtype=np.uint64))
    assert [int(x) for x in vec] == expect


def test_mix_np_matches_scalar():
    rng = np.random.default_rng(1)
    z = rng.integers(0, 2 ** 63, size=1000, dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    assert [int(x) for x in synth.mix_np(z)] == [synth.mix(int(x)) for x in z]


def test_irwin_hall_exact_and_moments():
    h = np.arange(200000, dtype=np.uint64) * np.uint64(7919)
    v = synth.irwin_hall_np(h)
    assert v.dtype == np.float32
    # exact: an integer multiple of 2**-20 inside [-6, 6]
    i = v.astype(np.float64) * 2.0 ** 20
    assert np.all(i == np.round(i))
    assert np.all(np.abs(v) <= 6.0)
    assert abs(v.mean()) < 0.01 and abs(v.var() - 1.0) < 0.02
    # scalar and vector forms agree
    for x in [0, 1, 12345, 2 ** 63 + 5]:
        assert synth.irwin_hall_int(x) * 2.0 ** -20 == float(synth.irwin_hall_np(np.array([x], dtype=np.uint64))[0])


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.0e-3], dtype=np.float32)
    b = synth.bf16_bits(x)
    assert b[0] == 0x3F80 and b[1] == 0x3F80 and b[2] == 0x3F82
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    assert np.array_equal(b, ref)
    rng = np.random.default_rng(0)
    y = rng.standard_normal(100000).astype(np.float32)
    ref = torch.from_numpy(y).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    assert np.array_equal(synth.bf16_bits(y), ref)
    assert np.array_equal(synth.bf16_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_weights_scale_and_determinism():
    cfg = synth.get_config("tiny")
    W = synth.make_weights(cfg)
    assert W.shape == (cfg.V, cfg.H) and W.dtype == np.uint16
    w = synth.bf16_to_f32(W)
    assert abs(w.std() * np.sqrt(cfg.H) - 1.0) < 0.05
    assert np.array_equal(W, synth.make_weights(cfg))
    # element (v, i) follows its definition
    v, i = 17, 5
    h = synth.mix((synth.mix(cfg.seed + synth.TAG_W) + v * cfg.H + i) & synth.M64)
    val = np.float32(synth.irwin_hall_int(h) * 2.0 ** -20) * synth.inv_sqrt_f32(cfg.H)
    assert W[v, i] == synth.bf16_bits(np.array([val], dtype=np.float32))[0]


def test_hidden_state_follows_history_hash():
    cfg = synth.get_config("small")
    hist = (5, 17, 1999)
    hh = synth.initial_hash(cfg, 3)
    for y in hist:
        hh = synth.mix(hh ^ (y + 1))
    assert hh == synth.history_hash(cfg, 3, hist)
    row = synth.hidden_state(cfg, 3, hist)
    assert row.shape == (cfg.H,)
    i = 7
    val = np.float32(synth.irwin_hall_int(synth.mix((hh + i) & synth.M64)) * 2.0 ** -20)
    assert row[i] == synth.bf16_bits(np.array([val]))[0]
    # different histories give different states
    assert not np.array_equal(row, synth.hidden_state(cfg, 3, (5, 17, 1998)))


@pytest.mark.parametrize("name,lo,hi", [("tiny", 600, 900), ("small", 20000, 27000)])
def test_posteriors_invariants(name, lo, hi):
    cfg = synth.get_config(name)
    paths, w = synth.make_lattice(cfg, 0)
    assert paths.shape == (cfg.paths, cfg.path_len + 1)
    assert np.all(paths[:, -1] == synth.EOS)
    assert np.all((paths[:, :-1] >= 2) & (paths[:, :-1] < cfg.V))
    assert abs(w.sum() - 1.0) < 1e-12 and np.all(w > 0)
    order, toks, post = synth.posteriors(cfg, 0)
    assert lo <= len(order) <= hi
    assert np.all(post > 0) and np.all(post <= 1.0)
    d = synth.ngram_dict(order, toks, post)
    assert len(d) == len(order)                       # no duplicates
    # every 1..4-gram on every path is present, with the summed path weight
    for p in range(0, cfg.paths, max(1, cfg.paths // 7)):
        row = paths[p].tolist()
        for n in range(1, 5):
            for i in range(len(row) - n + 1):
                assert tuple(row[i:i + n]) in d
    g = tuple(paths[0, :2].tolist())
    expect = sum(w[p] for p in range(cfg.paths)
                 if any(tuple(paths[p, i:i + 2]) == g for i in range(paths.shape[1] - 1)))
    assert d[g] == min(np.float32(expect), np.float32(1.0))
    # posterior never grows when an n-gram is extended on either side
    for gram, p in d.items():
        if len(gram) > 1:
            assert p <= d[gram[1:]] and p <= d[gram[:-1]]


def test_eos_bias_schedule():
    cfg = synth.get_config("base")
    tab = synth.eos_bias_table(cfg)
    assert tab.shape == (cfg.T, cfg.B)
    assert np.all(tab[:30] == 0)
    assert np.all(tab[30:, 1::2] == 6.0) and np.all(tab[30:, 0::2] == 0)
    assert np.all(synth.eos_bias_table(synth.get_config("small")) == 0)
