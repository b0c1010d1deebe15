"""The C ABI on the CPU: exported symbols, host table construction, validation.

No GPU calls are made here (lmbr_table_build is host-only)."""
import os
import re

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lmbr.h")


@pytest.fixture(scope="module")
def P():
    import paper_1804_11324_amd as P
    P.lib()
    return P


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lmbr_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function(P):
    import ctypes
    names = declared_functions()
    assert len(names) >= 15
    lib = ctypes.CDLL(P._abi.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in lmbr.h but not exported"
    assert sorted(P._abi.EXPORTS) == names


def test_header_constants_match_binding(P):
    text = open(HEADER).read()
    for name, val in [("LMBR_MAX_K", P._abi.LMBR_MAX_K), ("LMBR_MAX_V", P._abi.LMBR_MAX_V)]:
        m = re.search(rf"#define {name}\s+(\d+)", text)
        assert m and int(m.group(1)) == val
    for name, val in [("LMBR_OK", 0), ("LMBR_E_INVALID", -1), ("LMBR_E_CAPACITY", -2),
                      ("LMBR_E_HIP", -3), ("LMBR_E_STATE", -4), ("LMBR_E_DEVICE", P._abi.LMBR_E_DEVICE),
                      ("LMBR_DEV_NONFINITE", P._abi.LMBR_DEV_NONFINITE),
                      ("LMBR_DEV_TABLE", P._abi.LMBR_DEV_TABLE)]:
        assert re.search(rf"{name}\s*=\s*{val}\b", text), name


def _probe(img, key):
    """Linear probing as documented in lmbr.h: slot = SplitMix64(key) & (cap-1)."""
    cap = img["slot_key"].shape[0]
    h = synth.mix(key) & (cap - 1)
    for _ in range(cap):
        k = int(img["slot_key"][h])
        if k == key:
            return int(img["slot_off"][h]), int(img["slot_cnt"][h])
        if k == (1 << 64) - 1:
            return None
        h = (h + 1) & (cap - 1)
    return None


def _pack(words):
    key = 0
    for w in words:
        key = (key << 21) | (w + 1)
    return key


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_table_build_matches_ngram_dict(P, name):
    cfg = synth.get_config(name)
    order, toks, post = synth.posteriors(cfg, 3)
    img = P.lmbr_table_build(cfg.V, order, toks, post, 0.5)
    d = synth.ngram_dict(order, toks, post)
    succ = {}
    for gram, p in d.items():
        succ.setdefault(gram[:-1], []).append((gram[-1], p))
    n_ctx = sum(1 for h in succ if h)
    cap = img["slot_key"].shape[0]
    assert cap & (cap - 1) == 0 and n_ctx / cap <= 0.5
    assert int(np.sum(img["slot_key"] != np.uint64(2 ** 64 - 1))) == n_ctx
    for hist, lst in succ.items():
        lst.sort()
        if hist == ():
            off, cnt = img["uni_off"], img["uni_cnt"]
        else:
            r = _probe(img, _pack(hist))
            assert r is not None, hist
            off, cnt = r
        assert cnt == len(lst)
        assert img["entry_tok"][off:off + cnt].tolist() == [w for w, _ in lst]
        assert np.array_equal(img["entry_post"][off:off + cnt], np.array([p for _, p in lst], np.float32))
    # histories that are not in the evidence space miss
    rng = np.random.default_rng(0)
    for _ in range(200):
        h = tuple(int(x) for x in rng.integers(2, cfg.V, size=rng.integers(1, 4)))
        if h not in succ:
            assert _probe(img, _pack(h)) is None


def test_table_build_empty(P):
    img = P.lmbr_table_build(100, np.zeros(0, np.int32), np.zeros((0, 4), np.int32), np.zeros(0, np.float32))
    assert img["uni_cnt"] == 0 and img["entry_tok"].size == 0
    assert np.all(img["slot_key"] == np.uint64(2 ** 64 - 1))


@pytest.mark.parametrize("order,tokens,post,msg", [
    ([1, 1], [[3, -1, -1, -1], [3, -1, -1, -1]], [0.5, 0.4], "duplicate"),
    ([2], [[3, 100, -1, -1]], [0.5], "outside"),
    ([1], [[-1, -1, -1, -1]], [0.5], "outside"),
    ([1], [[3, -1, -1, -1]], [0.0], "posterior"),
    ([1], [[3, -1, -1, -1]], [1.5], "posterior"),
    ([1], [[3, -1, -1, -1]], [float("nan")], "posterior"),
    ([0], [[3, -1, -1, -1]], [0.5], "order"),
    ([5], [[3, 4, 5, 6]], [0.5], "order"),
])
def test_table_build_rejects_bad_input(P, order, tokens, post, msg):
    with pytest.raises(P.LmbrError) as e:
        P.lmbr_table_build(100, np.array(order), np.array(tokens), np.array(post, np.float32))
    assert e.value.code == -1 and msg in str(e.value)


def test_table_build_rejects_bad_load_factor(P):
    with pytest.raises(P.LmbrError):
        P.lmbr_table_build(100, np.array([1]), np.array([[3, -1, -1, -1]]), np.array([0.5], np.float32), 0.95)


@pytest.mark.parametrize("kw,code", [(dict(K=17), -2), (dict(K=0), -2), (dict(V=1), -2),
                                     (dict(V=300000), -2), (dict(H=100), -1), (dict(H=0), -1),
                                     (dict(T_max=0), -1), (dict(eos_id=1000), -1), (dict(B=0), -1)])
def test_create_validates_config_before_device(P, kw, code):
    base = dict(B=1, K=4, V=1000, H=64, T_max=10, eos_id=1)
    base.update(kw)
    with pytest.raises(P.LmbrError) as e:
        P.lmbr_create(P.make_config(**base))
    assert e.value.code == code


def test_host_only_lmbr_table_pack_convention():
    # histories are packed oldest first with the newest word lowest; the
    # device packs a slot's last words the same way when it extends them
    assert _pack((7,)) == 8
    assert _pack((7, 9)) == (8 << 21) | 10
    c = 0
    for y in (5, 7, 9, 11):
        c = ((c << 21) | (y + 1)) & ((1 << 63) - 1)
    assert c == _pack((7, 9, 11))


def test_workspace_bytes_host_only(P):
    """lmbr_workspace_bytes is host arithmetic: 0 (with the reason) for an invalid
    config, else at least the step buffers the header lists (the two-pass
    step's logits dominate: M x ceil(V/64)*64 floats)."""
    assert P.lmbr_workspace_bytes(P.make_config(0, 4, 1000, 64, 10)) == 0
    assert b"B=0" in P.lib().lmbr_last_error(None)
    for B, K, V, H, T in [(1, 4, 1000, 64, 10), (256, 8, 64000, 1024, 128), (3, 16, 257, 128, 5)]:
        n = P.lmbr_workspace_bytes(P.make_config(B, K, V, H, T))
        M = B * K
        assert n % 256 == 0
        assert n >= M * ((V + 63) // 64 * 64) * 4 + M * H * 2 + B * T * 4


def test_create_checks_workspace_before_device(P):
    """A caller workspace that is too small or misaligned is refused before any
    device call (the pointers are never touched)."""
    import ctypes
    cfg = P.make_config(2, 4, 1000, 64, 10)
    need = P.lmbr_workspace_bytes(cfg)
    h = ctypes.c_void_p()
    assert P.lib().lmbr_create(ctypes.byref(cfg), 1 << 20, need - 256, ctypes.byref(h)) == -2
    assert b"needed" in P.lib().lmbr_last_error(None)
    assert P.lib().lmbr_create(ctypes.byref(cfg), (1 << 20) + 16, need, ctypes.byref(h)) == -1
    assert h.value is None


@pytest.mark.parametrize("name", ["tiny", "small"])
def test_dense_rows_match_oracle_lmbr_row(P, name):
    """Section 2's dense arrangement (lmbr_table_dense): every history's row,
    plus lambda * theta0, is lambda times the oracle's L row of that history;
    and any hypothesis -- including histories absent from the evidence space --
    gets its L row from the row of its longest last-words suffix that is a
    history of the table (the rule the dense layout's probes follow)."""
    from oracle.beam import Posteriors
    cfg = synth.get_config(name).replace(paths=17, path_len=12)
    order, toks, post = synth.posteriors(cfg, 3)
    lam = 1.5
    ld = (cfg.V + 255) // 256 * 256
    img = P.lmbr_table_build(cfg.V, order, toks, post, dense_ld=ld, dense_lambda=lam, dense_theta=cfg.theta)
    rows, slot_row = img["dense"]["rows"], img["dense"]["slot_row"]
    occupied = img["slot_key"] != (1 << 64) - 1
    assert rows.shape[0] == 1 + occupied.sum() <= 500
    assert np.all(rows[:, cfg.V:] == 0)
    oracle = Posteriors(order, toks, post)

    def words(key):
        w = []
        while key:
            w.append((key & ((1 << 21) - 1)) - 1)
            key >>= 21
        return tuple(reversed(w))

    def row_of(hist):
        for n in range(min(3, len(hist)), 0, -1):
            k = _pack(hist[len(hist) - n:])
            r = _probe_slot(img, k)
            if r is not None:
                return int(slot_row[r])
        return 0

    lth0 = np.float32(lam * cfg.theta[0])
    hists = [()] + [words(int(k)) for k in img["slot_key"][occupied]]
    rng = np.random.default_rng(4)
    for _ in range(200):                      # random hypotheses: mostly unseen contexts
        base = hists[rng.integers(len(hists))]
        extra = tuple(int(x) for x in rng.integers(2, cfg.V, size=rng.integers(0, 3)))
        hists.append((base + extra)[-rng.integers(1, 5):] if base + extra else ())
    for h in hists:
        want = lam * oracle.lmbr_row(h, cfg.V, cfg.theta)
        got = (rows[row_of(h), :cfg.V] + lth0).astype(np.float64)
        assert np.max(np.abs(got - want)) < 2e-6, h
    # each occupied slot's row is its own history's
    assert sorted(slot_row[occupied].tolist()) == list(range(1, rows.shape[0]))


def _probe_slot(img, key):
    cap = img["slot_key"].shape[0]
    h = synth.mix(key) & (cap - 1)
    for _ in range(cap):
        k = int(img["slot_key"][h])
        if k == key:
            return h
        if k == (1 << 64) - 1:
            return None
        h = (h + 1) & (cap - 1)
    return None


@pytest.mark.parametrize("sorted_", [True, False])
def test_plan_batches(P, sorted_):
    """lmbr_plan_batches: a stable length sort (or corpus order) cut into
    batches of B, each batch decoded for its longest sentence."""
    cfg = synth.get_config("base")
    lengths = synth.corpus_lengths(cfg, 203, 10)
    assert lengths.min() >= 10 and lengths.max() <= cfg.T
    order, steps = P.lmbr_plan_batches(lengths, 64, sorted_)
    want = sorted(range(203), key=lambda i: -lengths[i]) if sorted_ else list(range(203))
    assert order.tolist() == want
    assert steps.tolist() == [int(lengths[want[b:b + 64]].max()) for b in range(0, 203, 64)]
    if sorted_:
        _, unsorted_steps = P.lmbr_plan_batches(lengths, 64, False)
        assert steps.sum() <= unsorted_steps.sum()
    with pytest.raises(P.LmbrError):
        P.lmbr_plan_batches(np.array([3, 0], np.int32), 2)
