"""Seeded synthetic inputs for the LMBR batched beam decoder.

This module is the one source of inputs shared by the fp64 oracle (``oracle/``)
and the HIP path (``paper_1804_11324_amd``).  It holds none of the decoder's
arithmetic: no projection, no log-softmax, no LMBR lookup, no top-K, no EOS
handling.  It produces

* the five workload configurations (sentences B, beams K, vocabulary V, hidden
  size H, steps T, LMBR weights, lattice recipe),
* the output projection W (bf16 bit patterns, [V, H]),
* per-sentence lattice paths and the n-gram posteriors computed from them,
* the stand-in decoder state: a hidden vector per (sentence, token history),
  drawn by hashing.  The HIP library has its own implementation of this
  generator (it runs inside the decode loop); both follow the published
  definitions of SplitMix64 (Steele, Lea and Flood, "Fast splittable
  pseudorandom number generators", OOPSLA 2014; output function as given by
  Vigna) and of the Irwin-Hall sum of uniforms.

The paper's workload (WMT17 newstest-2017 with 200-best PBMT posteriors, and a
trained GRU/Transformer model; Section 4.1 and 4.3) is not available here; these
inputs stand in for it with the shapes of Section 4.3's deployment setting.

Generator definitions
---------------------
mix(z): SplitMix64 output function on z + golden gamma (all mod 2**64).
IH(h): 12 uniforms of 20 bits taken from mix(h), ..., mix(h+3) (three per
       word, bits 0-19, 20-39, 40-59), summed, centred by 6*(2**20-1) and
       scaled by 2**-20: an exact fp32 value with mean 0 and variance ~1.
Seeds: S = 180411324 + config index; domain tags 'H' 0x48, 'W' 0x57,
       'P' 0x50, 'G' 0x47.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Sequence, Tuple

import numpy as np

M64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
MUL1 = 0xBF58476D1CE4E5B9
MUL2 = 0x94D049BB133111EB
SEED_BASE = 180411324
TAG_H, TAG_W, TAG_P, TAG_G, TAG_L = 0x48, 0x57, 0x50, 0x47, 0x4C
EOS = 1


# --------------------------------------------------------------------------
# SplitMix64 and Irwin-Hall, scalar (Python int) and vectorised (numpy uint64)
# --------------------------------------------------------------------------
def mix(z: int) -> int:
    """SplitMix64 output function applied to z (Python int, mod 2**64)."""
    z = (z + GOLDEN) & M64
    z = ((z ^ (z >> 30)) * MUL1) & M64
    z = ((z ^ (z >> 27)) * MUL2) & M64
    return z ^ (z >> 31)


def mix_np(z: np.ndarray) -> np.ndarray:
    """Vectorised SplitMix64 output function (uint64 arithmetic wraps)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = z + np.uint64(GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(MUL1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(MUL2)
    return z ^ (z >> np.uint64(31))


def irwin_hall_int(h: int) -> int:
    """Centred integer Irwin-Hall(12) sum from hash h; value is this * 2**-20."""
    s = 0
    for r in range(4):
        w = mix((h + r) & M64)
        for c in range(3):
            s += (w >> (20 * c)) & 0xFFFFF
    return s - 6 * (2 ** 20 - 1)


def irwin_hall_np(h: np.ndarray) -> np.ndarray:
    """Vectorised Irwin-Hall normal: fp32 values (exact) for uint64 hashes h."""
    h = np.asarray(h, dtype=np.uint64)
    s = np.zeros(h.shape, dtype=np.int64)
    mask = np.uint64(0xFFFFF)
    with np.errstate(over="ignore"):
        for r in range(4):
            w = mix_np(h + np.uint64(r))
            for c in range(3):
                s += ((w >> np.uint64(20 * c)) & mask).astype(np.int64)
    s -= 6 * (2 ** 20 - 1)
    return (s.astype(np.float32) * np.float32(2.0 ** -20)).astype(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); uint16 bits.

    Inputs are finite (the generator never produces inf or NaN)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    with np.errstate(over="ignore"):
        return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


# --------------------------------------------------------------------------
# Workload configurations
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    index: int          # 0..4, also the seed offset
    B: int              # sentences
    K: int              # beams per sentence
    V: int              # vocabulary
    H: int              # decoder hidden size
    T: int              # decode steps
    lam: float          # weight of the LMBR term
    theta: Tuple[float, float, float, float, float]   # theta0..theta4
    paths: int          # lattice paths per sentence
    path_len: int       # words per path (EOS appended)
    zipf_a: float
    load_factor: float = 0.5
    eos_boost: float = 0.0      # added to the EOS logit of odd sentences ...
    eos_boost_from: int = 0     # ... from this 1-based step on (0 = never)

    @property
    def seed(self) -> int:
        return SEED_BASE + self.index

    @property
    def M(self) -> int:
        return self.B * self.K

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


THETA = (-0.5, 1.0, 0.8, 0.6, 0.4)

CONFIGS = [
    Config("tiny", 0, B=1, K=4, V=1000, H=64, T=10, lam=1.0, theta=THETA,
           paths=20, path_len=12, zipf_a=1.1),
    Config("small", 1, B=16, K=4, V=32000, H=512, T=64, lam=1.0, theta=THETA,
           paths=200, path_len=40, zipf_a=1.1),
    Config("base", 2, B=64, K=4, V=32000, H=512, T=100, lam=1.0, theta=THETA,
           paths=500, path_len=40, zipf_a=1.1, eos_boost=6.0, eos_boost_from=31),
    Config("big", 3, B=64, K=12, V=32000, H=1024, T=100, lam=1.0, theta=THETA,
           paths=500, path_len=40, zipf_a=1.1),
    Config("large", 4, B=256, K=8, V=64000, H=1024, T=128, lam=1.5, theta=THETA,
           paths=1000, path_len=60, zipf_a=1.05),
]
BY_NAME = {c.name: c for c in CONFIGS}


def corpus_lengths(cfg: Config, n: int, lo: int) -> np.ndarray:
    """Decode lengths T_s of an n-sentence corpus, uniform in [lo, cfg.T]:
    lo + (mix(mix(S + 'L') ^ s) mod (cfg.T - lo + 1)) for sentence s."""
    base = mix((cfg.seed + TAG_L) & M64)
    span = cfg.T - lo + 1
    return np.array([lo + mix(base ^ s) % span for s in range(n)], dtype=np.int32)


def dense_evidence_config() -> Config:
    """The small workload's shape with a 200-best-sized evidence space: 17
    lattice paths of 12 words per sentence, at most 484 n-gram histories per
    sentence (the paper's dense L has at most 500 rows for 200 hypotheses)."""
    return BY_NAME["small"].replace(name="small-dense-L", paths=17, path_len=12)


def get_config(name_or_index) -> Config:
    if isinstance(name_or_index, int):
        return CONFIGS[name_or_index]
    return BY_NAME[name_or_index]


# --------------------------------------------------------------------------
# Output projection
# --------------------------------------------------------------------------
def inv_sqrt_f32(H: int) -> np.float32:
    """fp32(1/sqrt(H)), correctly rounded."""
    return np.float32(1.0 / math.sqrt(H))


def make_weights(cfg: Config) -> np.ndarray:
    """W as bf16 bits, shape [V, H]: bf16(fp32(IH(mix(mix(S+'W') + v*H + i)) * c_H))."""
    base = mix((cfg.seed + TAG_W) & M64)
    c = inv_sqrt_f32(cfg.H)
    out = np.empty((cfg.V, cfg.H), dtype=np.uint16)
    rows = max(1, (1 << 15) // cfg.H)      # ~32K elements per chunk stays in cache
    idx_h = np.arange(cfg.H, dtype=np.uint64)
    with np.errstate(over="ignore"):
        for v0 in range(0, cfg.V, rows):
            v1 = min(cfg.V, v0 + rows)
            v = np.arange(v0, v1, dtype=np.uint64)[:, None]
            h = np.uint64(base) + v * np.uint64(cfg.H) + idx_h[None, :]
            val = irwin_hall_np(mix_np(h)) * c
            out[v0:v1] = bf16_bits(val.astype(np.float32))
    return out


# --------------------------------------------------------------------------
# Stand-in decoder state: hidden vector per (sentence, history)
# --------------------------------------------------------------------------
def initial_hash(cfg: Config, s: int) -> int:
    return mix(mix((cfg.seed + TAG_H) & M64) ^ s)


def next_hash(hh: int, y: int) -> int:
    return mix(hh ^ (y + 1))


def history_hash(cfg: Config, s: int, hist: Sequence[int]) -> int:
    hh = initial_hash(cfg, s)
    for y in hist:
        hh = next_hash(hh, y)
    return hh


def hidden_from_hashes(hh: np.ndarray, H: int) -> np.ndarray:
    """bf16 bits [n, H]: hidden[i] = bf16(IH(mix(hh + i)))."""
    hh = np.asarray(hh, dtype=np.uint64).reshape(-1, 1)
    out = np.empty((hh.shape[0], H), dtype=np.uint16)
    rows = max(1, (1 << 15) // H)
    ih = np.arange(H, dtype=np.uint64)[None, :]
    with np.errstate(over="ignore"):
        for r0 in range(0, hh.shape[0], rows):
            z = mix_np(hh[r0:r0 + rows] + ih)
            out[r0:r0 + rows] = bf16_bits(irwin_hall_np(z))
    return out


def hidden_state(cfg: Config, s: int, hist: Sequence[int]) -> np.ndarray:
    """bf16 bits [H] of the stand-in state after history `hist` of sentence s."""
    return hidden_from_hashes(np.array([history_hash(cfg, s, hist)], dtype=np.uint64), cfg.H)[0]


def eos_bias(cfg: Config, t: int, s: int) -> float:
    """Extra EOS logit at 1-based step t for sentence s (forced-EOS workload)."""
    if cfg.eos_boost_from and t >= cfg.eos_boost_from and (s % 2 == 1):
        return cfg.eos_boost
    return 0.0


def eos_bias_table(cfg: Config, T: int | None = None) -> np.ndarray:
    """fp32 [T, B] of eos_bias(t, s) for t = 1..T."""
    T = cfg.T if T is None else T
    out = np.zeros((T, cfg.B), dtype=np.float32)
    for t in range(1, T + 1):
        for s in range(cfg.B):
            out[t - 1, s] = eos_bias(cfg, t, s)
    return out


# --------------------------------------------------------------------------
# Lattice paths and n-gram posteriors
# --------------------------------------------------------------------------
_ZIPF_CACHE = {}


def zipf_cdf(n_ranks: int, a: float) -> np.ndarray:
    key = (n_ranks, a)
    if key not in _ZIPF_CACHE:
        w = np.arange(1, n_ranks + 1, dtype=np.float64) ** (-a)
        c = np.cumsum(w)
        _ZIPF_CACHE[key] = c / c[-1]
    return _ZIPF_CACHE[key]


def make_lattice(cfg: Config, s: int):
    """Paths int32 [P, L+1] (last column EOS) and fp64 path weights [P]."""
    P, L = cfg.paths, cfg.path_len
    base = mix(mix((cfg.seed + TAG_P) & M64) ^ s)
    idx = np.arange(P * L, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = mix_np(np.uint64(base) + idx)
    u = (z >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)
    cdf = zipf_cdf(cfg.V - 2, cfg.zipf_a)
    rank = np.searchsorted(cdf, u, side="right") + 1      # first r with cdf[r] > u
    rank = np.minimum(rank, cfg.V - 2)
    words = (rank + 1).astype(np.int32).reshape(P, L)
    paths = np.concatenate([words, np.full((P, 1), EOS, dtype=np.int32)], axis=1)
    gbase = mix(mix((cfg.seed + TAG_G) & M64) ^ s)
    with np.errstate(over="ignore"):
        g = irwin_hall_np(np.uint64(gbase) + np.arange(P, dtype=np.uint64)).astype(np.float64)
    e = np.exp(g - g.max())
    w = e / np.sum(e)
    return paths, w


def posteriors_from_paths(paths: np.ndarray, w: np.ndarray, max_order: int = 4):
    """n-gram posteriors over a weighted path list.

    p(u) = sum of w_p over the paths that contain n-gram u at least once, in
    fp64, then rounded to fp32 and clamped to 1.  Returns (order int32 [n],
    tokens int32 [n, 4] (first `order` entries used, oldest word first, the
    rest -1), post float32 [n]), sorted by (order, tokens)."""
    P, Lp = paths.shape
    orders, toks, posts = [], [], []
    for n in range(1, max_order + 1):
        if Lp < n:
            continue
        nw = Lp - n + 1
        win = np.stack([paths[:, i:i + nw] for i in range(n)], axis=2)  # [P, nw, n]
        pid = np.repeat(np.arange(P), nw)
        flat = win.reshape(-1, n).astype(np.int64)
        # sort by (tokens..., path) and drop repeats of an n-gram inside one path
        keys = [pid] + [flat[:, j] for j in range(n - 1, -1, -1)]
        o = np.lexsort(keys)
        f = flat[o]
        p = pid[o]
        same_gram = np.all(f[1:] == f[:-1], axis=1)
        keep = np.ones(len(f), dtype=bool)
        keep[1:] = ~(same_gram & (p[1:] == p[:-1]))
        f, p = f[keep], p[keep]
        new_gram = np.ones(len(f), dtype=bool)
        new_gram[1:] = ~np.all(f[1:] == f[:-1], axis=1)
        gid = np.cumsum(new_gram) - 1
        ng = int(gid[-1]) + 1
        acc = np.zeros(ng, dtype=np.float64)
        np.add.at(acc, gid, w[p])             # accumulates in path order per n-gram
        post = np.minimum(acc.astype(np.float32), np.float32(1.0))
        t4 = np.full((ng, 4), -1, dtype=np.int32)
        t4[:, :n] = f[new_gram].astype(np.int32)
        orders.append(np.full(ng, n, dtype=np.int32))
        toks.append(t4)
        posts.append(post)
    return (np.concatenate(orders), np.concatenate(toks, axis=0),
            np.concatenate(posts).astype(np.float32))


def posteriors(cfg: Config, s: int):
    """(order, tokens, post) for sentence s; see posteriors_from_paths."""
    paths, w = make_lattice(cfg, s)
    return posteriors_from_paths(paths, w)


def ngram_dict(order: np.ndarray, tokens: np.ndarray, post: np.ndarray) -> dict:
    """{(w1, ..., wn): p} view of a posterior list (p widened to fp64)."""
    out = {}
    for n, t, p in zip(order.tolist(), tokens.tolist(), post.tolist()):
        out[tuple(t[:n])] = float(p)
    return out
