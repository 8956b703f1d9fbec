"""Seeded token streams: contexts, planted acceptance targets and drafts.

Every generator takes a ``numpy.random.Generator``; ``rng_for`` derives one
from the base seed 42 and a purpose tuple, so each input has its own stream.

Drafts are chains (the cache draft of the paper is a token sequence, §3.1).
A planted draft of length k with target acceptance a is built from a greedy
continuation ``greedy`` (the target's argmax tokens after the current prefix,
supplied by the caller): the first a tokens are copied from it, the token at
index a (if a < k) is any token different from greedy[a], and the tail is
filler.  Whatever produced ``greedy`` decides whether the plant holds; this
module only arranges tokens.
"""

import numpy as np

BASE_SEED = 42

PURPOSE = {"context": 1, "draft": 2, "accept": 3, "batch": 4, "weights": 5, "misc": 9}


def rng_for(*key) -> np.random.Generator:
    """Generator seeded from SeedSequence([42, *key]); string keys map through PURPOSE."""
    ints = [BASE_SEED] + [PURPOSE[k] if isinstance(k, str) else int(k) for k in key]
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(ints)))


# ---------------------------------------------------------------- contexts

def uniform_context(rng, n: int, vocab: int) -> np.ndarray:
    return rng.integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def zipf_context(rng, n: int, vocab: int, s: float = 1.1) -> np.ndarray:
    """Tokens whose rank r in 1..vocab has probability proportional to r^-s;
    token id = r - 1."""
    r = np.arange(1, vocab + 1, dtype=np.float64)
    cdf = np.cumsum(r ** (-s))
    cdf /= cdf[-1]
    u = rng.random(n)
    return np.minimum(np.searchsorted(cdf, u, side="right"), vocab - 1).astype(np.int32)


def segment_context(rng, n: int, vocab: int, seg: int = 64, n_base: int = 16,
                    mutate: float = 0.2) -> np.ndarray:
    """Agentic-style long context: n/seg segments of seg tokens, each a copy of
    one of n_base seeded base segments with a fraction ``mutate`` of its tokens
    replaced by uniform tokens."""
    base = zipf_context(rng, n_base * seg, vocab).reshape(n_base, seg)
    n_seg = -(-n // seg)
    pick = rng.integers(0, n_base, size=n_seg)
    out = base[pick].copy()
    mask = rng.random(out.shape) < mutate
    out[mask] = rng.integers(0, vocab, size=int(mask.sum()))
    return out.reshape(-1)[:n].astype(np.int32)


# ------------------------------------------------------- acceptance targets

def geometric_accept(rng, p: float, k: int) -> int:
    """min(G, k) with G ~ Geometric on {0, 1, ...}: each token rejected with prob p."""
    return int(min(rng.geometric(p) - 1, k))


def bimodal_accept(rng, k: int) -> int:
    """Half the time U{0..2}, otherwise U{ceil(k/2)..k}."""
    if rng.random() < 0.5:
        return int(rng.integers(0, min(2, k) + 1))
    return int(rng.integers(-(-k // 2), k + 1))


def uniform_accept(rng, k: int) -> int:
    return int(rng.integers(0, k + 1))


# ------------------------------------------------------------------ drafts

def _other_token(rng, avoid: int, vocab: int) -> int:
    t = int(rng.integers(0, vocab - 1))
    return t + 1 if t >= avoid else t


def plant_chain(rng, greedy, a: int, k: int, vocab: int) -> np.ndarray:
    """Chain draft of length k: greedy[:a], then a token != greedy[a], then
    uniform filler.  Needs len(greedy) >= min(a + 1, k)."""
    assert 0 <= a <= k
    greedy = np.asarray(greedy, dtype=np.int64)
    d = np.empty(k, dtype=np.int32)
    d[:a] = greedy[:a]
    if a < k:
        d[a] = _other_token(rng, int(greedy[a]), vocab)
        if k > a + 1:
            d[a + 1:] = rng.integers(0, vocab, size=k - a - 1)
    return d


def plant_cache_draft(rng, context, greedy, a: int, k: int, vocab: int) -> np.ndarray:
    """Cache-style draft: greedy[:a], a mismatching token x, then the tokens that
    followed an earlier occurrence of x in ``context`` (a 1-token suffix match),
    or uniform filler if x never occurs."""
    d = plant_chain(rng, greedy, a, k, vocab)
    if a + 1 < k:
        x = int(d[a])
        ctx = np.asarray(context)
        hits = np.flatnonzero(ctx[:-1] == x)
        if hits.size:
            j = int(hits[rng.integers(0, hits.size)]) + 1
            span = ctx[j:j + (k - a - 1)]
            d[a + 1:a + 1 + span.size] = span
    return d


def random_chain(rng, k: int, vocab: int) -> np.ndarray:
    return rng.integers(0, vocab, size=k, dtype=np.int64).astype(np.int32)


def corrupt_stream(rng, greedy, p: float, vocab: int) -> np.ndarray:
    """Token stream for a copy drafter with planted acceptance: ``greedy``
    with each token independently replaced, with probability p, by a uniform
    token different from it.  Drafts copied from the stream at the current
    position are then accepted up to the next replaced token, so the accepted
    length of a k-token draft is min(Geometric(p), k)."""
    g = np.asarray(greedy, dtype=np.int64)
    out = g.copy()
    hit = rng.random(g.shape[0]) < p
    shift = rng.integers(1, vocab, size=g.shape[0])
    out[hit] = (g[hit] + shift[hit]) % vocab
    return out.astype(np.int32)
