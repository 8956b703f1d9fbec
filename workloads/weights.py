"""Random-init weights: every matrix iid N(0, 0.02^2), rounded to bf16.

Each tensor is drawn in fixed-size chunks, chunk c of tensor (layer, id) from
``numpy.random.SeedSequence([seed, layer + 1, id, c])``, so the values do not
depend on the number of threads used to draw them.  fp32 samples are rounded
to bf16 with round-to-nearest-even and returned as their uint16 bit patterns.

Norm gains are 1.0 unless ``gain_std`` > 0, in which case they are
1 + gain_std * N(0, 1) (used by tests that must see the gains applied).

Tensor layout follows the torch ``Linear`` convention, [out_features,
in_features], row-major.  Canonical order (the order ``hvd_model_load`` takes):
embed [V, D]; then per layer attn_norm [D], wq [Hq*dh, D], wk [Hkv*dh, D],
wv [Hkv*dh, D], wo [D, Hq*dh], mlp_norm [D], wg [F, D], wu [F, D], wd [D, F];
then final_norm [D], lm_head [V, D].
"""

from concurrent.futures import ThreadPoolExecutor
import os

import numpy as np

from .configs import ModelConfig

CHUNK = 1 << 22
WEIGHT_STD = 0.02

_LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu", "wd")
_TENSOR_ID = {"embed": 0, "final_norm": 1, "lm_head": 2}
_TENSOR_ID.update({n: 10 + i for i, n in enumerate(_LAYER_TENSORS)})


def canonical_tensors(cfg: ModelConfig):
    """List of (name, shape, layer, kind) in canonical order."""
    D, F, V = cfg.d_model, cfg.ffn_dim, cfg.vocab
    qd, kd = cfg.q_dim, cfg.kv_dim
    shapes = {
        "attn_norm": (D,), "wq": (qd, D), "wk": (kd, D), "wv": (kd, D), "wo": (D, qd),
        "mlp_norm": (D,), "wg": (F, D), "wu": (F, D), "wd": (D, F),
    }
    out = [("embed", (V, D), -1, "embed")]
    for l in range(cfg.n_layers):
        for n in _LAYER_TENSORS:
            kind = "norm" if n.endswith("norm") else n
            out.append((f"layers.{l}.{n}", shapes[n], l, kind))
    out.append(("final_norm", (D,), -1, "norm"))
    out.append(("lm_head", (V, D), -1, "lm_head"))
    return out


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); return uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def _short_name(name: str) -> str:
    return name.rsplit(".", 1)[-1]


def _chunk(seed, layer, tid, c, n, std, offset):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, layer + 1, tid, c])))
    x = rng.standard_normal(n, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    if offset:
        x += np.float32(offset)
    return f32_to_bf16_bits(x)


def make_tensor(cfg: ModelConfig, name: str, seed: int = 42, gain_std: float = 0.0,
                pool: ThreadPoolExecutor = None) -> np.ndarray:
    """Draw one canonical tensor; returns uint16 bf16 bits with the canonical shape."""
    shape = dict((n, s) for n, s, _, _ in canonical_tensors(cfg))[name]
    layer = int(name.split(".")[1]) if name.startswith("layers.") else -1
    short = _short_name(name)
    tid = _TENSOR_ID[short]
    n = int(np.prod(shape))
    if short.endswith("norm"):
        if gain_std <= 0.0:
            return np.full(shape, 0x3F80, dtype=np.uint16)  # bf16(1.0)
        return _chunk(seed, layer, tid, 0, n, gain_std, 1.0).reshape(shape)
    out = np.empty(n, dtype=np.uint16)
    starts = list(range(0, n, CHUNK))

    def work(ci):
        s = starts[ci]
        m = min(CHUNK, n - s)
        out[s:s + m] = _chunk(seed, layer, tid, ci, m, WEIGHT_STD, 0.0)

    if pool is None or len(starts) == 1:
        for ci in range(len(starts)):
            work(ci)
    else:
        list(pool.map(work, range(len(starts))))
    return out.reshape(shape)


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def make_weights(cfg: ModelConfig, seed: int = 42, gain_std: float = 0.0, threads: int = None,
                 names=None, progress=None) -> dict:
    """Draw the canonical tensors (all, or ``names``); dict name -> uint16 array."""
    threads = threads or default_threads()
    out = {}
    with ThreadPoolExecutor(max_workers=threads) as pool:
        for n, _, _, _ in canonical_tensors(cfg):
            if names is not None and n not in names:
                continue
            out[n] = make_tensor(cfg, n, seed=seed, gain_std=gain_std, pool=pool)
            if progress is not None:
                progress(n)
    return out


class LazyWeights:
    """Mapping name -> tensor that draws each tensor on first use and caches it
    only if ``cache`` is True (large shapes are re-drawn instead of kept)."""

    def __init__(self, cfg: ModelConfig, seed: int = 42, gain_std: float = 0.0, cache: bool = False,
                 threads: int = None):
        self.cfg, self.seed, self.gain_std, self.cache = cfg, seed, gain_std, cache
        self._store = {}
        self._pool = ThreadPoolExecutor(max_workers=threads or default_threads())

    def __getitem__(self, name):
        if name in self._store:
            return self._store[name]
        t = make_tensor(self.cfg, name, seed=self.seed, gain_std=self.gain_std, pool=self._pool)
        if self.cache:
            self._store[name] = t
        return t

    def keys(self):
        return [n for n, _, _, _ in canonical_tensors(self.cfg)]
