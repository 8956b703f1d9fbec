"""Pins of the streamed float32 oracle (oracle/streamed.py) that writes the
full-depth 32B-shaped reference: its bf16 matrix product against exact
float64 products within the float32 rounding bound, and its verify step
against the float64 oracle (itself pinned by brute force and the library
cross-checks in test_oracle_pins.py)."""

import os
import sys

import numpy as np

import oracle
from oracle.model import OracleModel, bf16_bits_to_float
from oracle.streamed import StreamedOracleModel, gemv_bf16
from workloads import TINY, make_weights, tokens as wt
from workloads.weights import f32_to_bf16_bits, make_tensor


def _bf16(rng, shape, std=0.02):
    return f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * np.float32(std))


def test_gemv_bf16_within_float32_bound():
    rng = np.random.default_rng(5)
    for M, N, K in [(1, 7, 5), (3, 130, 4096), (65, 64, 27648), (2, 33, 17)]:
        w = _bf16(rng, (N, K))
        h = rng.standard_normal((M, K)).astype(np.float32)
        y = gemv_bf16(h, w).astype(np.float64)
        W = bf16_bits_to_float(w)
        exact = h.astype(np.float64) @ W.T
        # float32 sum of K products, each product rounded once: |err| <= ~(K/16 + 17) u sum|x w|
        bound = (K / 16 + 18) * 2.0 ** -24 * (np.abs(h.astype(np.float64)) @ np.abs(W).T)
        assert np.all(np.abs(y - exact) <= bound), (M, N, K)


def test_gemv_bf16_rows_independent():
    """Each output row depends only on its own input row (no cross-row mixing)."""
    rng = np.random.default_rng(6)
    w = _bf16(rng, (96, 256))
    h = rng.standard_normal((5, 256)).astype(np.float32)
    full = gemv_bf16(h, w)
    for r in range(5):
        assert np.array_equal(gemv_bf16(h[r:r + 1], w)[0], full[r])


def test_streamed_oracle_matches_float64_oracle_tiny():
    w = make_weights(TINY, seed=42, gain_std=0.1)
    ctx = wt.uniform_context(wt.rng_for("context", 1), 96, TINY.vocab)
    d = wt.random_chain(wt.rng_for("draft", 7), 6, TINY.vocab)
    ref = oracle.verify(OracleModel(TINY, w), oracle.prefill(OracleModel(TINY, w), ctx), d)
    for gemv_rows in (0, 256):  # numpy product for the prefill only / for everything
        m = StreamedOracleModel(TINY, w, gemv_rows=gemv_rows)
        res = oracle.verify(m, oracle.prefill(m, ctx), d)
        assert np.abs(res.logits.astype(np.float64) - ref.logits).max() < 1e-4
        assert res.accepted == ref.accepted and res.next_token == ref.next_token


def test_spill_store_round_trip(tmp_path):
    sys.path.insert(0, os.path.join(os.path.dirname(__file__), "golden"))
    from make_golden import SpillStore
    st = SpillStore(TINY, resident=1, spill_dir=str(tmp_path))
    for name in ("layers.0.wq", "layers.1.wd", "lm_head", "layers.1.mlp_norm"):
        assert np.array_equal(st[name], make_tensor(TINY, name, seed=42)), name
    assert os.path.exists(tmp_path / "tiny.layers.1.wd.bf16")
    assert not os.path.exists(tmp_path / "tiny.layers.0.wd.bf16")
    again = SpillStore(TINY, resident=0, spill_dir=None)
    assert np.array_equal(again["layers.1.wu"], make_tensor(TINY, "layers.1.wu", seed=42))
