"""The full-size references (tests/golden/*.json) come from the oracle run in
float32.  Pin that choice: at the 8B width, with two decoder layers, the
float32 and float64 oracle agree far inside the GPU parity tolerance."""

import numpy as np

import oracle
from oracle.model import OracleModel
from workloads import SHAPE_8B, make_weights, tokens as wt


def test_float32_oracle_matches_float64_at_8b_width():
    cfg = SHAPE_8B.with_layers(2)
    w = make_weights(cfg, seed=42)
    ctx = wt.zipf_context(wt.rng_for("context", 3), 48, cfg.vocab)
    d = wt.random_chain(wt.rng_for("draft", 3), 4, cfg.vocab)
    res = {}
    for dt in (np.float32, np.float64):
        m = OracleModel(cfg, w, dtype=dt, cache=False)
        st = oracle.prefill(m, ctx)
        res[dt] = oracle.verify(m, st, d).logits.astype(np.float64)
    err = np.abs(res[np.float32] - res[np.float64]).max()
    assert err < 1e-3, err
