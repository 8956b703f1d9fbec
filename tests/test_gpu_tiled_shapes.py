"""GPU parity of every MFMA-tiled GEMM variant, whatever the launch policy
would pick: each of the five tile shapes (128x128, 128x256 with four waves
of 64x128 or eight of 64x64, 256x256 with eight waves of 64x128 or four of
128x128), without a K split and with a two-way split summed inside the
launch, forced for all five GEMM families at once.

The decoder has one layer of model width 2048, so the attention projections
have enough K steps for a split too: 16 q / 4 kv heads of 128, SwiGLU 4096,
vocab 8192. One verify of 4 sequences x 65 rows = 260 rows (ragged against
every tile height) over contexts from a one-token prompt to 500 tokens
covers the QKV epilogue (rotary + paged K/V write), the residual epilogue
with both activation encodings (fp16 hi + lo for O, one fp16 for down), the
SwiGLU epilogue and the LM-head argmax partials. Tolerances as everywhere:
logits max-abs 2e-2; argmax, accepted length and next token exact except
near ties."""

import numpy as np
import pytest

import oracle
from tests._parity import Report, check_step
from workloads import ModelConfig, make_weights, tokens as wt

pytestmark = pytest.mark.gpu

WIDE = ModelConfig("wide1", 1, 2048, 16, 4, 128, 4096, 8192, 5.0e5, max_pos=1024)
FAMILIES = ("qkv", "o", "gateup", "down", "lm")


@pytest.fixture(scope="module")
def wide_case():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = make_weights(WIDE, seed=11, gain_std=0.1)
    om = oracle.OracleModel(WIDE, w)
    k = WIDE.max_draft
    lens = [1, 33, 200, 500]
    drng = wt.rng_for("draft", 90)
    ctxs, states, drafts, results = [], [], [], []
    for s, L in enumerate(lens):
        c = wt.uniform_context(wt.rng_for("context", 90 + s), L, WIDE.vocab)
        st = oracle.prefill(om, c)
        g, _ = oracle.greedy_decode(om, st, 9)
        full = np.concatenate([g, wt.random_chain(drng, k + 1 - len(g), WIDE.vocab)])
        d = wt.plant_chain(drng, full, int(drng.integers(0, 9)), k, WIDE.vocab)
        ctxs.append(c)
        states.append(st)
        drafts.append(d)
        results.append(oracle.verify(om, st, d))
    return torch, w, ctxs, states, drafts, results


@pytest.mark.parametrize("splits", [1, 2])
@pytest.mark.parametrize("tile", [0, 1, 2, 3, 4])
def test_forced_tile_shape_matches_oracle(wide_case, tile, splits):
    import paper_2606_01019_amd as hvd
    torch, w, ctxs, states, drafts, results = wide_case
    gm = hvd.Model(WIDE, w)
    kv = None
    try:
        B, k = len(ctxs), WIDE.max_draft
        kv = hvd.KVCache(gm, max_seqs=B, n_pages=sum((len(c) + k + 16) // 16 + 1 for c in ctxs) + 8)
        for f in FAMILIES:
            kv.set_tiled_shape(f, tile, splits)
        for s, c in enumerate(ctxs):
            kv.prefill(s, c)
        rows = B * (k + 1)
        print(f"tile {tile}, {splits} split(s): {rows} rows", flush=True)
        lg = torch.empty((rows, WIDE.vocab), dtype=torch.float32, device="cuda")
        a, n = kv.verify(list(range(B)), [st.ctx for st in states], drafts, logits=lg)
        lg = lg.cpu().numpy().astype(np.float64)
        rep = Report()
        for s in range(B):
            check_step(rep, results[s], lg[s * (k + 1):(s + 1) * (k + 1)], int(a[s]), int(n[s]), drafts[s])
        print(rep)
    finally:
        if kv is not None:
            kv.close()
        gm.close()
