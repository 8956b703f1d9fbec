"""GPU parity of the weight-streaming GEMM under every strip count, whatever
the launch policy would pick: 1, 2, 4 or 8 16-column strips per workgroup,
without a K split and with a three-way split plus its finish pass, forced
for all five GEMM families at once (the library reads the override when a
model is loaded; shapes a kernel does not support fall back to the policy:
one strip for the SwiGLU GEMM, eight strips above two row tiles).

Verifies of k = 3, 20, 50 and 64 draft tokens give 1, 2, 4 and 5 row tiles
(the last as two row blocks) on the mid-size grouped-query decoder, over a
600-token context (whose prefill also runs under the forced shapes).
Tolerances as everywhere: logits max-abs 2e-2; argmax, accepted length and
next token exact except near ties."""

import numpy as np
import pytest

import oracle
from tests._parity import Report, check_step
from workloads import ModelConfig, make_weights, tokens as wt

pytestmark = pytest.mark.gpu

MID = ModelConfig("mid", 2, 1024, 8, 2, 128, 8192, 16384, 5.0e5, max_pos=4096)
FAMILIES = ("qkv", "o", "gateup", "down", "lm")
DRAFT_LENS = (3, 20, 50, 64)


@pytest.fixture(scope="module")
def mid_cases():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = make_weights(MID, seed=5, gain_std=0.1)
    om = oracle.OracleModel(MID, w)
    cases = []
    for k in DRAFT_LENS:
        ctx = wt.uniform_context(wt.rng_for("context", 140 + k), 600, MID.vocab)
        st = oracle.prefill(om, ctx)
        drng = wt.rng_for("draft", 140 + k)
        g, _ = oracle.greedy_decode(om, st, min(k, 9) + 1)
        full = np.concatenate([g, wt.random_chain(drng, k + 1 - len(g), MID.vocab)])
        d = wt.plant_chain(drng, full, min(len(g) - 1, wt.uniform_accept(drng, k)), k, MID.vocab)
        cases.append((ctx, st, d, oracle.verify(om, st, d)))
    return torch, w, cases


@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("strips", [1, 2, 4, 8])
def test_forced_strip_count_matches_oracle(mid_cases, strips, splits):
    import paper_2606_01019_amd as hvd
    torch, w, cases = mid_cases
    gm = hvd.Model(MID, w)
    kv = None
    try:
        kv = hvd.KVCache(gm, max_seqs=1, n_pages=128)
        for f in FAMILIES:
            kv.set_gemm_shape(f, strips, splits)
        rep = Report()
        for ctx, st, d, res in cases:
            print(f"{strips} strips, {splits} split(s), k = {len(d)}", flush=True)
            kv.prefill(0, ctx)
            lg = torch.empty((len(d) + 1, MID.vocab), dtype=torch.float32, device="cuda")
            a, n = kv.verify([0], [st.ctx], [d], logits=lg)
            check_step(rep, res, lg.cpu().numpy().astype(np.float64), int(a[0]), int(n[0]), d)
            kv.seq_free(0)
        print(rep)
    finally:
        if kv is not None:
            kv.close()
        gm.close()
