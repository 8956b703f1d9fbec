"""GPU parity on a mid-size grouped-query decoder that exercises the code
paths the tiny decoder does not: 8 q / 2 kv heads of 128 (group 4), rotary
theta 5e5, weight-streaming GEMMs with 2 and 4 strips per workgroup, the
pipelined K loop with its tail, the K split with its finish pass (down
projection, K = 8192), split-KV attention with the combine pass, prefill
in 512-row chunks with a ragged tail, 1 to 5 row tiles per verify
(k = 0 .. 64), and the largest batch a 32-sequence handle takes."""

import numpy as np
import pytest

import oracle
from tests._parity import Report, check_step, oracle_commit_as
from workloads import ModelConfig, make_weights, tokens as wt

pytestmark = pytest.mark.gpu

MID = ModelConfig("mid", 2, 1024, 8, 2, 128, 8192, 16384, 5.0e5, max_pos=4096)


@pytest.fixture(scope="module")
def mid():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    w = make_weights(MID, seed=5, gain_std=0.1)
    return torch, oracle.OracleModel(MID, w), hvd.Model(MID, w)


def _verify(torch, kv, ids, ctxs, drafts):
    rows = sum(len(d) + 1 for d in drafts)
    lg = torch.empty((rows, kv.model.cfg.vocab), dtype=torch.float32, device="cuda")
    a, n = kv.verify(ids, ctxs, drafts, logits=lg)
    return a, n, lg.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("k", [0, 3, 15, 16, 33, 64])
def test_mid_verify_matches_oracle(mid, k):
    import paper_2606_01019_amd as hvd
    torch, om, gm = mid
    kv = hvd.KVCache(gm, max_seqs=1, n_pages=128)
    ctx = wt.uniform_context(wt.rng_for("context", 40 + k), 600, MID.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(0, ctx)
    drng = wt.rng_for("draft", 40 + k)
    g, _ = oracle.greedy_decode(om, st, min(k, 12) + 1)
    a_plan = min(len(g) - 1, wt.uniform_accept(drng, k))
    full = np.concatenate([g, wt.random_chain(drng, max(0, k + 1 - len(g)), MID.vocab)])
    d = wt.plant_chain(drng, full, a_plan, k, MID.vocab)
    res = oracle.verify(om, st, d)
    a, n, lg = _verify(torch, kv, [0], [st.ctx], [d])
    rep = Report()
    check_step(rep, res, lg, int(a[0]), int(n[0]), d)
    print(f"k={k}: accepted {int(a[0])} (oracle {res.accepted}) {rep}")


def test_mid_batched_decode_loop(mid):
    """Three sequences, five verify+commit cycles with mixed draft lengths."""
    import paper_2606_01019_amd as hvd
    torch, om, gm = mid
    kv = hvd.KVCache(gm, max_seqs=3, n_pages=256)
    lens = [130, 257, 700]
    states = []
    for s, L in enumerate(lens):
        c = wt.uniform_context(wt.rng_for("context", 60 + s), L, MID.vocab)
        states.append(oracle.prefill(om, c))
        kv.prefill(s, c)
    drng = wt.rng_for("draft", 60)
    rep = Report()
    for step in range(5):
        drafts, results = [], []
        for s in range(3):
            k = int(drng.integers(0, 20))
            g, _ = oracle.greedy_decode(om, states[s], k + 1)
            d = wt.plant_chain(drng, g, wt.geometric_accept(drng, 0.3, k), k, MID.vocab)
            drafts.append(d)
            results.append(oracle.verify(om, states[s], d))
        a, n, lg = _verify(torch, kv, [0, 1, 2], [st.ctx for st in states], drafts)
        kv.commit([0, 1, 2])
        row = 0
        for s in range(3):
            k = len(drafts[s])
            div = check_step(rep, results[s], lg[row:row + k + 1], int(a[s]), int(n[s]), drafts[s])
            row += k + 1
            states[s] = (oracle_commit_as(states[s], results[s], int(a[s]), int(n[s])) if div
                         else oracle.commit(states[s], results[s]))
            assert kv.seq_info(s)[:2] == (states[s].ctx, states[s].pending)
    print(rep)


def test_mid_maximum_rows_ragged_contexts(mid):
    """The largest verify a handle of 32 sequences takes: every sequence
    drafts max_draft = 64 tokens (2080 rows: MFMA-tiled GEMMs, two attention
    row groups per kv head), over ragged contexts from the degenerate empty
    cache (a one-token prompt) to 700 tokens."""
    import paper_2606_01019_amd as hvd
    torch, om, gm = mid
    B, k = 32, MID.max_draft
    lens = [1, 2, 17, 31] + [int(x) for x in wt.rng_for("misc", 70).integers(40, 700, size=B - 4)]
    kv = hvd.KVCache(gm, max_seqs=B, n_pages=sum((L + k + 16) // 16 + 1 for L in lens) + 8)
    states, drafts, results = [], [], []
    drng = wt.rng_for("draft", 70)
    for s, L in enumerate(lens):
        c = wt.uniform_context(wt.rng_for("context", 70 + s), L, MID.vocab)
        st = oracle.prefill(om, c)
        kv.prefill(s, c)
        g, _ = oracle.greedy_decode(om, st, 9)
        full = np.concatenate([g, wt.random_chain(drng, k + 1 - len(g), MID.vocab)])
        d = wt.plant_chain(drng, full, int(drng.integers(0, 9)), k, MID.vocab)
        states.append(st)
        drafts.append(d)
        results.append(oracle.verify(om, st, d))
    print(f"{B} sequences, {B * (k + 1)} rows, contexts {min(lens) - 1}..{max(lens) - 1}", flush=True)
    a, n, lg = _verify(torch, kv, list(range(B)), [st.ctx for st in states], drafts)
    rep = Report()
    for s in range(B):
        check_step(rep, results[s], lg[s * (k + 1):(s + 1) * (k + 1)], int(a[s]), int(n[s]), drafts[s])
    kv.commit(list(range(B)))
    for s in range(B):
        assert kv.seq_info(s)[0] == states[s].ctx + int(a[s]) + 1
    print(rep)
