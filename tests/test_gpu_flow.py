"""The one-launch verify step (HVD_OPT_FLOW): on a grouped-query decoder with
head dim 128 (8 q / 2 kv heads), verify steps of 1 and 2 row tiles and a
batch of three sequences, run once with the per-kernel launches and once as
one launch, each checked against the oracle (logits max-abs 2e-2; argmax,
accepted length and next token exact except near ties); and the timeline
diagnostics of the one-launch step are consistent."""

import numpy as np
import pytest

import oracle
from tests._parity import LOGIT_TOL, Report, check_step
from workloads import ModelConfig, make_weights, tokens as wt

pytestmark = pytest.mark.gpu

MID = ModelConfig("mid", 2, 1024, 8, 2, 128, 8192, 16384, 5.0e5, max_pos=4096)


@pytest.fixture(scope="module")
def mid():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    w = make_weights(MID, seed=7, gain_std=0.1)
    return torch, oracle.OracleModel(MID, w), hvd.Model(MID, w)


def _verify(torch, kv, ids, ctxs, drafts, flow):
    kv.set_flow(flow)
    rows = sum(len(d) + 1 for d in drafts)
    lg = torch.empty((rows, kv.model.cfg.vocab), dtype=torch.float32, device="cuda")
    a, n = kv.verify(ids, ctxs, drafts, logits=lg)
    return a, n, lg.cpu().numpy().astype(np.float64)


def test_flow_single_sequence_matches_oracle(mid):
    import paper_2606_01019_amd as hvd
    torch, om, gm = mid
    kv = hvd.KVCache(gm, max_seqs=1, n_pages=160)
    ctx = wt.uniform_context(wt.rng_for("context", 80), 900, MID.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(0, ctx)
    g, _ = oracle.greedy_decode(om, st, 9)
    for k in (0, 5, 8, 16, 31):  # 1 and 2 row tiles; 4..128 query rows per kv head
        full = np.concatenate([g, wt.random_chain(wt.rng_for("draft", 80, k), max(0, k + 1 - len(g)), MID.vocab)])
        d = wt.plant_chain(wt.rng_for("draft", 81, k), full, min(k, 8) // 2, k, MID.vocab)
        res = oracle.verify(om, st, d)
        out = {}
        for flow in (False, True):
            a, n, lg = _verify(torch, kv, [0], [st.ctx], [d], flow)
            kv.truncate(0, st.ctx, st.pending)
            rep = Report()
            check_step(rep, res, lg, int(a[0]), int(n[0]), d)
            out[flow] = lg
            print(f"k={k} flow={flow}: accepted {int(a[0])} (oracle {res.accepted}) {rep}", flush=True)
        assert np.abs(out[True] - out[False]).max() <= LOGIT_TOL


def test_flow_batch_decode_loop_matches_oracle(mid):
    import paper_2606_01019_amd as hvd
    from tests._parity import oracle_commit_as
    torch, om, gm = mid
    kv = hvd.KVCache(gm, max_seqs=3, n_pages=3 * 80)
    sts = []
    for b in range(3):
        ctx = wt.uniform_context(wt.rng_for("context", 82, b), 300 + 211 * b, MID.vocab)
        sts.append(oracle.prefill(om, ctx))
        kv.prefill(b, ctx)
    kv.set_flow(True)
    rep = Report()
    for step in range(3):
        drafts, ress = [], []
        for b, st in enumerate(sts):
            k = (3, 0, 9)[(b + step) % 3]
            g, _ = oracle.greedy_decode(om, st, min(k, 4) + 1)
            full = np.concatenate([g, wt.random_chain(wt.rng_for("draft", 82, b, step), max(0, k + 1 - len(g)),
                                                      MID.vocab)])
            drafts.append(wt.plant_chain(wt.rng_for("draft", 83, b, step), full, min(k, 3), k, MID.vocab))
            ress.append(oracle.verify(om, st, drafts[-1]))
        a, n, lg = _verify(torch, kv, [0, 1, 2], [st.ctx for st in sts], drafts, True)
        r0 = 0
        for b in range(3):
            rows = len(drafts[b]) + 1
            check_step(rep, ress[b], lg[r0:r0 + rows], int(a[b]), int(n[b]), drafts[b])
            sts[b] = oracle_commit_as(sts[b], ress[b], int(a[b]), int(n[b]))
            r0 += rows
        kv.commit([0, 1, 2])
        for b in range(3):
            assert kv.seq_info(b)[0] == sts[b].ctx
    print(rep, flush=True)


def test_flow_trace_is_a_consistent_timeline(mid):
    import paper_2606_01019_amd as hvd
    torch, om, gm = mid
    kv = hvd.KVCache(gm, max_seqs=1, n_pages=80)
    ctx = wt.uniform_context(wt.rng_for("context", 84), 500, MID.vocab)
    kv.prefill(0, ctx)
    c0, p0, _ = kv.seq_info(0)
    buf = torch.zeros(4 * 8192, dtype=torch.int64, device="cuda")
    kv.set_flow(True)
    kv.flow_trace(buf)
    kv.verify([0], [c0], [np.arange(1, 6, dtype=np.int32)])
    kv.flow_trace(None)
    tr = buf.cpu().numpy().reshape(-1, 4)
    used = tr[:, 0] > 0
    assert used.sum() > 100 and not used[used.sum():].any()  # a prefix of the buffer, one entry per workgroup
    t = tr[used]
    assert np.all(t[:, 1] >= t[:, 0]) and np.all(t[:, 2] >= t[:, 1])
    assert len(np.unique(t[:, 3] >> 32)) > 1  # ran on several XCDs
