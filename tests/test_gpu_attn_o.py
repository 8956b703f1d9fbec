"""Attention, split-KV merge and O projection as one launch per layer
(HVD_OPT_ATTN_O): verify steps of 1 and 2 row tiles on two grouped-query
decoders with head dim 128 -- O GEMMs of K = 1024 (64 strips) and K = 4096
(128 strips) -- at short and long contexts (one and several K/V sub-chunks
per attention item), a batch decode loop with commits and a token tree,
each checked against the oracle (logits max-abs 2e-2; argmax, accepted
length and next token exact except near ties) and against the separate
launches (logits within 2e-2)."""

import numpy as np
import pytest

import oracle
from tests._parity import LOGIT_TOL, Report, check_step, oracle_commit_as
from tests.test_gpu_tree import check_tree
from workloads import ModelConfig, make_weights, tokens as wt, trees

pytestmark = pytest.mark.gpu

MID = ModelConfig("mid", 2, 1024, 8, 2, 128, 8192, 16384, 5.0e5, max_pos=4096)
QWIDE = ModelConfig("qwide", 2, 2048, 32, 8, 128, 4096, 8192, 5.0e5, max_pos=4096)


def _load(cfg, seed):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    w = make_weights(cfg, seed=seed, gain_std=0.1)
    return torch, oracle.OracleModel(cfg, w), hvd.Model(cfg, w)


@pytest.fixture(scope="module")
def mid():
    return _load(MID, 7)


@pytest.fixture(scope="module")
def qwide():
    return _load(QWIDE, 11)


def _verify(torch, kv, ids, ctxs, drafts, fused):
    kv.set_attn_o(fused)
    rows = sum(len(d) + 1 for d in drafts)
    lg = torch.empty((rows, kv.model.cfg.vocab), dtype=torch.float32, device="cuda")
    a, n = kv.verify(ids, ctxs, drafts, logits=lg)
    return a, n, lg.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("which,ctx_len", [("mid", 900), ("mid", 4000), ("qwide", 700), ("qwide", 3000)])
def test_single_sequence_matches_oracle(mid, qwide, which, ctx_len):
    import paper_2606_01019_amd as hvd
    torch, om, gm = mid if which == "mid" else qwide
    cfg = om.cfg
    kv = hvd.KVCache(gm, max_seqs=1, n_pages=(ctx_len + 64) // 16 + 8)
    ctx = wt.uniform_context(wt.rng_for("context", 180, ctx_len), ctx_len, cfg.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(0, ctx)
    g, _ = oracle.greedy_decode(om, st, 9)
    for k in (0, 5, 8, 16, 31):  # 1 and 2 row tiles
        full = np.concatenate([g, wt.random_chain(wt.rng_for("draft", 180, k), max(0, k + 1 - len(g)), cfg.vocab)])
        d = wt.plant_chain(wt.rng_for("draft", 181, k), full, min(k, 8) // 2, k, cfg.vocab)
        res = oracle.verify(om, st, d)
        out = {}
        for fused in (False, True):
            print(f"{which} ctx={ctx_len} k={k} fused={fused}", flush=True)
            a, n, lg = _verify(torch, kv, [0], [st.ctx], [d], fused)
            kv.truncate(0, st.ctx, st.pending)
            rep = Report()
            check_step(rep, res, lg, int(a[0]), int(n[0]), d)
            out[fused] = lg
            print(f"  accepted {int(a[0])} (oracle {res.accepted}) {rep}", flush=True)
        assert np.abs(out[True] - out[False]).max() <= LOGIT_TOL
    kv.close()


def test_batch_decode_loop_matches_oracle(mid):
    import paper_2606_01019_amd as hvd
    torch, om, gm = mid
    kv = hvd.KVCache(gm, max_seqs=3, n_pages=3 * 80)
    sts = []
    for b in range(3):
        ctx = wt.uniform_context(wt.rng_for("context", 182, b), 300 + 211 * b, MID.vocab)
        sts.append(oracle.prefill(om, ctx))
        kv.prefill(b, ctx)
    rep = Report()
    for step in range(3):
        drafts, ress = [], []
        for b, st in enumerate(sts):
            k = (3, 0, 9)[(b + step) % 3]
            g, _ = oracle.greedy_decode(om, st, min(k, 4) + 1)
            full = np.concatenate([g, wt.random_chain(wt.rng_for("draft", 182, b, step), max(0, k + 1 - len(g)),
                                                      MID.vocab)])
            drafts.append(wt.plant_chain(wt.rng_for("draft", 183, b, step), full, min(k, 3), k, MID.vocab))
            ress.append(oracle.verify(om, st, drafts[-1]))
        print(f"step {step}: k = {[len(d) for d in drafts]}", flush=True)
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
    kv.close()


def test_token_tree_matches_oracle(qwide):
    import paper_2606_01019_amd as hvd
    torch, om, gm = qwide
    kv = hvd.KVCache(gm, max_seqs=1, n_pages=120)
    ctx = wt.uniform_context(wt.rng_for("context", 184), 1100, QWIDE.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(0, ctx)
    greedy, _ = oracle.greedy_decode(om, st, 9)
    rng = wt.rng_for("draft", 184)
    rep = Report()
    for n_nodes in (15, 31):  # 16 and 32 rows
        par = trees.eagle_tree(rng, n_nodes, 8, 4)
        tok = trees.plant_path(rng, par, greedy, 4, QWIDE.vocab)
        res = oracle.verify_tree(om, st, tok, par)
        out = {}
        for fused in (False, True):
            print(f"tree of {n_nodes} nodes, fused={fused}", flush=True)
            kv.set_attn_o(fused)
            lg = torch.empty((n_nodes + 1, QWIDE.vocab), dtype=torch.float32, device="cuda")
            a, n, paths = kv.verify_tree([0], [st.ctx], [(tok, par)], logits=lg)
            L = lg.cpu().numpy().astype(np.float64)
            check_tree(rep, res, L, int(a[0]), int(n[0]), paths[0])
            kv.truncate(0, st.ctx, st.pending)
            out[fused] = L
        assert np.abs(out[True] - out[False]).max() <= LOGIT_TOL
    print(rep, flush=True)
    kv.close()
