"""GPU parity of hvd_verify_tree against the oracle's tree verification on
the tiny decoder (2 layers, d_model 256, 4/4 heads of 64, vocab 4096): trees
shaped like the model drafter's (App. A: depth 8, top-k 4, 32 nodes) with a
planted acceptance along a deepest path, the degenerate shapes (no node, a
chain, a star, 63 nodes), a batch of trees, and commits followed by further
verifies (which read the K/V the tree verify moved into place).  Tolerances
as everywhere: logits max-abs 2e-2; argmax, path and next token exact except
at near ties (top-2 margin < 2e-2) on the accepted path."""

import numpy as np
import pytest

import oracle
from tests._parity import LOGIT_TOL, TIE_MARGIN, Report, check_step, top2_margin
from workloads import TINY, make_weights, tokens as wt, trees

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    w = make_weights(TINY, seed=42, gain_std=0.1)
    return oracle.OracleModel(TINY, w), hvd.Model(TINY, w)


def _kv(gm, max_seqs=4, n_pages=256):
    import paper_2606_01019_amd as hvd
    return hvd.KVCache(gm, max_seqs, n_pages)


def _verify_tree(kv, ids, ctxs, tree_list):
    import torch
    rows = sum(len(t) + 1 for t, _ in tree_list)
    lg = torch.empty((rows, kv.model.cfg.vocab), dtype=torch.float32, device="cuda")
    a, n, paths = kv.verify_tree(ids, ctxs, tree_list, logits=lg)
    return a, n, paths, lg.cpu().numpy().astype(np.float64)


def check_tree(rep: Report, res, L, a_gpu, next_gpu, path_gpu):
    """One sequence's tree verify (logit rows L) against the oracle result.
    Returns True when a near tie on the accepted path sent the GPU elsewhere."""
    err = float(np.abs(L - res.logits).max())
    rep.max_err = max(rep.max_err, err)
    assert err <= LOGIT_TOL, f"logit error {err:.3e}"
    tie = top2_margin(res.logits) < TIE_MARGIN
    g_gpu = L.argmax(axis=1)
    rep.rows += L.shape[0]
    rep.excused += int(tie.sum())
    bad = (g_gpu != res.argmax) & ~tie
    assert not bad.any(), f"argmax differs at non-tie rows {np.flatnonzero(bad)}"
    # the GPU's path follows its own argmax
    assert path_gpu == oracle.tree_accept(g_gpu, res.tokens, res.parents)
    assert a_gpu == len(path_gpu) and next_gpu == int(g_gpu[(path_gpu[-1] + 1) if path_gpu else 0])
    on_path = [0] + [j + 1 for j in res.path]
    if not tie[on_path].any():
        assert path_gpu == res.path and next_gpu == res.next_token
        return False
    return path_gpu != res.path or next_gpu != res.next_token


def test_eagle_trees_planted_acceptance(tiny):
    om, gm = tiny
    kv = _kv(gm)
    ctx = wt.uniform_context(wt.rng_for("context", 61), 300, TINY.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(0, ctx)
    greedy, _ = oracle.greedy_decode(om, st, 9)
    rng = wt.rng_for("draft", 61)
    rep = Report()
    for accept in (0, 1, 3, 5, 8):
        par = trees.eagle_tree(rng, 32, 8, 4)
        tok = trees.plant_path(rng, par, greedy, accept, TINY.vocab)
        res = oracle.verify_tree(om, st, tok, par)
        a, n, paths, L = _verify_tree(kv, [0], [st.ctx], [(tok, par)])
        check_tree(rep, res, L, int(a[0]), int(n[0]), paths[0])
        kv.truncate(0, st.ctx, st.pending)
    print(rep)


def test_degenerate_trees(tiny):
    om, gm = tiny
    kv = _kv(gm)
    ctx = wt.uniform_context(wt.rng_for("context", 62), 150, TINY.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(0, ctx)
    greedy, _ = oracle.greedy_decode(om, st, 64)
    rng = wt.rng_for("draft", 62)
    rep = Report()
    cases = [
        ([], []),                                          # no node: one greedy step
        (greedy[:6], [-1, 0, 1, 2, 3, 4]),                 # chain, fully accepted
        ([int(greedy[0]), 5, 6, 7], [-1, -1, -1, -1]),     # star
        (greedy[:63], [-1] + list(range(62))),             # 63 nodes, the most a tree holds
    ]
    for tok, par in cases:
        res = oracle.verify_tree(om, st, tok, par)
        a, n, paths, L = _verify_tree(kv, [0], [st.ctx], [(tok, par)])
        check_tree(rep, res, L, int(a[0]), int(n[0]), paths[0])
        kv.truncate(0, st.ctx, st.pending)
    # a chain-shaped tree is the chain verify, bit for bit on the GPU too
    d = np.asarray(greedy[:6])
    a1, n1, _, L1 = _verify_tree(kv, [0], [st.ctx], [(d, [-1, 0, 1, 2, 3, 4])])
    kv.truncate(0, st.ctx, st.pending)
    import torch
    lg = torch.empty((7, TINY.vocab), dtype=torch.float32, device="cuda")
    a2, n2 = kv.verify([0], [st.ctx], [d], logits=lg)
    kv.truncate(0, st.ctx, st.pending)
    assert np.array_equal(L1, lg.cpu().numpy().astype(np.float64))
    assert int(a1[0]) == int(a2[0]) and int(n1[0]) == int(n2[0])
    print(rep)


def test_batch_of_trees_then_commit_and_continue(tiny):
    """Three sequences verified as trees in one call, committed (full and
    partial keeps), then verified again as chains and once more as trees:
    the later verifies read the K/V the tree verify moved into place."""
    om, gm = tiny
    kv = _kv(gm)
    rng = wt.rng_for("draft", 63)
    states = []
    for b, n in enumerate((120, 257, 64)):
        ctx = wt.uniform_context(wt.rng_for("context", 63, b), n, TINY.vocab)
        states.append(oracle.prefill(om, ctx))
        kv.prefill(b, ctx)
    rep = Report()
    for step in range(3):
        items, results = [], []
        for b, st in enumerate(states):
            greedy, _ = oracle.greedy_decode(om, st, 9)
            par = trees.eagle_tree(rng, int(rng.integers(8, 40)), 8, 4)
            tok = trees.plant_path(rng, par, greedy, int(rng.integers(0, 9)), TINY.vocab)
            items.append((tok, par))
            results.append(oracle.verify_tree(om, st, tok, par))
        a, n, paths, L = _verify_tree(kv, [0, 1, 2], [s.ctx for s in states], items)
        r0 = 0
        for b, res in enumerate(results):
            rows = len(items[b][0]) + 1
            diverged = check_tree(rep, res, L[r0:r0 + rows], int(a[b]), int(n[b]), paths[b])
            assert not diverged, "near tie on the accepted path (re-seed the test)"
            r0 += rows
        keep = [int(a[0]), max(0, int(a[1]) - 1), 0]
        kv.commit([0, 1, 2], keep)
        states = [oracle.commit_tree(st, res, kp) for st, res, kp in zip(states, results, keep)]
        for b, st in enumerate(states):
            assert kv.seq_info(b)[:2] == (st.ctx, st.pending)
        # a chain verify on the committed state
        for b, st in enumerate(states):
            greedy, _ = oracle.greedy_decode(om, st, 5)
            d = wt.plant_chain(rng, greedy, int(rng.integers(0, 5)), 4, TINY.vocab)
            res = oracle.verify(om, st, d)
            import torch
            lg = torch.empty((5, TINY.vocab), dtype=torch.float32, device="cuda")
            ac, nx = kv.verify([b], [st.ctx], [d], logits=lg)
            check_step(rep, res, lg.cpu().numpy().astype(np.float64), int(ac[0]), int(nx[0]), d)
            kv.truncate(b, st.ctx, st.pending)
    print(rep)


def test_tree_argument_errors(tiny):
    from paper_2606_01019_amd import hvd
    om, gm = tiny
    kv = _kv(gm)
    ctx = wt.uniform_context(wt.rng_for("context", 64), 40, TINY.vocab)
    kv.prefill(0, ctx)
    with pytest.raises(hvd.HvdError) as e:
        kv.verify_tree([0], [39], [([1, 2], [-1, 1])])  # a node may not be its own parent
    assert e.value.status == hvd.HVD_ERR_ARG
    with pytest.raises(hvd.HvdError) as e:
        kv.verify_tree([0], [39], [(list(range(64)), [-1] * 64)])  # 64 nodes
    assert e.value.status == hvd.HVD_ERR_RANGE
    with pytest.raises(hvd.HvdError) as e:
        kv.verify_tree([0], [39], [([TINY.vocab], [-1])])  # token out of range
    assert e.value.status == hvd.HVD_ERR_RANGE
    a, n, paths = kv.verify_tree([0], [39], [([1, 2], [-1, 0])])  # the state is unchanged by the failures
    assert 0 <= int(a[0]) <= 2



@pytest.fixture(scope="module")
def mid():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    from tests.test_gpu_mid import MID as cfg
    w = make_weights(cfg, seed=5, gain_std=0.1)
    return cfg, oracle.OracleModel(cfg, w), hvd.Model(cfg, w)


@pytest.mark.parametrize("n_nodes,accept", [(15, 4), (32, 6), (63, 8)])
def test_mid_trees_grouped_query(mid, n_nodes, accept):
    """Group-4 attention with head dim 128: 16 tree rows (64 query rows, the
    4-wave items), 33 and 64 rows (132 and 256 query rows, the 8-wave items
    of two row tiles per wave)."""
    import paper_2606_01019_amd as hvd
    cfg, om, gm = mid
    kv = hvd.KVCache(gm, max_seqs=1, n_pages=128)
    ctx = wt.uniform_context(wt.rng_for("context", 70 + n_nodes), 600, cfg.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(0, ctx)
    greedy, _ = oracle.greedy_decode(om, st, accept + 1)
    rng = wt.rng_for("draft", 70 + n_nodes)
    par = trees.eagle_tree(rng, n_nodes, 8, 4) if n_nodes < 63 else [-1] + [j // 4 for j in range(62)]
    tok = trees.plant_path(rng, par, greedy, accept, cfg.vocab)
    res = oracle.verify_tree(om, st, tok, par)
    a, n, paths, L = _verify_tree(kv, [0], [st.ctx], [(tok, par)])
    rep = Report()
    check_tree(rep, res, L, int(a[0]), int(n[0]), paths[0])
    print(f"{n_nodes} nodes: accepted {int(a[0])} (oracle {res.accepted}) {rep}")


def test_8b_trees_against_oracle_record(model8b):
    """Full 8B shape at the workload-2 context: four trees (tests/golden/
    tree2.json, written by tests/golden/make_golden.py from the oracle alone),
    compared at the sampled and top logits, per-row argmax and the accepted
    path."""
    import torch
    import paper_2606_01019_amd as hvd
    from tests.conftest import load_golden
    gold = load_golden("tree2.json")
    V = gold["model"]["vocab"]
    kv = hvd.KVCache(model8b, max_seqs=1, n_pages=(gold["context_len"] + 96) // 16 + 8)
    ctx = wt.zipf_context(wt.rng_for(*gold["context_seed"]), gold["context_len"], V)
    kv.prefill(0, ctx)
    c0, p0 = len(ctx) - 1, int(ctx[-1])
    ids = np.asarray(gold["sample_ids"])
    rep = Report()
    for st in gold["steps"]:
        tok, par = st["tokens"], st["parents"]
        lg = torch.empty((len(tok) + 1, V), dtype=torch.float32, device="cuda")
        a, n, paths = kv.verify_tree([0], [c0], [(tok, par)], logits=lg)
        kv.truncate(0, c0, p0)
        L = lg.cpu().numpy()
        err = float(np.abs(L[:, ids] - np.asarray(st["sample_logits"])).max())
        top = np.asarray(st["top_ids"])
        err = max(err, max(float(np.abs(L[r, top[r]] - np.asarray(st["top_logits"][r])).max())
                           for r in range(L.shape[0])))
        rep.max_err = max(rep.max_err, err)
        assert err <= LOGIT_TOL, f"logit error {err:.3e}"
        tie = np.asarray(st["margin"]) < TIE_MARGIN
        g_gpu = L.argmax(1)
        rep.rows += L.shape[0]
        rep.excused += int(tie.sum())
        assert not ((g_gpu != np.asarray(st["argmax"])) & ~tie).any()
        assert paths[0] == oracle.tree_accept(g_gpu, np.asarray(tok), np.asarray(par))
        on_path = [0] + [j + 1 for j in st["path"]]
        if not tie[on_path].any():
            assert paths[0] == st["path"] and int(n[0]) == st["next"]
        print(f"{len(tok)} nodes: path {paths[0]} (oracle {st['path']}) {rep}", flush=True)
