"""GPU parity of hvd_verify / hvd_commit against the CPU oracle on the tiny
decoder (2 layers, d_model 256, 4/4 heads of 64, SwiGLU 1024, vocab 4096):
context 512 uniform tokens, chain drafts of k = 8 planted from the oracle's
greedy continuation with the first mismatch at j in 0..8, plus the degenerate
and batched cases.  Every call goes through the C ABI of libhvd.so."""

import numpy as np
import pytest

import oracle
from tests._parity import Report, check_step, oracle_commit_as
from workloads import TINY, ModelConfig, make_weights, tokens as wt

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.fixture(scope="module")
def tiny(torch_cuda):
    import paper_2606_01019_amd as hvd
    w = make_weights(TINY, seed=42, gain_std=0.1)
    om = oracle.OracleModel(TINY, w)
    gm = hvd.Model(TINY, w)
    return om, gm


def _kv(gm, max_seqs=4, n_pages=512):
    import paper_2606_01019_amd as hvd
    return hvd.KVCache(gm, max_seqs, n_pages)


def _verify(torch, kv, ids, ctxs, drafts):
    rows = sum(len(d) + 1 for d in drafts)
    lg = torch.empty((rows, kv.model.cfg.vocab), dtype=torch.float32, device="cuda")
    a, n = kv.verify(ids, ctxs, drafts, logits=lg)
    return a, n, lg.cpu().numpy().astype(np.float64)


def test_tiny_config_planted_chain_k8(torch_cuda, tiny):
    om, gm = tiny
    kv = _kv(gm)
    rng = wt.rng_for("context", 1)
    ctx = wt.uniform_context(rng, 512, TINY.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(0, ctx)
    assert kv.seq_info(0)[:2] == (511, int(ctx[-1]))
    greedy, _ = oracle.greedy_decode(om, st, 9)
    rep = Report()
    drng = wt.rng_for("draft", 1)
    for j in range(9):
        d = wt.plant_chain(drng, greedy, j, 8, TINY.vocab)
        res = oracle.verify(om, st, d)
        assert res.accepted == j
        a, n, lg = _verify(torch_cuda, kv, [0], [st.ctx], [d])
        check_step(rep, res, lg, int(a[0]), int(n[0]), d)
        kv.truncate(0, st.ctx, st.pending)  # cancel: verify the next plant from the same state
    print(rep)


def test_tiny_decode_loop_commit_matches_oracle(torch_cuda, tiny):
    """Eight verify+commit cycles with planted drafts of varying length; the
    committed streams stay identical (re-synced only after a reported near tie)."""
    om, gm = tiny
    kv = _kv(gm)
    rng = wt.rng_for("context", 2)
    ctx = wt.uniform_context(rng, 200, TINY.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(1, ctx)
    rep = Report()
    drng = wt.rng_for("draft", 2)
    for step in range(8):
        k = int(drng.integers(0, 12))
        greedy, _ = oracle.greedy_decode(om, st, k + 1)
        a_plan = wt.geometric_accept(drng, 0.3, k)
        d = wt.plant_chain(drng, greedy, a_plan, k, TINY.vocab)
        res = oracle.verify(om, st, d)
        a, n, lg = _verify(torch_cuda, kv, [1], [st.ctx], [d])
        a, n = int(a[0]), int(n[0])
        diverged = check_step(rep, res, lg, a, n, d)
        kv.commit([1])
        st = oracle_commit_as(st, res, a, n) if diverged else oracle.commit(st, res)
        assert kv.seq_info(1)[:2] == (st.ctx, st.pending)
    print(rep)


def test_k0_is_greedy_step_and_full_acceptance(torch_cuda, tiny):
    om, gm = tiny
    kv = _kv(gm)
    ctx = wt.uniform_context(wt.rng_for("context", 3), 77, TINY.vocab)
    st = oracle.prefill(om, ctx)
    kv.prefill(2, ctx)
    rep = Report()
    res = oracle.verify(om, st, [])
    a, n, lg = _verify(torch_cuda, kv, [2], [st.ctx], [np.zeros(0, np.int32)])
    assert int(a[0]) == 0
    check_step(rep, res, lg, 0, int(n[0]), [])
    kv.truncate(2, st.ctx, st.pending)
    greedy, _ = oracle.greedy_decode(om, st, 17)
    res = oracle.verify(om, st, greedy[:16])
    a, n, lg = _verify(torch_cuda, kv, [2], [st.ctx], [greedy[:16]])
    check_step(rep, res, lg, int(a[0]), int(n[0]), greedy[:16])
    print(rep)


def test_batched_mixed_drafts_match_per_sequence_oracle(torch_cuda, tiny):
    """Four sequences of different context lengths (crossing page boundaries)
    and draft lengths (0, 1, 15, 64) in one verify."""
    om, gm = tiny
    kv = _kv(gm, max_seqs=4)
    rng = wt.rng_for("context", 4)
    lens = [15, 16, 300, 33]
    ks = [0, 1, 15, 64]
    states, drafts = [], []
    drng = wt.rng_for("draft", 4)
    for s, (L, k) in enumerate(zip(lens, ks)):
        c = wt.uniform_context(rng, L + 1, TINY.vocab)
        st = oracle.prefill(om, c)
        kv.prefill(s, c)
        g, _ = oracle.greedy_decode(om, st, min(k, 20) + 1)
        a_plan = min(len(g) - 1, wt.uniform_accept(drng, k))
        full = np.concatenate([g, wt.random_chain(drng, max(0, k + 1 - len(g)), TINY.vocab)])
        d = wt.plant_chain(drng, full, a_plan, k, TINY.vocab)
        states.append(st)
        drafts.append(d)
    a, n, lg = _verify(torch_cuda, kv, [0, 1, 2, 3], [s.ctx for s in states], drafts)
    rep = Report()
    row = 0
    for s in range(4):
        res = oracle.verify(om, states[s], drafts[s])
        k = len(drafts[s])
        check_step(rep, res, lg[row:row + k + 1], int(a[s]), int(n[s]), drafts[s])
        row += k + 1
    print(rep)


def test_rollback_and_reverify_is_bitwise_identical(torch_cuda, tiny):
    import torch
    om, gm = tiny
    kv = _kv(gm)
    ctx = wt.uniform_context(wt.rng_for("context", 5), 130, TINY.vocab)
    kv.prefill(0, ctx)
    d = wt.random_chain(wt.rng_for("draft", 5), 12, TINY.vocab)
    a1, n1, l1 = _verify(torch, kv, [0], [129], [d])
    kv.commit([0], keep=[0])
    # advance a few steps, then roll back to the first state and re-verify
    for _ in range(3):
        c, p, _ = kv.seq_info(0)
        a, n = kv.verify([0], [c], [d[:5]])
        kv.commit([0])
    kv.truncate(0, 129, int(ctx[-1]))
    a2, n2, l2 = _verify(torch, kv, [0], [129], [d])
    assert np.array_equal(l1, l2) and a1[0] == a2[0] and n1[0] == n2[0]


def test_page_assignment_does_not_change_results(torch_cuda, tiny):
    """Same sequence verified from different physical pages gives identical bits."""
    import torch
    om, gm = tiny
    kv = _kv(gm, max_seqs=3, n_pages=64)
    ctx = wt.uniform_context(wt.rng_for("context", 6), 100, TINY.vocab)
    filler = wt.uniform_context(wt.rng_for("context", 7), 250, TINY.vocab)
    d = wt.random_chain(wt.rng_for("draft", 6), 9, TINY.vocab)
    kv.prefill(0, ctx)
    a1, n1, l1 = _verify(torch, kv, [0], [99], [d])
    kv.seq_free(0)
    kv.prefill(1, filler)    # occupies the low pages
    kv.prefill(2, ctx)
    a2, n2, l2 = _verify(torch, kv, [2], [99], [d])
    assert np.array_equal(l1, l2)


def test_abi_errors_leave_state_unchanged(torch_cuda, tiny):
    import paper_2606_01019_amd as hvd
    om, gm = tiny
    kv = _kv(gm, max_seqs=2, n_pages=8)
    ctx = wt.uniform_context(wt.rng_for("context", 8), 40, TINY.vocab)
    kv.prefill(0, ctx)
    free0 = kv.free_pages()

    def err(fn, code):
        with pytest.raises(hvd.HvdError) as e:
            fn()
        assert e.value.status == code, str(e.value)

    err(lambda: kv.verify([0], [38], [[1, 2]]), hvd.hvd.HVD_ERR_STATE)          # ctx mismatch
    err(lambda: kv.verify([0], [39], [[1, TINY.vocab]]), hvd.hvd.HVD_ERR_RANGE)  # token out of range
    err(lambda: kv.verify([0], [39], [list(range(65))]), hvd.hvd.HVD_ERR_RANGE)  # k > max_draft
    err(lambda: kv.verify([1], [0], [[1]]), hvd.hvd.HVD_ERR_ARG)                 # unknown seq
    err(lambda: kv.verify([0, 0], [39, 39], [[1], [1]]), hvd.hvd.HVD_ERR_ARG)    # duplicate seq
    err(lambda: kv.commit([0]), hvd.hvd.HVD_ERR_STATE)                           # commit without verify
    big = wt.uniform_context(wt.rng_for("context", 9), 200, TINY.vocab)
    err(lambda: kv.prefill(1, big), hvd.hvd.HVD_ERR_OOM)                         # pool too small
    assert kv.free_pages() == free0 and kv.seq_info(0) == (39, int(ctx[-1]), False)
    a, n = kv.verify([0], [39], [[1, 2, 3]])
    err(lambda: kv.verify([0], [39], [[1]]), hvd.hvd.HVD_ERR_STATE)              # verify twice
    err(lambda: kv.commit([0], keep=[int(a[0]) + 1]), hvd.hvd.HVD_ERR_ARG)       # keep > accepted
    kv.commit([0])
    assert kv.seq_info(0)[0] == 39 + int(a[0]) + 1
