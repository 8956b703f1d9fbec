"""GPU parity of the device-resident verify loop (hvd_async_begin / _step /
_end) against the CPU oracle.

Each step of the loop is the verify step followed by the commit of the whole
accepted block (Alg. 1, Verify then append z_t), with the drafts read from
device memory.  The drafts come from the library's copy drafter over a
token stream (the oracle's greedy continuation with tokens replaced at rate
0.3, so acceptance is geometric) or from the host between steps.  The
expected (accepted, next) of every step follows from the oracle's greedy
continuation alone: a draft is accepted up to its first token that differs
from the continuation, and the next token is the continuation's.  Steps
whose decisions include an oracle near tie (top-2 margin below 2e-2) end
the comparison, as in the other parity tests.  After the loop, a
synchronous verify on the loop's KV cache is checked against the oracle."""


import numpy as np
import pytest

import oracle
from tests._parity import TIE_MARGIN, Report, check_step, oracle_commit_as
from workloads import TINY, ModelConfig, make_weights, tokens as wt

pytestmark = pytest.mark.gpu

MID = ModelConfig("mid", 2, 1024, 8, 2, 128, 8192, 16384, 5.0e5, max_pos=4096)


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
    return oracle.OracleModel(TINY, w), hvd.Model(TINY, w)


@pytest.fixture(scope="module")
def mid(torch_cuda):
    import paper_2606_01019_amd as hvd
    w = make_weights(MID, seed=5, gain_std=0.1)
    return oracle.OracleModel(MID, w), hvd.Model(MID, w)


def greedy(om, st, n):
    return np.array(oracle.greedy_decode(om, st, n)[0], dtype=np.int64)


class Follow:
    """Checks a loop's steps one by one against the oracle, which follows
    the committed stream: each step's draft is verified by the oracle from
    the state the GPU reached; (accepted, next) must match unless a near tie
    lies on the accepted path, and then the GPU's first differing token must
    be within the tie margin of the oracle's best, and the oracle continues
    from the GPU's block."""

    def __init__(self, om):
        self.om = om
        self.rep = Report()
        self.diverged = 0
        self.steps = 0

    def step(self, st, d, a_g, n_g):
        # a token outside the vocabulary is never accepted, and no later row
        # can be: the oracle verifies the draft up to it
        d = np.asarray(d, dtype=np.int64)
        bad = np.flatnonzero((d < 0) | (d >= self.om.cfg.vocab))
        d = d[:bad[0]] if bad.size else d
        assert a_g <= len(d)
        res = oracle.verify(self.om, st, d)
        self.steps += 1
        if not check_step(self.rep, res, None, a_g, n_g, d):
            return oracle.commit(st, res)
        rows = [int(t) for t in d[:a_g]] + [int(n_g)]
        for r, t in enumerate(rows):
            if t != int(res.argmax[r]):
                assert 0 <= t < self.om.cfg.vocab
                assert res.logits[r, t] >= res.logits[r].max() - TIE_MARGIN, (r, t)
                break
        self.diverged += 1
        return oracle_commit_as(st, res, a_g, n_g)

    def __str__(self):
        return f"{self.steps} steps, {self.diverged} near-tie re-syncs, {self.rep}"


def ref_drafter(ref, ref_start, k):
    def at(c):
        j = np.arange(c + 1, c + 1 + k) - ref_start
        return np.where((j >= 0) & (j < len(ref)), ref[np.clip(j, 0, len(ref) - 1)], -1)
    return at


def check_after_loop(torch, om, kv, sid, st, rep, k=8):
    """The loop's KV cache continues correctly: the host state equals the
    oracle's, and a synchronous verify of the oracle's next k greedy tokens
    matches the oracle."""
    assert kv.seq_info(sid)[:2] == (st.ctx, st.pending)
    d = greedy(om, st, k)
    res = oracle.verify(om, st, d)
    lg = torch.empty((len(d) + 1, om.cfg.vocab), dtype=torch.float32, device="cuda")
    a, n = kv.verify([sid], [st.ctx], [d], logits=lg)
    check_step(rep, res, lg.cpu().numpy().astype(np.float64), int(a[0]), int(n[0]), d)
    kv.commit([sid])


def run_copy_loop(torch, om, gm, seqs, steps, n_pages=512, seed=0, attn_min_items=None):
    """seqs: list of (context length, k).  Returns the mean accepted length per sequence."""
    import paper_2606_01019_amd as hvd
    kv = hvd.KVCache(gm, max_seqs=len(seqs), n_pages=n_pages)
    if attn_min_items:
        kv.set_option(hvd.hvd.HVD_OPT_ATTN_MIN_ITEMS, attn_min_items)
    V = om.cfg.vocab
    sts, refs = [], []
    for b, (L, k) in enumerate(seqs):
        ctx = wt.uniform_context(wt.rng_for("context", 300 + seed + b), L, V)
        st = oracle.prefill(om, ctx)
        kv.prefill(b, ctx)
        G = greedy(om, st, steps * (k + 1) + 1)
        sts.append(st)
        refs.append(wt.corrupt_stream(wt.rng_for("draft", 300 + seed + b), G, 0.3, V))
    R = max(len(r) for r in refs)
    ref = np.full((len(seqs), R), -1, dtype=np.int32)
    for b, r in enumerate(refs):
        ref[b, :len(r)] = r
    starts = [st.ctx + 1 for st in sts]
    print(f"loop: seqs={seqs} steps={steps}", flush=True)
    loop = kv.async_loop(list(range(len(seqs))), [st.ctx for st in sts], [k for _, k in seqs], steps,
                         ref=torch.tensor(ref, device="cuda"), ref_start=starts)
    loop.step(steps)
    assert loop.end() == steps
    hist = loop.history.cpu().numpy()
    state = loop.state.cpu().numpy()
    B = len(seqs)
    assert int(state[2 * B]) == steps
    means = []
    for b, (L, k) in enumerate(seqs):
        f = Follow(om)
        st = sts[b]
        draft_at = ref_drafter(refs[b], starts[b], k)
        for s in range(steps):
            st = f.step(st, draft_at(st.ctx), int(hist[s, b, 0]), int(hist[s, b, 1]))
        assert (int(state[b]), int(state[B + b])) == (st.ctx, st.pending)
        check_after_loop(torch, om, kv, b, st, f.rep)
        print(f"seq {b} (ctx {L}, k {k}): accepted per step {hist[:, b, 0].tolist()}; {f}")
        means.append(float(hist[:, b, 0].mean()))
    kv.close()
    return means


@pytest.mark.parametrize("min_items", [None, 4])
def test_async_copy_drafter_tiny(torch_cuda, tiny, min_items):
    """Batch 1, k = 8, twelve steps.  min_items 4 plans 256-position KV chunks
    (several sub-chunks per item, chunk ends moving inside them); the
    default plans 32-position chunks whose count grows during the loop."""
    om, gm = tiny
    m = run_copy_loop(torch_cuda, om, gm, [(512, 8)], 12, seed=1 if min_items else 0, attn_min_items=min_items)
    assert m[0] > 0.5  # drafts were accepted: the loop followed the stream


def test_async_copy_drafter_batch_mixed_k_tiny(torch_cuda, tiny):
    """Three sequences (contexts 100, 333, 700; k = 0, 3, 8): plain greedy
    steps on the device beside drafts, ten steps."""
    om, gm = tiny
    m = run_copy_loop(torch_cuda, om, gm, [(100, 0), (333, 3), (700, 8)], 10, seed=10)
    assert m[0] == 0 and m[2] > 0.5


def test_async_copy_drafter_mid_gqa_row_groups(torch_cuda, mid):
    """Grouped-query decoder (group 4, head 128): k = 16 (68 query rows per
    kv head) and k = 64 (260 rows: two row groups of the attention items)."""
    om, gm = mid
    m = run_copy_loop(torch_cuda, om, gm, [(600, 16), (900, 64)], 5, n_pages=256, seed=20)
    assert max(m) > 0.5


def test_async_host_written_drafts_and_invalid_tokens(torch_cuda, tiny):
    """Drafts written into the loop's buffer between steps (a stand-in for a
    GPU drafter), planted from the oracle's continuation of the state
    reached, including tokens outside the vocabulary (never accepted)."""
    torch = torch_cuda
    import paper_2606_01019_amd as hvd
    om, gm = tiny
    V = TINY.vocab
    kv = hvd.KVCache(gm, max_seqs=1, n_pages=128)
    ctx = wt.uniform_context(wt.rng_for("context", 330), 257, V)
    st = oracle.prefill(om, ctx)
    kv.prefill(0, ctx)
    k, steps = 4, 8
    drng = wt.rng_for("draft", 330)
    loop = kv.async_loop([0], [st.ctx], [k], steps)
    f = Follow(om)
    for s in range(steps):
        kv.stream.synchronize()
        assert int(loop.state[0].item()) == st.ctx
        g = greedy(om, st, k + 1)
        d = wt.plant_chain(drng, g, wt.geometric_accept(drng, 0.4, k), k, V).astype(np.int64)
        if s == 2:
            d[0] = -7          # rejected at once
        elif s == 5:
            d[:2] = g[:2]
            d[2] = V + 5       # two accepted, then rejected
        with torch.cuda.stream(kv.stream):
            loop.drafts.copy_(torch.tensor(d.astype(np.int32)))
        loop.step(1)
        kv.stream.synchronize()
        a_g, n_g = (int(x) for x in loop.history[s, 0].cpu())
        if s == 2:
            assert a_g == 0
        if s == 5:
            assert a_g <= 2
        st = f.step(st, d, a_g, n_g)
    assert loop.end() == steps
    check_after_loop(torch, om, kv, 0, st, f.rep)
    print(f)
    kv.close()


def test_async_loop_errors_and_lock(torch_cuda, tiny):
    import paper_2606_01019_amd as hvd
    from paper_2606_01019_amd.hvd import HVD_ERR_OOM, HVD_ERR_RANGE, HVD_ERR_STATE, HvdError
    torch = torch_cuda
    om, gm = tiny
    kv = hvd.KVCache(gm, max_seqs=2, n_pages=48)
    ctx = wt.uniform_context(wt.rng_for("context", 340), 300, TINY.vocab)
    kv.prefill(0, ctx)
    kv.prefill(1, ctx)
    free0 = kv.free_pages()
    with pytest.raises(HvdError) as e:  # 40 steps of 9 tokens need 42 pages for one sequence
        kv.async_loop([0, 1], [299, 299], [8, 8], 40)
    assert e.value.status == HVD_ERR_OOM and kv.free_pages() == free0
    loop = kv.async_loop([0], [299], [2], 3)
    with pytest.raises(HvdError) as e:
        kv.verify([0], [299], [[1]])
    assert e.value.status == HVD_ERR_STATE
    a, n = kv.verify([1], [299], [[5]])  # the other sequence is free to verify
    kv.commit([1])
    loop.step(2)
    with pytest.raises(HvdError) as e:
        loop.step(2)
    assert e.value.status == HVD_ERR_RANGE
    loop.step(1)
    assert loop.end() == 3
    h = loop.history.cpu().numpy()
    ctx_after = 299 + sum(int(h[s, 0, 0]) + 1 for s in range(3))
    assert kv.seq_info(0)[:2] == (ctx_after, int(h[2, 0, 1]))
    # with no drafter and an all-zero draft buffer, each step commits at least the target token
    assert ctx_after >= 302
    a, n = kv.verify([0], [ctx_after], [[1, 2]])  # the sequence is back under host control
    kv.commit([0])
    kv.close()


def test_async_loop_interleaved_with_host_verifies(torch_cuda, tiny):
    """A device-resident loop on one sequence while the host verifies and
    commits another on the same handle between its steps (shared workspace,
    page-table updates of the other sequence, cached step graphs on): both
    streams follow the oracle."""
    torch = torch_cuda
    import paper_2606_01019_amd as hvd
    om, gm = tiny
    V = TINY.vocab
    kv = hvd.KVCache(gm, max_seqs=2, n_pages=256)
    kv.set_graphs(True)
    ctx0 = wt.uniform_context(wt.rng_for("context", 350), 300, V)
    ctx1 = wt.uniform_context(wt.rng_for("context", 351), 200, V)
    st0, st1 = oracle.prefill(om, ctx0), oracle.prefill(om, ctx1)
    kv.prefill(0, ctx0)
    kv.prefill(1, ctx1)
    k, steps = 4, 6
    G = greedy(om, st0, steps * (k + 1) + 1)
    ref = wt.corrupt_stream(wt.rng_for("draft", 350), G, 0.3, V)
    loop = kv.async_loop([0], [st0.ctx], [k], steps, ref=torch.tensor(ref[None, :], device="cuda"),
                         ref_start=[st0.ctx + 1])
    f0, rep1 = Follow(om), Report()
    drng = wt.rng_for("draft", 351)
    for s in range(steps):
        loop.step(1)
        # the host-driven sequence, between the loop's steps
        g = greedy(om, st1, 7)
        d = wt.plant_chain(drng, g, wt.geometric_accept(drng, 0.4, 6), 6, V)
        res = oracle.verify(om, st1, d)
        lg = torch.empty((7, V), dtype=torch.float32, device="cuda")
        a, n = kv.verify([1], [st1.ctx], [d], logits=lg)
        kv.commit([1])
        div = check_step(rep1, res, lg.cpu().numpy().astype(np.float64), int(a[0]), int(n[0]), d)
        st1 = oracle_commit_as(st1, res, int(a[0]), int(n[0])) if div else oracle.commit(st1, res)
    assert loop.end() == steps
    hist = loop.history.cpu().numpy()
    draft_at = ref_drafter(ref, st0.ctx + 1, k)
    for s in range(steps):
        st0 = f0.step(st0, draft_at(st0.ctx), int(hist[s, 0, 0]), int(hist[s, 0, 1]))
    check_after_loop(torch, om, kv, 0, st0, f0.rep)
    assert kv.seq_info(1)[:2] == (st1.ctx, st1.pending)
    print(f"loop: {f0}; host-driven: {rep1}")
    kv.close()
