"""hvd_verify_noalloc (the allocation-free verify: step scratch in the
library's static device array) against hvd_verify on the same states: two
calls in a row, the second with a smaller batch, on a grouped-query decoder
whose steps use the down GEMM's K split and split-KV attention (both keep
their partials in that scratch); and a step too large for the static array is
refused before any state changes."""

import numpy as np
import pytest

from tests._parity import LOGIT_TOL, TIE_MARGIN, top2_margin
from workloads import ModelConfig, make_weights, tokens as wt

pytestmark = pytest.mark.gpu

MID = ModelConfig("mid", 2, 1024, 8, 2, 128, 8192, 16384, 5.0e5, max_pos=4096)


def _run(torch, kv, ids, ctxs, drafts, noalloc):
    rows = sum(len(d) + 1 for d in drafts)
    lg = torch.empty((rows, kv.model.cfg.vocab), dtype=torch.float32, device="cuda")
    a, n = kv.verify(ids, ctxs, drafts, logits=lg, noalloc=noalloc)
    return a, n, lg.cpu().numpy()


def test_noalloc_matches_verify_twice_then_smaller():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    w = make_weights(MID, seed=5, gain_std=0.1)
    gm = hvd.Model(MID, w)
    kv = hvd.KVCache(gm, max_seqs=4, n_pages=512)
    ctxs = [wt.uniform_context(wt.rng_for("context", 70 + b), 700 + 97 * b, MID.vocab) for b in range(3)]
    for b in range(3):
        kv.prefill(b, ctxs[b])
    lens = [len(c) - 1 for c in ctxs]
    cases = [([0, 1, 2], [16, 5, 33]), ([1], [3])]  # second call: a smaller input
    for ids, ks in cases:
        drafts = [wt.random_chain(wt.rng_for("draft", 70, b, len(ids)), k, MID.vocab) for b, k in zip(ids, ks)]
        c = [lens[b] for b in ids]
        a0, n0, L0 = _run(torch, kv, ids, c, drafts, noalloc=False)
        for b in ids:
            kv.truncate(b, lens[b], int(ctxs[b][-1]))  # cancel the uncommitted verify
        a1, n1, L1 = _run(torch, kv, ids, c, drafts, noalloc=True)
        err = float(np.abs(L1.astype(np.float64) - L0).max())
        assert err <= LOGIT_TOL, err
        tie = top2_margin(L0) < TIE_MARGIN
        assert np.all((L1.argmax(1) == L0.argmax(1)) | tie)
        assert np.array_equal(a1, a0) and np.array_equal(n1, n0), (a0, a1, n0, n1)
        print(f"batch {ids} k={ks}: max|noalloc - verify| = {err:.3e} "
              f"({'bitwise equal' if err == 0.0 else 'rounding differs'}), accepted {a1.tolist()}", flush=True)
        kv.commit(ids)
        for j, b in enumerate(ids):
            lens[b] += int(a1[j]) + 1
            ctxs[b] = np.concatenate([ctxs[b], np.asarray(drafts[j][:a1[j]]), [n1[j]]])
    assert kv.free_pages() > 0


def test_noalloc_refuses_a_step_too_large_for_the_static_scratch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    wide = ModelConfig("wide-vocab", 1, 256, 4, 4, 64, 1024, 262144, 1.0e4, max_pos=4096)
    gm = hvd.Model(wide, make_weights(wide, seed=3))
    kv = hvd.KVCache(gm, max_seqs=8, n_pages=64)
    drafts = [np.zeros(64, dtype=np.int32)] * 8  # 520 rows: LM-head partials alone exceed 64 MiB
    with pytest.raises(hvd.HvdError) as e:
        kv.verify(list(range(8)), [0] * 8, drafts, noalloc=True)
    assert e.value.status == hvd.hvd.HVD_ERR_RANGE and "static scratch" in str(e.value)
    ctx = wt.uniform_context(wt.rng_for("context", 71), 40, wide.vocab)
    kv.prefill(0, ctx)  # the handle still works, and the refused call changed no state
    a, n = kv.verify([0], [len(ctx) - 1], [np.asarray([1, 2, 3], dtype=np.int32)], noalloc=True)
    assert 0 <= int(a[0]) <= 3 and kv.seq_info(0)[2]
