"""Full-size parity on the 8B-shaped decoder (32 layers, d_model 4096, 32 q /
8 kv heads of 128, SwiGLU 14336, vocab 128256, rotary theta 5e5), batch 1,
context 2048 Zipf(1.1) tokens, chain drafts k = 1, 2, 4, 8, 16 planted from
the oracle's greedy continuation (tests/golden/cfg2.json, written by
tests/golden/make_golden.py from the oracle alone).

Compared per verify: logits at 64 fixed vocabulary ids and at each row's
oracle top-8 ids (max-abs <= 2e-2), rows 0 and k whole against the oracle's
complete rows (tests/golden/cfg2_rows.npz, when written), per-row argmax
(except near-tie rows), accepted length and next token.  The same hvd_verify launch configuration as
bench.py's timed steps (batch 1, k <= 16)."""

import json
import os

import numpy as np
import pytest

from tests._parity import LOGIT_TOL, TIE_MARGIN, check_whole_rows, load_whole_rows

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def setup8b(model8b):
    import torch
    import paper_2606_01019_amd as hvd
    from workloads import SHAPE_8B, tokens as wt
    with open(os.path.join(HERE, "golden", "cfg2.json")) as f:
        gold = json.load(f)
    model = model8b
    kv = hvd.KVCache(model, max_seqs=1, n_pages=256)
    ctx = wt.zipf_context(wt.rng_for(*gold["context_seed"]), gold["context_len"], SHAPE_8B.vocab)
    kv.prefill(0, ctx)
    print("prefill done", flush=True)
    return torch, kv, gold, ctx


def test_8b_verify_matches_oracle_golden(setup8b):
    torch, kv, gold, ctx = setup8b
    ids = np.asarray(gold["sample_ids"])
    V = kv.model.cfg.vocab
    c0, p0 = len(ctx) - 1, int(ctx[-1])
    whole = load_whole_rows("cfg2_rows.npz")
    worst, worst_row, excused = 0.0, 0.0, 0
    for i, st in enumerate(gold["steps"]):
        d = np.asarray(st["draft"], dtype=np.int32)
        k = len(d)
        lg = torch.empty((k + 1, V), dtype=torch.float32, device="cuda")
        a, n = kv.verify([0], [c0], [d], logits=lg)
        L = lg.cpu().numpy()
        ref_s = np.asarray(st["sample_logits"])
        err = np.abs(L[:, ids] - ref_s).max()
        top_ids = np.asarray(st["top_ids"])
        err_top = max(np.abs(L[r, top_ids[r]] - np.asarray(st["top_logits"][r])).max() for r in range(k + 1))
        worst = max(worst, err, err_top)
        assert err <= LOGIT_TOL and err_top <= LOGIT_TOL, (k, err, err_top)
        if whole is not None:
            worst_row = max(worst_row, check_whole_rows(L, whole[0][f"step{i}"], whole[1]))
        margin = np.asarray(st["margin"])
        g_gpu = L.argmax(axis=1)
        g_ref = np.asarray(st["argmax"])
        tie = margin < TIE_MARGIN
        excused += int(tie.sum())
        assert np.all((g_gpu == g_ref) | tie), (k, np.flatnonzero(g_gpu != g_ref))
        if not tie[:st["accepted"] + 1].any():
            assert int(a[0]) == st["accepted"] and int(n[0]) == st["next"], (k, a, n, st["accepted"], st["next"])
        kv.truncate(0, c0, p0)
        print(f"k={k}: accepted={int(a[0])} (oracle {st['accepted']}) max|dlogit|={max(err, err_top):.2e}", flush=True)
    print(f"worst max|dlogit| = {worst:.3e} (whole rows {worst_row:.3e}), near-tie rows = {excused}")


def test_8b_bitwise_determinism_and_k0_greedy(setup8b):
    """Re-verifying the same state gives identical bits; k = 0 returns the
    argmax of the pending row (the greedy step)."""
    torch, kv, gold, ctx = setup8b
    V = kv.model.cfg.vocab
    c0, p0 = len(ctx) - 1, int(ctx[-1])
    d = np.asarray(gold["steps"][-1]["draft"], dtype=np.int32)
    outs = []
    for _ in range(2):
        lg = torch.empty((len(d) + 1, V), dtype=torch.float32, device="cuda")
        a, n = kv.verify([0], [c0], [d], logits=lg)
        kv.truncate(0, c0, p0)
        outs.append((lg.cpu().numpy(), int(a[0]), int(n[0])))
    assert np.array_equal(outs[0][0], outs[1][0]) and outs[0][1:] == outs[1][1:]
    lg = torch.empty((1, V), dtype=torch.float32, device="cuda")
    a, n = kv.verify([0], [c0], [np.zeros(0, np.int32)], logits=lg)
    kv.truncate(0, c0, p0)
    assert int(a[0]) == 0 and int(n[0]) == int(lg.cpu().numpy()[0].argmax())
    if gold["steps"][0]["margin"][0] >= TIE_MARGIN:
        assert int(n[0]) == gold["steps"][0]["argmax"][0]
