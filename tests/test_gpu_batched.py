"""Full-size parity of the long-draft and batched workloads against stored
oracle records (tests/golden/cfg3.json, cfg4.json, cfg5.json, written by
tests/golden/make_golden.py from the oracle alone):

* long context, cache drafts: 8B shape, one sequence at context 16384 built
  from mutated 64-token segments, drafts of k = 32, 48, 64 (65-row verifies,
  sub-chunked split-KV attention);
* mixed batch: 8B shape, 32 sequences with contexts 1024..8192 in one verify
  of ~850 rows (MFMA-tiled GEMMs, batched attention over the paged cache);
  the oracle checks 4 of them (shortest and longest context per draft kind)
  and two others are cross-checked against their own single-sequence verify;
* multi-step batch: 32B widths (64 q / 8 kv heads, SwiGLU 27648, vocab
  152064) at 4 layers, 8 sequences at context 8192, 16 verify + commit steps
  with k in 4..64; sequences 0 and 1 follow the oracle's trajectory.

Where make_golden.py has kept them (cfg3_rows.npz, cfg4_rows.npz), rows 0
and k of every checked verify are also compared whole, over the full
vocabulary.  Tolerances as everywhere: logits max-abs 2e-2; argmax, accepted length and
next token exact except near ties (top-2 margin < 2e-2)."""

import numpy as np
import pytest

from tests._parity import (LOGIT_TOL, TIE_MARGIN, Report, check_golden, check_whole_rows, load_whole_rows,
                           top2_margin)
from tests.conftest import load_golden
from workloads import SHAPE_32B, SHAPE_8B, batches, make_weights, tokens as wt

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _split_rows(L, drafts):
    out, r = [], 0
    for d in drafts:
        out.append(L[r:r + len(d) + 1])
        r += len(d) + 1
    return out


def test_long_context_cache_drafts(model8b):
    import torch
    import paper_2606_01019_amd as hvd
    gold = load_golden("cfg3.json")
    kv = hvd.KVCache(model8b, max_seqs=1, n_pages=(gold["context_len"] + 80) // 16 + 8)
    ctx = wt.segment_context(wt.rng_for(*gold["context_seed"]), gold["context_len"], SHAPE_8B.vocab)
    kv.prefill(0, ctx)
    c0, p0 = len(ctx) - 1, int(ctx[-1])
    whole = load_whole_rows("cfg3_rows.npz")
    rep = Report()
    for i, st in enumerate(gold["steps"]):
        d = np.asarray(st["draft"], dtype=np.int32)
        lg = torch.empty((len(d) + 1, SHAPE_8B.vocab), dtype=torch.float32, device="cuda")
        a, n = kv.verify([0], [c0], [d], logits=lg)
        L = lg.cpu().numpy()
        check_golden(rep, L, st, gold["sample_ids"], int(a[0]), int(n[0]))
        wr = check_whole_rows(L, whole[0][f"step{i}"], whole[1]) if whole is not None else float("nan")
        kv.truncate(0, c0, p0)
        print(f"k={len(d)}: accepted={int(a[0])} (oracle {st['accepted']}) {rep} whole rows {wr:.3e}", flush=True)


def test_mixed_batch(model8b):
    import torch
    import paper_2606_01019_amd as hvd
    gold = load_golden("cfg4.json")
    V = SHAPE_8B.vocab
    plans = batches.mixed_batch_plan()
    recs = {r["seq"]: r for r in gold["seqs"]}
    pages = sum((p.ctx_len + p.k + 16) // 16 + 1 for p in plans) + 64
    kv = hvd.KVCache(model8b, max_seqs=len(plans), n_pages=pages)
    ctxs = []
    for p in plans:
        c = batches.mixed_batch_context(p, V)
        kv.prefill(p.seq, c)
        ctxs.append(c)
    print(f"prefilled {sum(p.ctx_len for p in plans)} tokens", flush=True)
    drafts = []
    for p in plans:
        if p.seq in recs:
            drafts.append(np.asarray(recs[p.seq]["draft"], dtype=np.int32))
        else:  # unchecked sequences: any draft of the planned length
            drafts.append(wt.random_chain(wt.rng_for("draft", 4, p.seq, 1), p.k, V))
    ids = [p.seq for p in plans]
    ctx_lens = [p.ctx_len - 1 for p in plans]
    M = sum(len(d) + 1 for d in drafts)
    lg = torch.empty((M, V), dtype=torch.float32, device="cuda")
    a, n = kv.verify(ids, ctx_lens, drafts, logits=lg)
    L = _split_rows(lg.cpu().numpy(), drafts)
    rep = Report()
    whole = load_whole_rows("cfg4_rows.npz")
    worst_row = 0.0
    for b in gold["sampled"]:
        check_golden(rep, L[b], recs[b], gold["sample_ids"], int(a[b]), int(n[b]))
        if whole is not None:
            worst_row = max(worst_row, check_whole_rows(L[b], whole[0][f"seq{b}"], whole[1]))
    print(f"batch of {len(plans)} sequences, {M} rows: {rep} whole rows {worst_row:.3e}", flush=True)
    # two unchecked sequences verified alone must agree with the batched rows
    for p in plans:
        kv.truncate(p.seq, p.ctx_len - 1, int(ctxs[p.seq][-1]))
    for b in (3, 25):
        lone = torch.empty((len(drafts[b]) + 1, V), dtype=torch.float32, device="cuda")
        a1, n1 = kv.verify([b], [ctx_lens[b]], [drafts[b]], logits=lone)
        kv.truncate(b, ctx_lens[b], int(ctxs[b][-1]))
        Lb = lone.cpu().numpy()
        assert np.abs(Lb - L[b]).max() <= 2 * LOGIT_TOL
        tie = top2_margin(Lb) < TIE_MARGIN
        assert np.all((Lb.argmax(1) == L[b].argmax(1)) | tie)
        if not tie[:min(int(a1[0]), int(a[b])) + 1].any():
            assert int(a1[0]) == int(a[b]) and int(n1[0]) == int(n[b])


def test_multistep_batch_32b_widths():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    gold = load_golden("cfg5.json")
    cfg = SHAPE_32B.with_layers(gold["n_layers"])
    V = cfg.vocab
    w = make_weights(cfg, seed=42)
    model = hvd.Model(cfg, w)
    del w
    plans = batches.multistep_plan()
    n_seqs = len(plans[0])
    kv = hvd.KVCache(model, max_seqs=n_seqs, n_pages=n_seqs * ((8192 + 16 * 66) // 16 + 4))
    ctxs = [batches.multistep_context(b, 8192, V) for b in range(n_seqs)]
    for b in range(n_seqs):
        kv.prefill(b, ctxs[b])
    lens = [8191] * n_seqs
    gseq = {g["seq"]: g["steps"] for g in gold["seqs"]}
    live = {b: True for b in gseq}
    rep = Report()
    for s, row in enumerate(plans):
        drafts = []
        for b in range(n_seqs):
            if b in gseq and live[b]:
                drafts.append(np.asarray(gseq[b][s]["draft"], dtype=np.int32))
            else:
                drafts.append(wt.random_chain(wt.rng_for("draft", 5, b, s, 1), row[b].k, V))
        M = sum(len(d) + 1 for d in drafts)
        lg = torch.empty((M, V), dtype=torch.float32, device="cuda")
        a, n = kv.verify(list(range(n_seqs)), lens, drafts, logits=lg)
        L = _split_rows(lg.cpu().numpy(), drafts)
        for b in gseq:
            if live[b] and check_golden(rep, L[b], gseq[b][s], gold["sample_ids"], int(a[b]), int(n[b])):
                live[b] = False  # a near tie sent the GPU down another branch
                print(f"sequence {b} left the oracle trajectory at step {s} (near tie)", flush=True)
        kv.commit(list(range(n_seqs)))
        lens = [lens[b] + int(a[b]) + 1 for b in range(n_seqs)]
        print(f"step {s}: {M} rows, {rep}", flush=True)
    assert rep.rows > 0
