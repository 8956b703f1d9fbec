"""Graph replay of the verify step: every replay equals the eager launch
bit for bit, with eager work and other shapes interleaved between replays."""

import numpy as np
import pytest

from workloads import TINY, make_weights, tokens as wt

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    gm = hvd.Model(TINY, make_weights(TINY, seed=42, gain_std=0.1))
    kv = hvd.KVCache(gm, max_seqs=2, n_pages=128)
    ctx = wt.uniform_context(wt.rng_for("context", 11), 300, TINY.vocab)
    kv.prefill(0, ctx)
    c0, p0 = 299, int(ctx[-1])
    drafts = [wt.random_chain(wt.rng_for("draft", 11 + i), k, TINY.vocab) for i, k in enumerate((3, 8, 0, 15))]

    def run(d):
        lg = torch.empty((len(d) + 1, TINY.vocab), dtype=torch.float32, device="cuda")
        a, n = kv.verify([0], [c0], [d], logits=lg)
        kv.truncate(0, c0, p0)
        return lg.cpu().numpy(), int(a[0]), int(n[0])

    kv.set_graphs(False)
    eager = [run(d) for d in drafts]
    kv.set_graphs(True)
    for rep in range(4):
        for d, ref in zip(drafts, eager):
            got = run(d)
            assert np.array_equal(got[0], ref[0]) and got[1:] == ref[1:], (rep, len(d))
        # eager work between replays: another sequence, other shapes
        kv.set_graphs(False)
        kv.prefill(1, ctx[:50])
        kv.verify([1], [49], [drafts[1]])
        kv.seq_free(1)
        kv.set_graphs(True)
