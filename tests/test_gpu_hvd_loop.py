"""The Hybrid Verified Decoding loop (Alg. 1) driving the GPU verify step on
the tiny decoder: whatever the draft selection, the committed stream is the
target's greedy stream (compared with the GPU's own one-token greedy steps;
a difference is allowed only at a near tie of the oracle's logits, where a
k-row verify may round the other way)."""

import numpy as np
import pytest

import oracle
from paper_2606_01019_amd import hvd_loop as hl
from tests._parity import TIE_MARGIN, top2_margin
from workloads import TINY, make_weights, tokens as wt

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    w = make_weights(TINY, seed=42, gain_std=0.1)
    return oracle.OracleModel(TINY, w), hvd.Model(TINY, w)


def _greedy(kv, sid, prompt, n):
    kv.prefill(sid, prompt)
    out = []
    for _ in range(n):
        c, _, _ = kv.seq_info(sid)
        _, nx = kv.verify([sid], [c], [np.zeros(0, np.int32)])
        kv.commit([sid])
        out.append(int(nx[0]))
    kv.seq_free(sid)
    return out


@pytest.mark.parametrize("policy", ["always", "mlp"])
def test_loop_on_gpu_commits_the_greedy_stream(tiny, policy):
    import paper_2606_01019_amd as hvd
    om, gm = tiny
    kv = hvd.KVCache(gm, max_seqs=2, n_pages=256)
    prompt = wt.segment_context(wt.rng_for("context", 91), 600, TINY.vocab, seg=32, n_base=4)
    n_new = 96
    ref = _greedy(kv, 1, prompt, n_new)
    if policy == "always":
        pred = lambda phi: np.full(len(phi), np.inf)
    else:  # trained on the replay of another prompt's greedy trace (App. B)
        other = wt.segment_context(wt.rng_for("context", 92), 600, TINY.vocab, seg=32, n_base=4)
        trace = list(other) + _greedy(kv, 1, other, 160)
        X, y = hl.replay_labels(trace, len(other))
        pred = hl.PayoffMLP()
        pred.fit(X, y, batch=4096, epochs=20)
    dec = hl.HybridVerifiedDecoder(kv, 0, pred)
    out, st = dec.generate(prompt, n_new)
    print(f"{policy}: {st.cycles} cycles for {st.generated} tokens ({st.cycles_per_1k:.0f} per 1K), "
          f"{st.cache_steps} cache verifies, accepted {st.cache_accepted}")
    if out != ref:
        p = next(i for i, (a, b) in enumerate(zip(out, ref)) if a != b)
        st0 = oracle.prefill(om, list(prompt) + ref[:p])
        r = oracle.verify(om, st0, [])
        assert top2_margin(r.logits)[0] < TIE_MARGIN, f"streams differ at {p} without a near tie"
        print(f"streams part at token {p} (near tie)")
