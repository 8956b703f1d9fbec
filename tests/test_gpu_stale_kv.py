"""K/V past the end of a sequence never reaches a result (Alg. 1 appends only
the committed block; the rejected suffix and unused slots must not matter),
checked bit for bit on a grouped-query decoder whose verify uses split-KV
attention with its merge (8 q / 2 kv heads of 128):

* every slot of the KV pool filled with fp16 NaN before the prompt is
  prefilled: unwritten slots of the last page and never-used pages hold
  NaN, the verify's logits and results equal a clean pool's bit for bit;
* rollback and re-verify: the K/V rows a longer, cancelled draft left past
  the new rows change nothing, and a committed step rolled back and
  re-verified reproduces the same bits;
* another page assignment (a different sequence holding the first pages)
  gives the same bits."""

import numpy as np
import pytest

from workloads import ModelConfig, make_weights, tokens as wt

pytestmark = pytest.mark.gpu

MID = ModelConfig("mid", 2, 1024, 8, 2, 128, 8192, 16384, 5.0e5, max_pos=4096)
NAN_F16 = 0x7E00


@pytest.fixture(scope="module")
def mid():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_01019_amd as hvd
    return torch, hvd.Model(MID, make_weights(MID, seed=9, gain_std=0.1))


def _pool_bytes(n_pages):
    # the KV pool opens the handle's buffer: [layer][page][K|V][kv head][16][head dim] fp16
    return MID.n_layers * n_pages * 2 * MID.n_kv_heads * 16 * MID.head_dim * 2


def _verify(torch, kv, sid, ctx, d):
    lg = torch.empty((len(d) + 1, MID.vocab), dtype=torch.float32, device="cuda")
    a, n = kv.verify([sid], [ctx], [d], logits=lg)
    return int(a[0]), int(n[0]), lg.cpu().numpy()


def test_stale_and_poisoned_kv_change_no_bit(mid):
    import paper_2606_01019_amd as hvd
    torch, gm = mid
    n_pages = 160
    ctx = wt.uniform_context(wt.rng_for("context", 95), 1133, MID.vocab)  # last page partly filled
    d9 = wt.random_chain(wt.rng_for("draft", 95, 9), 9, MID.vocab)
    d16 = wt.random_chain(wt.rng_for("draft", 95, 16), 16, MID.vocab)

    clean = hvd.KVCache(gm, max_seqs=2, n_pages=n_pages)
    clean.prefill(0, ctx)
    c0, p0, _ = clean.seq_info(0)
    ref = _verify(torch, clean, 0, c0, d9)

    pois = hvd.KVCache(gm, max_seqs=2, n_pages=n_pages)
    nb = _pool_bytes(n_pages)
    assert nb <= pois.buf.numel()
    pois.buf[:nb].view(torch.int16).fill_(NAN_F16)
    torch.cuda.synchronize()
    pois.prefill(0, ctx)
    got = _verify(torch, pois, 0, c0, d9)
    assert got[:2] == ref[:2] and np.array_equal(got[2], ref[2]), "NaN in unwritten K/V slots changed the result"
    assert np.isfinite(got[2]).all()

    # a longer draft writes K/V at ctx .. ctx+16; cancel it and verify the shorter one
    pois.truncate(0, c0, p0)
    _verify(torch, pois, 0, c0, d16)
    pois.truncate(0, c0, p0)
    got = _verify(torch, pois, 0, c0, d9)
    assert got[:2] == ref[:2] and np.array_equal(got[2], ref[2]), "stale rows of a cancelled draft changed the result"

    # commit, roll back to the same state, re-verify
    pois.commit([0])
    assert pois.seq_info(0)[0] == c0 + got[0] + 1
    pois.truncate(0, c0, p0)
    again = _verify(torch, pois, 0, c0, d9)
    assert again[:2] == ref[:2] and np.array_equal(again[2], ref[2]), "rollback + re-verify differs"

    # other pages: a second sequence takes the first pages of a fresh pool
    perm = hvd.KVCache(gm, max_seqs=2, n_pages=n_pages)
    perm.buf[:nb].view(torch.int16).fill_(NAN_F16)
    torch.cuda.synchronize()
    perm.prefill(1, wt.uniform_context(wt.rng_for("context", 96), 300, MID.vocab))
    perm.prefill(0, ctx)
    got = _verify(torch, perm, 0, c0, d9)
    assert got[:2] == ref[:2] and np.array_equal(got[2], ref[2]), "another page assignment changed the result"
    print(f"accepted {ref[0]}, next {ref[1]}: identical bits in all four cases", flush=True)
