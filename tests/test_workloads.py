"""The seeded input generators: deterministic, thread-count independent, and
shaped as the workloads state."""

import numpy as np

from workloads import ModelConfig, TINY, make_tensor, make_weights, canonical_tensors, tokens as wt
from workloads.weights import f32_to_bf16_bits


def test_weights_deterministic_and_thread_independent():
    from concurrent.futures import ThreadPoolExecutor
    cfg = ModelConfig("w", 1, 2048, 4, 4, 512, 4096, 3000, 1e4)
    a = make_tensor(cfg, "layers.0.wg", seed=42)
    with ThreadPoolExecutor(4) as pool:
        b = make_tensor(cfg, "layers.0.wg", seed=42, pool=pool)
    np.testing.assert_array_equal(a, b)
    c = make_tensor(cfg, "layers.0.wu", seed=42)
    assert not np.array_equal(a, c)
    x = (a.astype(np.uint32) << 16).view(np.float32)
    assert abs(x.std() - 0.02) < 2e-4 and abs(x.mean()) < 2e-4


def test_canonical_order_and_shapes():
    names = [n for n, *_ in canonical_tensors(TINY)]
    assert names[0] == "embed" and names[-2:] == ["final_norm", "lm_head"]
    assert names[1:10] == [f"layers.0.{n}" for n in
                           ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu", "wd")]
    w = make_weights(TINY, threads=2)
    assert w["layers.1.wd"].shape == (TINY.d_model, TINY.ffn_dim)
    assert w["layers.0.wk"].shape == (TINY.kv_dim, TINY.d_model)
    assert np.all(w["final_norm"] == 0x3F80)


def test_bf16_round_to_nearest_even():
    import torch
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 7
    x[:4] = [1.00390625, 1.01171875, -1.00390625, 65504.0]  # exact ties
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(f32_to_bf16_bits(x), ref)


def test_zipf_context_rank_frequency():
    rng = wt.rng_for("context", 0)
    t = wt.zipf_context(rng, 200000, 128256, s=1.1)
    assert t.min() >= 0 and t.max() < 128256
    c = np.bincount(t, minlength=10)
    # P(r=1)/P(r=2) = 2^1.1
    assert abs(c[0] / c[1] - 2 ** 1.1) < 0.1


def test_segment_context_repeats():
    rng = wt.rng_for("context", 1)
    t = wt.segment_context(rng, 16384, 128256)
    assert t.shape == (16384,)
    segs = t.reshape(256, 64)
    # each segment agrees with some other segment on most positions (shared base)
    agree = max(np.mean(segs[0] == segs[j]) for j in range(1, 256))
    assert agree > 0.5


def test_plant_chain():
    rng = wt.rng_for("draft", 0)
    g = np.arange(100, 120)
    for a in range(0, 9):
        d = wt.plant_chain(rng, g, a, 8, 50000)
        assert len(d) == 8
        assert list(d[:a]) == list(g[:a])
        if a < 8:
            assert d[a] != g[a]


def test_acceptance_samplers():
    rng = wt.rng_for("accept", 0)
    geo = [wt.geometric_accept(rng, 0.3, 8) for _ in range(20000)]
    # mean of min(G, 8), G geometric with P(G = n) = 0.3 * 0.7^n
    exact = sum(min(n, 8) * 0.3 * 0.7 ** n for n in range(200))
    assert abs(np.mean(geo) - exact) < 0.05
    bi = [wt.bimodal_accept(rng, 64) for _ in range(4000)]
    assert all(0 <= a <= 2 or 32 <= a <= 64 for a in bi)


def test_eagle_trees_are_breadth_first_and_bounded():
    from workloads import trees
    rng = wt.rng_for("misc", 41)
    for _ in range(200):
        n, depth, topk = int(rng.integers(1, 64)), int(rng.integers(1, 9)), int(rng.integers(1, 5))
        par = trees.eagle_tree(rng, n, depth, topk)
        assert 1 <= len(par) <= n
        assert all(-1 <= p < j for j, p in enumerate(par))
        assert max(len(trees.path_to(par, j)) for j in range(len(par))) <= depth
        assert all(len(k) <= topk * topk for k in trees.children(par).values())


def test_plant_path_gives_the_planted_acceptance_length():
    from workloads import trees
    rng = wt.rng_for("misc", 42)
    for _ in range(200):
        par = trees.eagle_tree(rng, 32, 8, 4)
        greedy = rng.integers(0, 50, size=10)
        a = int(rng.integers(0, 9))
        tok = trees.plant_path(rng, par, greedy, a, 50)
        for p, kids in trees.children(par).items():
            assert len({int(tok[c]) for c in kids}) == len(kids)
        # walk with the greedy continuation standing in for the target
        cur, n = -1, 0
        kids = trees.children(par)
        while True:
            nxt = [c for c in kids.get(cur, []) if tok[c] == greedy[n]]
            if not nxt:
                break
            cur, n = nxt[0], n + 1
        deepest = max(len(trees.path_to(par, j)) for j in range(len(par)))
        assert n == min(a, deepest)


def test_corrupt_stream_replaces_at_rate_p_with_different_tokens():
    rng = wt.rng_for("misc", 7)
    g = wt.uniform_context(rng, 20000, 4096)
    s = wt.corrupt_stream(wt.rng_for("misc", 8), g, 0.3, 4096)
    diff = s != g
    assert abs(diff.mean() - 0.3) < 0.02
    assert s.min() >= 0 and s.max() < 4096
    # runs of kept tokens are geometric: P(run >= 3) = 0.7^3
    starts = np.flatnonzero(diff[:-3])[:2000] + 1
    runs = np.array([np.argmax(diff[i:]) if diff[i:].any() else 0 for i in starts])
    assert abs((runs >= 3).mean() - 0.7 ** 3) < 0.05
    assert (wt.corrupt_stream(wt.rng_for("misc", 8), g, 0.0, 4096) == g).all()
