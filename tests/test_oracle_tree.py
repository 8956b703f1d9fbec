"""Pins of the oracle's tree verification (token-tree drafts of App. A's
model drafter) against independent formulations: hand-built trees, brute
force over every root-to-node path, plain no-cache forwards of each node's
path, and the chain verify it must reduce to.  No GPU."""

import itertools

import numpy as np
import pytest

import oracle
from oracle import model as om
from workloads import ModelConfig, make_weights, tokens as wt, trees

MICRO = ModelConfig("micro", 2, 64, 4, 2, 16, 128, 97, 1.0e4, max_pos=512)


@pytest.fixture(scope="module")
def micro():
    w = make_weights(MICRO, seed=7, gain_std=0.1, threads=1)
    from workloads.weights import f32_to_bf16_bits
    for n, t in list(w.items()):
        if t.ndim == 2:  # larger weights -> larger logit gaps
            w[n] = f32_to_bf16_bits(om.bf16_bits_to_float(t, np.float32) * np.float32(8.0))
    return om.OracleModel(MICRO, w, dtype=np.float64)


def test_depths_and_ancestors_hand_case():
    #        pending
    #        /     \
    #       0       1
    #      / \      |
    #     2   3     4
    #     |
    #     5
    parents = [-1, -1, 0, 0, 1, 2]
    assert oracle.tree_depths(parents).tolist() == [1, 1, 2, 2, 2, 3]
    allowed = oracle.tree_ancestors(parents)
    expect_rows = {0: [0], 1: [0, 1], 2: [0, 2], 3: [0, 1, 3], 4: [0, 1, 4], 5: [0, 2, 5], 6: [0, 1, 3, 6]}
    for r, cols in expect_rows.items():
        assert np.flatnonzero(allowed[r]).tolist() == cols


@pytest.mark.parametrize("g,tokens,parents,expect", [
    ([5, 7, 9, 1, 1, 1, 1], [5, 6, 7, 8, 9, 2], [-1, -1, 0, 0, 1, 2], [0, 2]),      # 5 then 7, then row of node 2 wants 9: no child
    ([6, 1, 8, 1, 1, 1, 1], [5, 6, 7, 8, 9, 2], [-1, -1, 0, 0, 1, 2], [1]),         # second root child; its child 9 != 8
    ([6, 1, 9, 1, 1, 1, 1], [5, 6, 7, 8, 9, 2], [-1, -1, 0, 0, 1, 2], [1, 4]),
    ([4, 1, 1, 1, 1, 1, 1], [5, 6, 7, 8, 9, 2], [-1, -1, 0, 0, 1, 2], []),          # nothing accepted
    ([5, 7, 1, 2, 1, 1, 1], [5, 6, 7, 8, 9, 2], [-1, -1, 0, 0, 1, 2], [0, 2, 5]),   # full depth
    ([3, 4, 5], [3, 4], [-1, 0], [0, 1]),                                            # chain, full acceptance
])
def test_tree_accept_hand_cases(g, tokens, parents, expect):
    assert oracle.tree_accept(np.array(g), np.array(tokens), np.array(parents)) == expect


def _all_paths(parents):
    """Every root-to-node path (lists of node indices), by brute force."""
    out = []
    for j in range(len(parents)):
        p, path = j, []
        while p >= 0:
            path.append(p)
            p = parents[p]
        out.append(path[::-1])
    return out


def test_tree_accept_is_the_longest_accepted_path_brute_force():
    rng = wt.rng_for("misc", 21)
    for trial in range(300):
        parents = trees.eagle_tree(rng, n_nodes=int(rng.integers(1, 40)), depth=int(rng.integers(1, 9)), topk=4)
        n = len(parents)
        V = 6  # tiny vocabulary: many accidental matches
        tokens = trees.distinct_sibling_tokens(rng, parents, V)
        g = rng.integers(0, V, size=n + 1)
        ok = [p for p in _all_paths(parents)
              if all(tokens[p[i]] == g[0 if i == 0 else p[i - 1] + 1] for i in range(len(p)))]
        best = max(ok, key=len) if ok else []
        assert len([p for p in ok if len(p) == len(best)]) <= 1 or not ok  # distinct siblings: unique
        assert oracle.tree_accept(g, tokens, parents) == best


def test_chain_shaped_tree_equals_chain_verify(micro):
    st = oracle.prefill(micro, wt.uniform_context(wt.rng_for("context", 31), 40, MICRO.vocab))
    d = wt.random_chain(wt.rng_for("draft", 31), 7, MICRO.vocab)
    chain = oracle.verify(micro, st, d)
    tree = oracle.verify_tree(micro, st, d, [-1] + list(range(len(d) - 1)))
    assert np.abs(tree.logits - chain.logits).max() < 1e-12
    assert tree.accepted == chain.accepted and tree.next_token == chain.next_token
    assert tree.path == list(range(chain.accepted))


def test_tree_rows_equal_no_cache_forward_of_each_path(micro):
    prompt = wt.uniform_context(wt.rng_for("context", 32), 30, MICRO.vocab)
    st = oracle.prefill(micro, prompt)
    rng = wt.rng_for("draft", 32)
    parents = trees.eagle_tree(rng, n_nodes=12, depth=4, topk=3)
    tokens = trees.distinct_sibling_tokens(rng, parents, MICRO.vocab)
    res = oracle.verify_tree(micro, st, tokens, parents)
    for path in _all_paths(parents):
        toks = list(prompt) + [int(tokens[j]) for j in path]
        logits, _, _ = om.forward(micro, None, None, toks, np.arange(len(toks)))
        assert np.abs(logits[-1] - res.logits[path[-1] + 1]).max() < 1e-9
    # the pending row is the plain next-token prediction
    logits, _, _ = om.forward(micro, None, None, list(prompt), np.arange(len(prompt)))
    assert np.abs(logits[-1] - res.logits[0]).max() < 1e-9


def test_star_tree_rows_are_one_token_verifies(micro):
    st = oracle.prefill(micro, wt.uniform_context(wt.rng_for("context", 33), 25, MICRO.vocab))
    tokens = [3, 17, 40, 88]
    res = oracle.verify_tree(micro, st, tokens, [-1] * len(tokens))
    for j, t in enumerate(tokens):
        one = oracle.verify(micro, st, [t])
        assert np.abs(one.logits[1] - res.logits[j + 1]).max() < 1e-12


def test_tree_commit_equals_chain_commit_of_the_accepted_path(micro):
    prompt = wt.uniform_context(wt.rng_for("context", 34), 35, MICRO.vocab)
    st = oracle.prefill(micro, prompt)
    cont, _ = oracle.greedy_decode(micro, st, 6)
    rng = wt.rng_for("draft", 34)
    parents = trees.eagle_tree(rng, n_nodes=20, depth=6, topk=4)
    tokens = trees.plant_path(rng, parents, cont, accept=4, vocab=MICRO.vocab)
    res = oracle.verify_tree(micro, st, tokens, parents)
    assert res.accepted == 4
    assert res.committed == cont[:5]
    for keep in (0, 2, 4):
        a = oracle.commit_tree(st, res, keep)
        chain = oracle.verify(micro, st, [int(tokens[j]) for j in res.path])
        b = oracle.commit(st, chain, keep)
        assert a.tokens == b.tokens
        for l in range(MICRO.n_layers):
            assert np.abs(a.K[l] - b.K[l]).max() < 1e-12 and np.abs(a.V[l] - b.V[l]).max() < 1e-12
