"""Token-tree drafts shaped like the model drafter's (App. A: EAGLE3 with tree
depth 8 and top-k 4), as parent arrays, and token planting along one path.

A tree is a list ``parents``: node j's parent is -1 (the pending token) or an
earlier node, so nodes are in breadth-first order and parents precede their
children.  Nothing here evaluates the model; planting takes the target's
greedy continuation from the caller.
"""

import numpy as np


def eagle_tree(rng, n_nodes: int = 32, depth: int = 8, topk: int = 4):
    """A breadth-first token tree of at most ``n_nodes`` nodes and ``depth``
    levels: each level offers up to ``topk`` children for each of the up to
    ``topk`` nodes kept from the level above, and keeps a random subset (at
    least one) while the node budget lasts."""
    parents = []
    frontier = [-1]
    for _ in range(depth):
        budget = n_nodes - len(parents)
        if budget <= 0 or not frontier:
            break
        offers = [p for p in frontier for _ in range(topk)]
        take = int(rng.integers(1, min(len(offers), budget) + 1))
        chosen = sorted(rng.choice(len(offers), size=take, replace=False).tolist())
        level = []
        for c in chosen:
            level.append(len(parents))
            parents.append(offers[c])
        frontier = level if len(level) <= topk else sorted(rng.choice(level, size=topk, replace=False).tolist())
    return parents


def children(parents):
    kids = {}
    for j, p in enumerate(parents):
        kids.setdefault(int(p), []).append(j)
    return kids


def distinct_sibling_tokens(rng, parents, vocab: int) -> np.ndarray:
    """Uniform tokens, distinct among the children of each node (as a top-k
    expansion produces)."""
    tok = np.zeros(len(parents), dtype=np.int64)
    for p, kids in children(parents).items():
        tok[kids] = rng.choice(vocab, size=len(kids), replace=False)
    return tok


def path_to(parents, j):
    """Node indices from the root's child down to node j."""
    out = []
    while j >= 0:
        out.append(j)
        j = int(parents[j])
    return out[::-1]


def plant_path(rng, parents, greedy, accept: int, vocab: int) -> np.ndarray:
    """Tokens for ``parents`` such that the accepted path has exactly
    ``accept`` nodes when the target's greedy continuation is ``greedy``
    (greedy[i] = the target's token after i accepted tokens): a deepest path
    is chosen, its first ``accept`` nodes carry greedy[0..accept-1], and no
    other child of an accepted row carries that row's greedy token."""
    tok = distinct_sibling_tokens(rng, parents, vocab)
    deep = max(range(len(parents)), key=lambda j: (len(path_to(parents, j)), -j)) if parents else -1
    path = path_to(parents, deep) if deep >= 0 else []
    accept = min(accept, len(path))
    kids = children(parents)
    for i in range(accept + 1):
        parent = -1 if i == 0 else path[i - 1]
        want = int(greedy[i])
        on_path = path[i] if i < accept else -1
        for c in kids.get(parent, []):
            if c == on_path:
                continue
            if tok[c] == want:  # move it to a token unused among its siblings
                used = {int(tok[s]) for s in kids[parent]} | {want}
                tok[c] = next(t for t in rng.permutation(vocab).tolist() if t not in used)
        if on_path >= 0:  # siblings no longer hold `want` (moved above)
            tok[on_path] = want
    return tok
