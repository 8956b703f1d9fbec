"""Plain CPU definition of the verification step (test infrastructure only).

Each function states the passage of the paper it follows.  The paper fixes the
verification interface and acceptance rule but not the target architecture; the
architecture below is the Llama-style decoder the workloads use, written as its
textbook definition.  Readings of points the paper leaves open:

* the committed block is always the accepted tokens plus one target token
  (also on full acceptance, where that token is the bonus), which the
  cycles-per-1K identity of App. C / Table 4 pins;
* the forward covers k + 1 rows: the pending (last committed, not yet cached)
  token followed by the k draft tokens; k = 0 is one greedy step;
* argmax ties go to the lowest token id;
* RMSNorm eps and the rotary base come from the model config; rotary uses the
  rotate-half pairing (j, j + dh/2) with angle p * theta^(-2j/dh) at 0-based
  absolute position p; no biases, no QK-norm, untied LM head; q-head h reads
  kv-head floor(h / (Hq / Hkv)).

Nothing here is blocked, fused or reordered beyond processing query rows in
groups during prefill, which leaves every row's arithmetic unchanged.
"""

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np


def bf16_bits_to_float(u16, dtype=np.float64) -> np.ndarray:
    """bf16 bit pattern -> float (exact widening)."""
    u = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(dtype)


class OracleModel:
    """Target model M: config plus a mapping from canonical tensor names to
    bf16 bit arrays ([out, in] row-major for matrices)."""

    def __init__(self, cfg, weights, dtype=np.float64, cache: bool = True):
        self.cfg = cfg
        self.weights = weights
        self.dtype = np.dtype(dtype)
        self.cache = cache
        self._conv = {}

    def w(self, name: str) -> np.ndarray:
        if name in self._conv:
            return self._conv[name]
        arr = bf16_bits_to_float(self.weights[name], self.dtype)
        if self.cache:
            self._conv[name] = arr
        return arr

    def linear(self, h: np.ndarray, name: str) -> np.ndarray:
        """h @ W^T for the [out, in] weight ``name`` (a plain matrix product)."""
        return h @ self.w(name).T


# ------------------------------------------------------------------ layers

def rms_norm(x, g, eps):
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rotary(x, pos, theta):
    """Rotate-half rotary embedding of x [n, H, dh] at positions pos [n]."""
    dh = x.shape[-1]
    half = dh // 2
    inv_freq = float(theta) ** (-(2.0 * np.arange(half, dtype=np.float64)) / dh)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    cos = np.cos(ang).astype(x.dtype)[:, None, :]
    sin = np.sin(ang).astype(x.dtype)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def softmax_rows(s):
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attend(q, K, V, q_pos):
    """Causal grouped-query attention.  q [n, Hq, dh]; K, V [T, Hkv, dh] hold
    positions 0..T-1; row i attends to key positions j <= q_pos[i]."""
    n, Hq, dh = q.shape
    T, Hkv, _ = K.shape
    group = Hq // Hkv
    j = np.arange(T)
    allowed = j[None, :] <= np.asarray(q_pos)[:, None]
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(dh)
    for h in range(Hq):
        g = h // group
        s = (q[:, h, :] @ K[:, g, :].T) * scale
        s = np.where(allowed, s, -np.inf)
        out[:, h, :] = softmax_rows(s) @ V[:, g, :]
    return out


def silu(z):
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def forward(model: OracleModel, K_cache, V_cache, tokens, positions, want_logits=True):
    """Decoder forward of rows ``tokens`` at ``positions`` over cached K/V.

    K_cache[l], V_cache[l]: [ctx, Hkv, dh] for positions 0..ctx-1 (None = empty);
    positions must be ctx, ctx+1, ....  Returns (logits [n, V] or None,
    new K rows per layer, new V rows per layer).
    """
    c = model.cfg
    dt = model.dtype
    tokens = np.asarray(tokens, dtype=np.int64)
    positions = np.asarray(positions, dtype=np.int64)
    n = tokens.shape[0]
    x = model.w("embed")[tokens] if model.cache else bf16_bits_to_float(
        np.asarray(model.weights["embed"])[tokens], dt)
    new_k, new_v = [], []
    for l in range(c.n_layers):
        p = f"layers.{l}."
        h = rms_norm(x, model.w(p + "attn_norm"), c.rms_eps)
        q = model.linear(h, p + "wq").reshape(n, c.n_q_heads, c.head_dim)
        k = model.linear(h, p + "wk").reshape(n, c.n_kv_heads, c.head_dim)
        v = model.linear(h, p + "wv").reshape(n, c.n_kv_heads, c.head_dim)
        q = rotary(q, positions, c.rope_theta)
        k = rotary(k, positions, c.rope_theta)
        Kc = k if K_cache is None or K_cache[l] is None else np.concatenate([K_cache[l], k], axis=0)
        Vc = v if V_cache is None or V_cache[l] is None else np.concatenate([V_cache[l], v], axis=0)
        o = attend(q, Kc, Vc, positions).reshape(n, c.q_dim)
        x = x + model.linear(o, p + "wo")
        h2 = rms_norm(x, model.w(p + "mlp_norm"), c.rms_eps)
        a = silu(model.linear(h2, p + "wg")) * model.linear(h2, p + "wu")
        x = x + model.linear(a, p + "wd")
        new_k.append(k)
        new_v.append(v)
    logits = None
    if want_logits:
        logits = model.linear(rms_norm(x, model.w("final_norm"), c.rms_eps), "lm_head")
    return logits, new_k, new_v


# ------------------------------------------------------- verification rule

def argmax_lowest(logits) -> np.ndarray:
    """Row-wise argmax; np.argmax returns the first (lowest-index) maximum."""
    return np.argmax(np.asarray(logits), axis=-1).astype(np.int64)


def accept_length(g, d) -> int:
    """Accepted length (label equation of §3.3 / App. B): the largest l in
    {0..k} such that the draft prefix d[0:l] equals the target continuation.
    Row i of the verify forward predicts the token after draft prefix d[0:i],
    so the target continuation token compared with d[i] is g[i]."""
    k = len(d)
    best = 0
    for l in range(k + 1):
        if all(int(d[j]) == int(g[j]) for j in range(l)):
            best = l
    return best


@dataclass
class SeqState:
    """Committed prefix x_{1:t} of one sequence (§3.1).  tokens includes the
    pending token tokens[-1], whose K/V is not cached yet; ctx = len - 1."""
    tokens: List[int]
    K: list = field(default_factory=list)
    V: list = field(default_factory=list)

    @property
    def ctx(self) -> int:
        return len(self.tokens) - 1

    @property
    def pending(self) -> int:
        return self.tokens[-1]


@dataclass
class VerifyResult:
    """(a_t, z_t) = Verify(x_{1:t}, d_t; M) of §3.1, plus the per-row argmax,
    the logits and the tentative K/V rows needed by commit."""
    accepted: int
    next_token: int
    draft: np.ndarray
    argmax: np.ndarray
    logits: Optional[np.ndarray]
    new_k: list
    new_v: list

    @property
    def committed(self) -> List[int]:
        """z_t: the accepted draft prefix followed by one target token."""
        return [int(t) for t in self.draft[:self.accepted]] + [int(self.next_token)]


def prefill(model: OracleModel, prompt, row_block: int = 2048) -> SeqState:
    """Cache K/V of prompt[0..n-2]; the last prompt token becomes pending."""
    prompt = [int(t) for t in prompt]
    assert len(prompt) >= 1
    c = model.cfg
    st = SeqState(tokens=list(prompt))
    K = [None] * c.n_layers
    V = [None] * c.n_layers
    body = np.asarray(prompt[:-1], dtype=np.int64)
    for s in range(0, body.shape[0], row_block):
        rows = body[s:s + row_block]
        _, nk, nv = forward(model, K, V, rows, np.arange(s, s + rows.shape[0]), want_logits=False)
        K = [nk[l] if K[l] is None else np.concatenate([K[l], nk[l]]) for l in range(c.n_layers)]
        V = [nv[l] if V[l] is None else np.concatenate([V[l], nv[l]]) for l in range(c.n_layers)]
    st.K, st.V = K, V
    return st


def verify(model: OracleModel, st: SeqState, draft, want_logits: bool = True) -> VerifyResult:
    """One verification step: forward the pending token and the draft at
    positions ctx..ctx+k, take the argmax of every row, and apply the accept
    rule (§3.1 Verify; §3.4; Alg. 1 Verify step)."""
    d = np.asarray(draft, dtype=np.int64).reshape(-1)
    rows = np.concatenate([[st.pending], d]).astype(np.int64)
    pos = np.arange(st.ctx, st.ctx + rows.shape[0])
    logits, nk, nv = forward(model, st.K if st.ctx else None, st.V if st.ctx else None, rows, pos)
    g = argmax_lowest(logits)
    a = accept_length(g, d)
    return VerifyResult(a, int(g[a]), d, g, logits if want_logits else None, nk, nv)


def commit(st: SeqState, res: VerifyResult, keep: Optional[int] = None) -> SeqState:
    """Append the committed block (Alg. 1: append z to x).  keep <= a draft
    tokens are kept (default a); the K/V of the pending row and the kept draft
    rows enter the cache, the rest is discarded."""
    keep = res.accepted if keep is None else int(keep)
    assert 0 <= keep <= res.accepted
    n_rows = keep + 1
    K = [nk[:n_rows] if (st.K is None or not st.K or st.K[l] is None)
         else np.concatenate([st.K[l], nk[:n_rows]]) for l, nk in enumerate(res.new_k)]
    V = [nv[:n_rows] if (st.V is None or not st.V or st.V[l] is None)
         else np.concatenate([st.V[l], nv[:n_rows]]) for l, nv in enumerate(res.new_v)]
    toks = list(st.tokens) + [int(t) for t in res.draft[:keep]] + [int(res.argmax[keep])]
    return SeqState(tokens=toks, K=K, V=V)


def greedy_decode(model: OracleModel, st: SeqState, n: int):
    """n plain greedy steps (verify with an empty draft, commit).  Returns the
    generated tokens and the final state."""
    out = []
    for _ in range(n):
        r = verify(model, st, [], want_logits=False)
        st = commit(st, r)
        out.append(r.next_token)
    return out, st


def brute_force_greedy(model: OracleModel, tokens, n: int):
    """Greedy decoding without any cache: recompute the whole forward over the
    full token list for every new token.  Returns (new tokens, last-row logits
    of every step)."""
    toks = [int(t) for t in tokens]
    out, rows = [], []
    for _ in range(n):
        logits, _, _ = forward(model, None, None, toks, np.arange(len(toks)))
        last = logits[-1]
        nxt = int(argmax_lowest(last[None, :])[0])
        out.append(nxt)
        rows.append(last)
        toks.append(nxt)
    return out, np.stack(rows)


# ------------------------------------------- tree-shaped drafts (App. A)
#
# The model drafter of App. A (EAGLE3, tree depth 8, top-k 4) proposes a
# token tree rather than a chain.  Verification is the same rule applied
# along the tree: every node is a draft token whose parent is the pending
# token or an earlier node; a node's row sees the cached context and the rows
# on its own path from the pending token, at position ctx + depth; the
# accepted path starts at the pending token and repeatedly moves to the child
# whose token equals the target's argmax of the current row.  With a chain
# (every node's parent the node before it) this is exactly `verify`.

def tree_depths(parents) -> np.ndarray:
    """Depth of each node: 1 for children of the pending token (parent -1),
    else 1 + the parent's depth.  Parents must precede their children."""
    par = [int(p) for p in parents]
    dep = np.zeros(len(par), dtype=np.int64)
    for j, p in enumerate(par):
        assert -1 <= p < j, "a node's parent is the pending token or an earlier node"
        dep[j] = 1 if p < 0 else dep[p] + 1
    return dep


def tree_ancestors(parents) -> np.ndarray:
    """allowed[i, j] over the rows [pending] + nodes: row j is row i itself or
    one of its ancestors (row 0, the pending token, is every row's root)."""
    n = len(parents)
    allowed = np.zeros((n + 1, n + 1), dtype=bool)
    allowed[0, 0] = True
    for j, p in enumerate(parents):
        r = j + 1
        allowed[r] = allowed[int(p) + 1]
        allowed[r, r] = True
    return allowed


def attend_masked(q, K, V, allowed):
    """Grouped-query attention with an explicit mask allowed [n, T] over the
    key rows of K, V [T, Hkv, dh]."""
    n, Hq, dh = q.shape
    group = Hq // K.shape[1]
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(dh)
    for h in range(Hq):
        g = h // group
        s = (q[:, h, :] @ K[:, g, :].T) * scale
        s = np.where(allowed, s, -np.inf)
        out[:, h, :] = softmax_rows(s) @ V[:, g, :]
    return out


def forward_tree(model: OracleModel, K_cache, V_cache, tokens, positions, row_allowed):
    """Decoder forward of rows ``tokens`` at ``positions`` over cached K/V of
    ctx positions; row i sees every cached position and the new rows j with
    row_allowed[i, j].  Same layer arithmetic as `forward`."""
    c = model.cfg
    tokens = np.asarray(tokens, dtype=np.int64)
    positions = np.asarray(positions, dtype=np.int64)
    n = tokens.shape[0]
    ctx = 0 if K_cache is None or K_cache[0] is None else K_cache[0].shape[0]
    allowed = np.concatenate([np.ones((n, ctx), dtype=bool), np.asarray(row_allowed, dtype=bool)], axis=1)
    x = model.w("embed")[tokens] if model.cache else bf16_bits_to_float(
        np.asarray(model.weights["embed"])[tokens], model.dtype)
    new_k, new_v = [], []
    for l in range(c.n_layers):
        p = f"layers.{l}."
        h = rms_norm(x, model.w(p + "attn_norm"), c.rms_eps)
        q = model.linear(h, p + "wq").reshape(n, c.n_q_heads, c.head_dim)
        k = model.linear(h, p + "wk").reshape(n, c.n_kv_heads, c.head_dim)
        v = model.linear(h, p + "wv").reshape(n, c.n_kv_heads, c.head_dim)
        q = rotary(q, positions, c.rope_theta)
        k = rotary(k, positions, c.rope_theta)
        Kc = k if ctx == 0 else np.concatenate([K_cache[l], k], axis=0)
        Vc = v if ctx == 0 else np.concatenate([V_cache[l], v], axis=0)
        o = attend_masked(q, Kc, Vc, allowed).reshape(n, c.q_dim)
        x = x + model.linear(o, p + "wo")
        h2 = rms_norm(x, model.w(p + "mlp_norm"), c.rms_eps)
        a = silu(model.linear(h2, p + "wg")) * model.linear(h2, p + "wu")
        x = x + model.linear(a, p + "wd")
        new_k.append(k)
        new_v.append(v)
    logits = model.linear(rms_norm(x, model.w("final_norm"), c.rms_eps), "lm_head")
    return logits, new_k, new_v


def tree_accept(g, tokens, parents):
    """The verification rule along a tree: from the pending token (row 0),
    move to the child whose token equals the argmax of the current row
    (lowest node index if several), until none does.  Returns the accepted
    node indices in order; their count is the accepted length a."""
    path, cur = [], -1
    while True:
        want = int(g[cur + 1])
        nxt = next((j for j, p in enumerate(parents) if int(p) == cur and int(tokens[j]) == want), None)
        if nxt is None:
            return path
        path.append(nxt)
        cur = nxt


@dataclass
class TreeVerifyResult:
    """Verify of a token tree: accepted node path, its length a, next token
    (argmax of the last accepted row), per-row argmax and logits (row 0 =
    pending, row j+1 = node j), and the tentative K/V rows."""
    path: List[int]
    next_token: int
    tokens: np.ndarray
    parents: np.ndarray
    argmax: np.ndarray
    logits: np.ndarray
    new_k: list
    new_v: list

    @property
    def accepted(self) -> int:
        return len(self.path)

    @property
    def committed(self) -> List[int]:
        return [int(self.tokens[j]) for j in self.path] + [int(self.next_token)]


def verify_tree(model: OracleModel, st: SeqState, tokens, parents) -> TreeVerifyResult:
    """One verification step over a token tree: forward the pending token
    and every node (node at position ctx + depth, seeing its own path), take
    each row's argmax and walk the accepted path."""
    tok = np.asarray(tokens, dtype=np.int64).reshape(-1)
    par = np.asarray(parents, dtype=np.int64).reshape(-1)
    assert tok.shape == par.shape
    dep = tree_depths(par)
    rows = np.concatenate([[st.pending], tok]).astype(np.int64)
    pos = st.ctx + np.concatenate([[0], dep])
    logits, nk, nv = forward_tree(model, st.K if st.ctx else None, st.V if st.ctx else None, rows, pos,
                                  tree_ancestors(par))
    g = argmax_lowest(logits)
    path = tree_accept(g, tok, par)
    last = 0 if not path else path[-1] + 1
    return TreeVerifyResult(path, int(g[last]), tok, par, g, logits, nk, nv)


def commit_tree(st: SeqState, res: TreeVerifyResult, keep: Optional[int] = None) -> SeqState:
    """Append the committed block of a tree verify: the pending row and the
    first ``keep`` (default a) accepted nodes enter the cache in path order
    (their positions are ctx, ctx + 1, ...), the rest is discarded."""
    keep = res.accepted if keep is None else int(keep)
    assert 0 <= keep <= res.accepted
    rows = [0] + [j + 1 for j in res.path[:keep]]
    K = [nk[rows] if (not st.K or st.K[l] is None) else np.concatenate([st.K[l], nk[rows]])
         for l, nk in enumerate(res.new_k)]
    V = [nv[rows] if (not st.V or st.V[l] is None) else np.concatenate([st.V[l], nv[rows]])
         for l, nv in enumerate(res.new_v)]
    last = rows[-1]
    toks = list(st.tokens) + [int(res.tokens[j]) for j in res.path[:keep]] + [int(res.argmax[last])]
    return SeqState(tokens=toks, K=K, V=V)
