"""Hybrid Verified Decoding around the verify step (§3.2-3.4, Alg. 1, App. A/B).

Host-side decoding loop: a suffix cache proposes a draft from the prompt and
the committed tokens (§3.2); a payoff predictor g_theta estimates its
accepted length from pre-verification features (§3.3, App. B); the cache
draft is verified when the estimate reaches the threshold tau (6 in App. A),
otherwise the model drafter's proposal is (§3.4).  Verification is the GPU
library's (``KVCache.verify`` / ``verify_tree``); the committed block is
appended, and the cache and the recent-history summary are updated.

Readings where the paper leaves details open (listed with the build notes):
* the cache follows the SuffixDecoding settings of App. A: drafts extend from
  the longest matched suffix (at most 64 tokens) along the most frequent next
  token among the match's occurrences while that token's share is at least
  0.1, for at most min(64, 1.0 x matched length + 0.0) tokens; its score is
  the sum over draft positions of the running product of those shares;
* the features are the App. B groups: suffix score, matched length, draft
  length; prompt length, generated length, relative decode position; recent
  cache-draft selection rate and mean accepted length (last 16 steps); and
  the fraction of draft tokens in five structure classes.  Synthetic token
  ids carry no text, so a token's class comes from a fixed hash of its id;
* g_theta is the App. B MLP (2 hidden layers of 256, ReLU) trained by
  squared error with Adam (learning rate 1e-3, batch 65536, 20 epochs,
  seed 42) on labels replayed from generation traces (App. B);
* without the paper's EAGLE3 checkpoint the model drafter is a callback; the
  default proposes nothing, so low-payoff states take a plain greedy step.

Nothing here computes a forward pass: the target's tokens come from the
verify calls only.
"""

import time
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

MAX_DEPTH = 64          # suffix cache: maximum matched length / tree depth (App. A)
MAX_DRAFT = 64          # maximum draft tokens (App. A)
SPEC_FACTOR = 1.0       # draft length <= factor * matched length + offset (App. A)
SPEC_OFFSET = 0.0
MIN_TOKEN_PROB = 0.1    # stop extending below this continuation share (App. A)
TAU = 6.0               # verify the cache draft when the predicted accepted length >= tau (App. A)
HISTORY = 16            # recent steps summarised in the features
_INDEX_N = 16           # n-gram lengths indexed directly; longer matches are extended by comparison


# ------------------------------------------------------------------ cache

class SuffixCache:
    """Suffix matches over the indexed token streams (warmup traces, the
    prompt, the committed tokens).  Streams are kept separate: a match and
    its continuation never cross from one stream into the next."""

    def __init__(self):
        self.streams: List[List[int]] = []
        self.index: Dict[Tuple[int, ...], List[Tuple[int, int]]] = {}

    def new_stream(self, tokens: Sequence[int] = ()) -> int:
        self.streams.append([])
        sid = len(self.streams) - 1
        self.extend(sid, tokens)
        return sid

    def extend(self, sid: int, tokens: Sequence[int]):
        s = self.streams[sid]
        for t in tokens:
            s.append(int(t))
            end = len(s)  # n-gram s[end-n:end] ends here; its continuation starts at end
            for n in range(1, min(_INDEX_N, end) + 1):
                self.index.setdefault(tuple(s[end - n:end]), []).append((sid, end))

    def _match(self, sid: int):
        """Longest suffix of stream sid (<= MAX_DEPTH tokens) that also ends
        earlier with at least one following token; returns (length, ends)."""
        s = self.streams[sid]
        cur = len(s)
        for n in range(min(_INDEX_N, cur), 0, -1):
            occ = [(q, e) for q, e in self.index.get(tuple(s[cur - n:]), ())
                   if not (q == sid and e == cur) and e < len(self.streams[q])]
            if not occ:
                continue
            if n < _INDEX_N:
                return n, occ
            # extend past the indexed length by direct comparison
            best, keep = n, []
            for q, e in occ:
                t, L = self.streams[q], n
                while L < MAX_DEPTH and L < e and L < cur and t[e - L - 1] == s[cur - L - 1]:
                    L += 1
                if L > best:
                    best, keep = L, [(q, e)]
                elif L == best:
                    keep.append((q, e))
            return best, keep
        return 0, []

    def draft(self, sid: int):
        """Cache draft for the current end of stream sid: (tokens, matched
        length, score)."""
        L, occ = self._match(sid)
        if L == 0:
            return [], 0, 0.0
        limit = int(min(MAX_DRAFT, SPEC_FACTOR * L + SPEC_OFFSET))
        out, score, run = [], 0.0, 1.0
        pos = [(q, e) for q, e in occ]
        while len(out) < limit and pos:
            counts: Dict[int, int] = {}
            recent: Dict[int, int] = {}
            for i, (q, e) in enumerate(pos):
                t = self.streams[q][e]
                counts[t] = counts.get(t, 0) + 1
                recent[t] = i  # later occurrences win ties
            tok = max(counts, key=lambda t: (counts[t], recent[t]))
            share = counts[tok] / len(pos)
            if share < MIN_TOKEN_PROB:
                break
            out.append(tok)
            run *= share
            score += run
            pos = [(q, e + 1) for q, e in pos if self.streams[q][e] == tok and e + 1 < len(self.streams[q])]
        return out, L, score


# --------------------------------------------------------------- features

N_CLASSES = 5  # whitespace, punctuation, line break, bracket, delimiter-like


def token_class(tok: int) -> int:
    """Structure class of a synthetic token id (-1: none).  Ids carry no
    text; a fixed multiplicative hash marks about 1 in 8 ids structural."""
    h = (int(tok) * 2654435761) & 0xFFFFFFFF
    return (h >> 8) % N_CLASSES if (h & 7) == 0 else -1


N_FEATURES = 8 + N_CLASSES


def features(score, matched, draft, prompt_len, generated, max_new, recent_sel, recent_acc) -> np.ndarray:
    """phi_t (App. B feature groups)."""
    cls = np.zeros(N_CLASSES)
    for t in draft:
        c = token_class(t)
        if c >= 0:
            cls[c] += 1
    if draft:
        cls /= len(draft)
    return np.concatenate([[score, np.log1p(matched), np.log1p(len(draft)), np.log1p(prompt_len),
                            np.log1p(generated), generated / max(1, max_new), recent_sel, recent_acc],
                           cls]).astype(np.float32)


# -------------------------------------------------------------- predictor

class PayoffMLP:
    """g_theta: features -> predicted accepted length (App. B: 2 hidden
    layers of 256, ReLU).  Inputs are standardised with the training set's
    mean and deviation."""

    def __init__(self, n_in=N_FEATURES, hidden=256, seed=42):
        rng = np.random.default_rng(seed)
        dims = [n_in, hidden, hidden, 1]
        self.W = [rng.normal(0, np.sqrt(2.0 / a), size=(a, b)).astype(np.float32) for a, b in zip(dims, dims[1:])]
        self.b = [np.zeros(b, np.float32) for b in dims[1:]]
        self.mu = np.zeros(n_in, np.float32)
        self.sd = np.ones(n_in, np.float32)

    def _forward(self, X):
        h = [(X - self.mu) / self.sd]
        for i, (W, b) in enumerate(zip(self.W, self.b)):
            z = h[-1] @ W + b
            h.append(np.maximum(z, 0) if i < len(self.W) - 1 else z)
        return h

    def __call__(self, X) -> np.ndarray:
        return self._forward(np.atleast_2d(np.asarray(X, np.float32)))[-1][:, 0]

    def grads(self, X, y):
        """Sum of squared errors of a batch and the gradients of its mean
        with respect to the weights and biases."""
        h = self._forward(X)
        err = h[-1][:, 0] - y
        g = (2.0 / len(y)) * err[:, None]
        gW, gb = [None] * len(self.W), [None] * len(self.b)
        for i in range(len(self.W) - 1, -1, -1):
            gW[i] = h[i].T @ g
            gb[i] = g.sum(0)
            if i:
                g = (g @ self.W[i].T) * (h[i] > 0)
        return float(np.sum(err * err)), gW, gb

    def fit(self, X, y, lr=1e-3, batch=65536, epochs=20, seed=42):
        """Squared-error regression with Adam; returns the loss per epoch."""
        X = np.asarray(X, np.float32)
        y = np.asarray(y, np.float32)
        self.mu = X.mean(0)
        self.sd = X.std(0) + 1e-6
        params = self.W + self.b
        m = [np.zeros_like(p) for p in params]
        v = [np.zeros_like(p) for p in params]
        b1, b2, eps, step = 0.9, 0.999, 1e-8, 0
        rng = np.random.default_rng(seed)
        losses = []
        for _ in range(epochs):
            order = rng.permutation(len(y))
            tot = 0.0
            for s in range(0, len(y), batch):
                idx = order[s:s + batch]
                sse, gW, gb = self.grads(X[idx], y[idx])
                tot += sse
                step += 1
                for j, (p, gp) in enumerate(zip(params, gW + gb)):
                    m[j] = b1 * m[j] + (1 - b1) * gp
                    v[j] = b2 * v[j] + (1 - b2) * gp * gp
                    p -= lr * (m[j] / (1 - b1 ** step)) / (np.sqrt(v[j] / (1 - b2 ** step)) + eps)
            losses.append(tot / len(y))
        return losses


class StepHistory:
    """The App. B recent-history features over the last HISTORY decoding
    steps: the share of steps that verified the cache draft, and the mean
    accepted length of the cache drafts among them.  The decoding loop and
    the training replay both keep one, so training and inference see the
    same quantity."""

    def __init__(self):
        self.sel: List[float] = []
        self.acc: List[int] = []

    def recent(self):
        s, a = self.sel[-HISTORY:], self.acc[-HISTORY:]
        return (float(np.mean(s)) if s else 0.0, float(np.mean(a)) if a else 0.0)

    def record(self, cache_selected: bool, accepted: int = 0):
        self.sel.append(1.0 if cache_selected else 0.0)
        if cache_selected:
            self.acc.append(int(accepted))


def replay_labels(trace: Sequence[int], prompt_len: int, cache_streams: Sequence[Sequence[int]] = (),
                  max_new: Optional[int] = None, policy: Optional[Callable] = None):
    """Training pairs from a recorded generation (App. B).  The replay walks
    the trace the way the decoding loop would with a verifier that commits
    the trace (the greedy stream) and no model drafter: at each decoding
    state the cache built from the warmup streams and the committed prefix
    proposes d_t, the label is the longest prefix of d_t equal to the
    trace's next tokens, and ``policy(phi) -> bool`` (default: always)
    decides whether the step verifies d_t (committing label + 1 tokens) or
    takes one greedy step.  Features, including the recent-history ones,
    come from the same helpers as in ``HybridVerifiedDecoder.generate``."""
    cache = SuffixCache()
    for s in cache_streams:
        cache.new_stream(s)
    sid = cache.new_stream(trace[:prompt_len])
    max_new = max_new or (len(trace) - prompt_len)
    hist = StepHistory()
    X, y = [], []
    t = prompt_len
    while t < len(trace) and t - prompt_len < max_new:
        generated = t - prompt_len
        room = max_new - generated - 1
        d, L, score = cache.draft(sid)
        d = d[:max(0, min(room, MAX_DRAFT))]
        selected, lab = False, 0
        if d:
            while lab < len(d) and t + lab < len(trace) and d[lab] == trace[t + lab]:
                lab += 1
            phi = features(score, L, d, prompt_len, generated, max_new, *hist.recent())
            X.append(phi)
            y.append(lab)
            selected = True if policy is None else bool(policy(phi))
        z = list(trace[t:t + (lab if selected else 0) + 1])
        hist.record(selected, lab)
        cache.extend(sid, z)
        t += len(z)
    return np.asarray(X, np.float32).reshape(-1, N_FEATURES), np.asarray(y, np.float32)


# ------------------------------------------------------------------- loop

@dataclass
class LoopStats:
    cycles: int = 0                 # verification steps
    generated: int = 0              # committed tokens after the prompt
    cache_steps: int = 0            # steps that verified the cache draft
    cache_accepted: List[int] = field(default_factory=list)
    model_accepted: List[int] = field(default_factory=list)
    decode_s: float = 0.0           # wall time of the decoding loop (after prefill)

    @property
    def cycles_per_1k(self) -> float:
        return 1000.0 * self.cycles / max(1, self.generated)


class HybridVerifiedDecoder:
    """Alg. 1 for one sequence of a KV cache (``verifier`` offers prefill,
    verify, commit and seq_info as ``paper_2606_01019_amd.KVCache``).
    ``model_drafter(tokens) -> draft`` is D_m; None proposes nothing."""

    def __init__(self, verifier, seq_id: int, predictor: Callable, tau: float = TAU,
                 model_drafter: Optional[Callable] = None, warmup_streams: Sequence[Sequence[int]] = ()):
        self.kv = verifier
        self.seq = seq_id
        self.g = predictor
        self.tau = tau
        self.model_drafter = model_drafter
        self.cache = SuffixCache()
        for s in warmup_streams:
            self.cache.new_stream(s)
        self.on_features: Optional[Callable] = None  # observer of each phi_t (tests)

    def generate(self, prompt: Sequence[int], max_new: int, eos: Optional[int] = None):
        prompt = [int(t) for t in prompt]
        self.kv.prefill(self.seq, prompt)
        sid = self.cache.new_stream(prompt)
        x = list(prompt)
        st = LoopStats()
        t0 = time.perf_counter()
        hist = StepHistory()
        max_draft = MAX_DRAFT
        while st.generated < max_new:
            room = max_new - st.generated - 1  # tokens the step may add beyond the next one
            d_c, L, score = self.cache.draft(sid)
            d_c = d_c[:max(0, min(room, max_draft))]
            use_cache = False
            if d_c:
                phi = features(score, L, d_c, len(prompt), st.generated, max_new, *hist.recent())
                if self.on_features is not None:
                    self.on_features(phi)
                use_cache = float(self.g(phi[None, :])[0]) >= self.tau
            if use_cache:
                d = d_c
            else:
                d = list(self.model_drafter(x))[:max(0, room)] if self.model_drafter else []
            ctx, _, _ = self.kv.seq_info(self.seq)
            a, nxt = self.kv.verify([self.seq], [ctx], [np.asarray(d, np.int32)])
            a, nxt = int(a[0]), int(nxt[0])
            self.kv.commit([self.seq])
            z = [int(t) for t in d[:a]] + [nxt]
            x += z
            self.cache.extend(sid, z)
            st.cycles += 1
            st.generated += len(z)
            hist.record(use_cache, a)
            if use_cache:
                st.cache_steps += 1
                st.cache_accepted.append(a)
            elif d:
                st.model_accepted.append(a)
            if eos is not None and eos in z:
                break
        st.decode_s = time.perf_counter() - t0
        return x[len(prompt):len(prompt) + max_new], st
