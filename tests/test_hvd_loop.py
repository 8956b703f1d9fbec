"""Host-side Hybrid Verified Decoding loop (Alg. 1): the suffix cache against
brute force, the App. B label replay, the payoff MLP's training, and
losslessness of the loop with the CPU oracle as the verifier (every
selection policy and drafter must commit exactly the greedy stream).  No
GPU."""

import numpy as np
import pytest

import oracle
from oracle import model as om
from paper_2606_01019_amd import hvd_loop as hl
from workloads import ModelConfig, make_weights, tokens as wt

MICRO = ModelConfig("micro", 2, 64, 4, 2, 16, 128, 97, 1.0e4, max_pos=1024)


def _repetitive(rng, n, vocab, period_choices=(5, 7, 11)):
    """A token stream of repeated random motifs with occasional mutations."""
    out = []
    while len(out) < n:
        motif = rng.integers(0, vocab, size=int(rng.choice(period_choices))).tolist()
        for _ in range(int(rng.integers(2, 6))):
            m = list(motif)
            if rng.random() < 0.3:
                m[int(rng.integers(0, len(m)))] = int(rng.integers(0, vocab))
            out += m
    return out[:n]


def _brute_match(streams, sid):
    s = streams[sid]
    cur = len(s)
    for L in range(min(hl.MAX_DEPTH, cur), 0, -1):
        occ = []
        for q, t in enumerate(streams):
            for e in range(L, len(t)):  # e: end of the occurrence, continuation at t[e]
                if (q, e) != (sid, cur) and t[e - L:e] == s[cur - L:]:
                    occ.append((q, e))
        if occ:
            return L, occ
    return 0, []


def test_suffix_match_equals_brute_force():
    rng = wt.rng_for("misc", 81)
    for trial in range(60):
        cache = hl.SuffixCache()
        streams = [_repetitive(rng, int(rng.integers(20, 200)), 9) for _ in range(int(rng.integers(1, 3)))]
        for s in streams:
            cache.new_stream(s)
        sid = len(streams) - 1
        L, occ = cache._match(sid)
        Lb, occb = _brute_match(cache.streams, sid)
        assert L == Lb
        assert sorted(occ) == sorted(occb)


def _brute_draft(streams, sid):
    L, pos = _brute_match(streams, sid)
    if L == 0:
        return [], 0, 0.0
    limit = int(min(hl.MAX_DRAFT, hl.SPEC_FACTOR * L + hl.SPEC_OFFSET))
    out, score, run = [], 0.0, 1.0
    while len(out) < limit and pos:
        nxt = [streams[q][e] for q, e in pos]
        best = max(set(nxt), key=lambda t: (nxt.count(t), max(i for i, x in enumerate(nxt) if x == t)))
        share = nxt.count(best) / len(nxt)
        if share < hl.MIN_TOKEN_PROB:
            break
        out.append(best)
        run *= share
        score += run
        pos = [(q, e + 1) for q, e in pos if streams[q][e] == best and e + 1 < len(streams[q])]
    return out, L, score


def test_cache_draft_equals_brute_force():
    rng = wt.rng_for("misc", 82)
    for trial in range(60):
        cache = hl.SuffixCache()
        streams = [_repetitive(rng, int(rng.integers(30, 160)), 6) for _ in range(2)]
        for s in streams:
            cache.new_stream(s)
        d, L, score = cache.draft(1)
        db, Lb, sb = _brute_draft(cache.streams, 1)
        assert (d, L) == (db, Lb) and abs(score - sb) < 1e-12
        assert len(d) <= min(hl.MAX_DRAFT, L)


def test_replay_labels_are_longest_agreeing_prefixes():
    rng = wt.rng_for("misc", 83)
    trace = _repetitive(rng, 300, 12)
    X, y = hl.replay_labels(trace, prompt_len=60)
    assert X.shape[1] == hl.N_FEATURES and len(y) == len(X) > 0
    # recompute the labels by brute force along the decoder's walk (every
    # cache draft verified: label + 1 tokens committed, else one token)
    cache = hl.SuffixCache()
    sid = cache.new_stream(trace[:60])
    labels = []
    t, max_new = 60, len(trace) - 60
    while t < len(trace):
        d, _, _ = _brute_draft(cache.streams, sid)
        d = d[:max(0, min(max_new - (t - 60) - 1, hl.MAX_DRAFT))]
        lab = 0
        if d:
            while lab < len(d) and t + lab < len(trace) and d[lab] == trace[t + lab]:
                lab += 1
            labels.append(lab)
        z = trace[t:t + lab + 1]
        cache.extend(sid, z)
        t += len(z)
    assert y.tolist() == labels


def test_payoff_mlp_learns_a_regression():
    rng = np.random.default_rng(0)
    X = rng.normal(size=(4096, hl.N_FEATURES)).astype(np.float32)
    y = (3.0 * X[:, 0] - 2.0 * np.abs(X[:, 1]) + 5.0).astype(np.float32)
    g = hl.PayoffMLP()
    losses = g.fit(X, y, batch=512, epochs=20)
    assert losses[-1] < 0.1 * losses[0]
    assert np.corrcoef(g(X), y)[0, 1] > 0.95


def test_payoff_mlp_gradient_matches_finite_differences():
    """The gradients fit() steps along, against central differences of the
    batch's mean squared error."""
    rng = np.random.default_rng(1)
    X = rng.normal(size=(64, hl.N_FEATURES)).astype(np.float64)
    y = rng.normal(size=64)
    g = hl.PayoffMLP(hidden=8)
    g.W = [w.astype(np.float64) for w in g.W]
    g.b = [b.astype(np.float64) for b in g.b]
    g.mu, g.sd = np.zeros(hl.N_FEATURES), np.ones(hl.N_FEATURES)

    def loss():
        return float(np.mean((g._forward(X)[-1][:, 0] - y) ** 2))

    _, grads, gbias = g.grads(X, y)
    for i in range(len(g.W)):
        for _ in range(5):
            a, b = rng.integers(0, g.W[i].shape[0]), rng.integers(0, g.W[i].shape[1])
            old = g.W[i][a, b]
            g.W[i][a, b] = old + 1e-6
            lp = loss()
            g.W[i][a, b] = old - 1e-6
            lm = loss()
            g.W[i][a, b] = old
            assert abs((lp - lm) / 2e-6 - grads[i][a, b]) < 1e-5 * max(1.0, abs(grads[i][a, b]))
        j = rng.integers(0, g.b[i].shape[0])
        old = g.b[i][j]
        g.b[i][j] = old + 1e-6
        lp = loss()
        g.b[i][j] = old - 1e-6
        lm = loss()
        g.b[i][j] = old
        assert abs((lp - lm) / 2e-6 - gbias[i][j]) < 1e-5 * max(1.0, abs(gbias[i][j]))


class OracleVerifier:
    """The CPU oracle behind the KVCache verify interface."""

    def __init__(self, model):
        self.m = model
        self.st, self.res = {}, {}

    def prefill(self, sid, tokens):
        self.st[sid] = oracle.prefill(self.m, tokens)

    def seq_info(self, sid):
        st = self.st[sid]
        return st.ctx, st.pending, sid in self.res

    def verify(self, ids, ctxs, drafts):
        a, n = [], []
        for sid, c, d in zip(ids, ctxs, drafts):
            assert c == self.st[sid].ctx
            r = oracle.verify(self.m, self.st[sid], d, want_logits=False)
            self.res[sid] = r
            a.append(r.accepted)
            n.append(r.next_token)
        return np.asarray(a), np.asarray(n)

    def commit(self, ids, keep=None):
        for sid in ids:
            self.st[sid] = oracle.commit(self.st[sid], self.res.pop(sid))


@pytest.fixture(scope="module")
def micro():
    w = make_weights(MICRO, seed=3, gain_std=0.1, threads=1)
    return om.OracleModel(MICRO, w, dtype=np.float64)


@pytest.mark.parametrize("policy", ["always", "never", "mlp"])
def test_loop_commits_exactly_the_greedy_stream(micro, policy):
    rng = wt.rng_for("misc", 84)
    prompt = _repetitive(rng, 80, MICRO.vocab)
    n_new = 40
    ref, _ = oracle.greedy_decode(micro, oracle.prefill(micro, prompt), n_new)
    if policy == "mlp":
        g = hl.PayoffMLP()
        X, y = hl.replay_labels(prompt + ref, len(prompt))
        g.fit(X, y, batch=256, epochs=5)
        pred = g
    else:
        pred = (lambda phi: np.full(len(phi), np.inf)) if policy == "always" else (lambda phi: np.full(len(phi), -np.inf))
    drafter = lambda x: wt.random_chain(np.random.default_rng(len(x)), 3, MICRO.vocab)  # a model drafter stand-in
    dec = hl.HybridVerifiedDecoder(OracleVerifier(micro), 0, pred, model_drafter=drafter)
    out, st = dec.generate(prompt, n_new)
    assert out == list(ref)
    assert st.generated >= n_new and st.cycles <= n_new
    if policy == "always":
        assert st.cache_steps > 0


def test_replay_features_equal_the_loops_features(micro):
    """Training features come from the same helpers as inference: replaying
    the loop's own greedy output under the loop's own selection policy
    reproduces every feature vector the loop computed, recent-history
    features included (App. B)."""
    rng = wt.rng_for("misc", 86)
    prompt = _repetitive(rng, 90, MICRO.vocab)
    n_new = 48
    g = hl.PayoffMLP(seed=5)
    X0, y0 = hl.replay_labels(prompt + _repetitive(rng, 60, MICRO.vocab), len(prompt))
    g.fit(X0, y0, batch=64, epochs=3)
    tau = float(np.median(g(X0)))  # a threshold that selects some drafts and rejects others
    seen = []
    dec = hl.HybridVerifiedDecoder(OracleVerifier(micro), 0, g, tau=tau)
    dec.on_features = lambda phi: seen.append(np.array(phi))
    out, st = dec.generate(prompt, n_new)
    assert 0 < st.cache_steps < len(seen)  # both choices occur
    X, y = hl.replay_labels(prompt + out, len(prompt), max_new=n_new,
                            policy=lambda phi: float(g(phi[None, :])[0]) >= tau)
    assert X.shape[0] == len(seen)
    np.testing.assert_array_equal(X, np.stack(seen))
    assert np.any((X[:, 6] > 0) & (X[:, 6] < 1))  # the selection rate varies
