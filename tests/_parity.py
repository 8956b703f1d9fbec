"""Shared helpers of the GPU parity tests (not collected by pytest).

The tolerance comes from the verify step's own statement of parity: logits
within max-abs 2e-2 of the oracle; argmax, accepted length and next token
identical except at rows whose oracle top-2 logit margin is below 2e-2
(near ties, where either answer is correct); such rows are counted and
reported, never silently accepted elsewhere.
"""

import numpy as np

LOGIT_TOL = 2e-2
TIE_MARGIN = 2e-2


def top2_margin(logits):
    part = np.partition(np.asarray(logits, dtype=np.float64), -2, axis=-1)
    return part[..., -1] - part[..., -2]


def accept_from_argmax(g, d):
    """Accepted length implied by a row-argmax vector (used to check the GPU's
    own consistency, not to decide parity)."""
    a = 0
    while a < len(d) and int(d[a]) == int(g[a]):
        a += 1
    return a


class Report:
    def __init__(self):
        self.max_err = 0.0
        self.rows = 0
        self.excused = 0
        self.excused_diff = 0

    def __str__(self):
        return (f"max|dlogit|={self.max_err:.3e} rows={self.rows} near-tie rows={self.excused} "
                f"(argmax differs on {self.excused_diff})")


def check_step(rep: Report, res, gpu_logits, a_gpu, next_gpu, draft, tol=LOGIT_TOL):
    """Compare one sequence's verify against the oracle result ``res``.

    Returns True when a near tie on the accepted path made the GPU and oracle
    take different branches (the caller then re-syncs the oracle)."""
    d = np.asarray(draft)
    k = len(d)
    ref = res.logits
    if gpu_logits is not None:
        err = float(np.max(np.abs(gpu_logits.astype(np.float64) - ref)))
        rep.max_err = max(rep.max_err, err)
        assert err <= tol, f"logit error {err:.3e} > {tol}"
    margin = top2_margin(ref)
    g_ref = res.argmax
    rep.rows += k + 1
    excused = margin < TIE_MARGIN
    rep.excused += int(excused.sum())
    if gpu_logits is not None:
        g_gpu = np.argmax(gpu_logits, axis=-1)
        bad = (g_gpu != g_ref) & ~excused
        assert not bad.any(), f"argmax differs at non-tie rows {np.flatnonzero(bad)}"
        rep.excused_diff += int(((g_gpu != g_ref) & excused).sum())
        # the GPU's own acceptance follows its own argmax exactly
        assert a_gpu == accept_from_argmax(g_gpu, d)
        assert next_gpu == int(g_gpu[a_gpu])
    # rows on the oracle's accepted path decide a and next; if none is a near
    # tie, the results must be identical
    path = excused[:min(res.accepted, a_gpu) + 1]
    if not path.any():
        assert a_gpu == res.accepted, (a_gpu, res.accepted)
        assert next_gpu == res.next_token, (next_gpu, res.next_token)
        return False
    return (a_gpu != res.accepted) or (next_gpu != res.next_token)


def oracle_commit_as(st, res, a_gpu, next_gpu):
    """Commit the GPU's block on the oracle side (re-sync after a near tie):
    keep a_gpu draft tokens (their K/V rows are in res) and make next_gpu the
    pending token."""
    from oracle.model import SeqState
    import numpy as _np
    n_rows = a_gpu + 1
    K = [_np.concatenate([st.K[l], nk[:n_rows]]) if st.K and st.K[l] is not None else nk[:n_rows]
         for l, nk in enumerate(res.new_k)]
    V = [_np.concatenate([st.V[l], nv[:n_rows]]) if st.V and st.V[l] is not None else nv[:n_rows]
         for l, nv in enumerate(res.new_v)]
    toks = list(st.tokens) + [int(t) for t in res.draft[:a_gpu]] + [int(next_gpu)]
    return SeqState(tokens=toks, K=K, V=V)


def check_golden(rep: Report, L, rec, sample_ids, a_gpu, next_gpu, tol=LOGIT_TOL, tie_margin=TIE_MARGIN):
    """Compare one sequence's GPU verify (logit rows L [k+1, V]) with a stored
    oracle record (tests/golden/*.json): logits at the sampled ids and at each
    row's oracle top ids, per-row argmax except near ties, accepted length
    and next token unless a near tie lies on the accepted path.

    Returns True when the GPU took another branch at a near tie (the caller
    stops following the oracle's trajectory for that sequence)."""
    k = len(rec["draft"])
    assert L.shape[0] == k + 1
    ids = np.asarray(sample_ids)
    err = float(np.abs(L[:, ids] - np.asarray(rec["sample_logits"])).max())
    top_ids = np.asarray(rec["top_ids"])
    err_top = max(float(np.abs(L[r, top_ids[r]] - np.asarray(rec["top_logits"][r])).max()) for r in range(k + 1))
    err = max(err, err_top)
    rep.max_err = max(rep.max_err, err)
    assert err <= tol, f"logit error {err:.3e} > {tol}"
    margin = np.asarray(rec["margin"])
    tie = margin < tie_margin
    rep.rows += k + 1
    rep.excused += int(tie.sum())
    g_gpu = L.argmax(axis=1)
    g_ref = np.asarray(rec["argmax"])
    bad = (g_gpu != g_ref) & ~tie
    assert not bad.any(), f"argmax differs at non-tie rows {np.flatnonzero(bad)}"
    rep.excused_diff += int(((g_gpu != g_ref) & tie).sum())
    assert a_gpu == accept_from_argmax(g_gpu, rec["draft"]) and next_gpu == int(g_gpu[a_gpu])
    if not tie[:min(rec["accepted"], a_gpu) + 1].any():
        assert a_gpu == rec["accepted"] and next_gpu == rec["next"], (a_gpu, rec["accepted"], next_gpu, rec["next"])
        return False
    return a_gpu != rec["accepted"] or next_gpu != rec["next"]


def load_whole_rows(name):
    """Whole oracle logit rows stored beside a record (tests/golden/<name>,
    written by make_golden.py): {key: float64 rows}, or None when absent.
    Values are int16 multiples of the stored step (|quantisation| <= step/2)."""
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", name)
    if not os.path.exists(path):
        return None
    z = np.load(path)
    step = float(z["step"])
    return {k: z[k].astype(np.float64) * step for k in z.files if k != "step"}, step


def check_whole_rows(L, stored, step, tol=LOGIT_TOL):
    """Rows 0 and k of one verify (L [k+1, V]) against the oracle's whole
    rows; returns the max abs difference (asserted <= tol + step/2)."""
    k = L.shape[0] - 1
    got = np.asarray(L, dtype=np.float64)[[0, k]]
    assert got.shape == stored.shape, (got.shape, stored.shape)
    err = float(np.abs(got - stored).max())
    assert err <= tol + step / 2, f"whole-row logit error {err:.3e} > {tol}"
    return err
