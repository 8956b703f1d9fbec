"""Seeded plans of the batched workloads: which sequences a verify batch
holds, their context lengths, draft kinds, draft lengths and planted
acceptance targets.  Pure functions of the seeds; no model arithmetic.

* Mixed batch (8B shape): 32 sequences with contexts uniform in [1024, 8192]
  over the paged cache; the first half carry model-drafter chains of k = 8
  with acceptance Geometric(p = 0.4), the second half cache drafts with k
  uniform in [16, 64] and acceptance uniform in [0, k].
* Long multi-step batch (32B shape): 8 sequences at context 8192, 16
  consecutive verify + commit steps, k uniform in {4, ..., 64} and acceptance
  uniform in [0, k] per sequence and step.
"""

from dataclasses import dataclass
from typing import List

from . import tokens as wt


@dataclass(frozen=True)
class SeqPlan:
    seq: int
    ctx_len: int      # context tokens (the last one becomes the pending token)
    kind: str         # "model" (chain from a drafter) or "cache" (copied span)
    k: int
    accept: int       # planted acceptance target


def mixed_batch_plan(n_seqs: int = 32, lo: int = 1024, hi: int = 8192) -> List[SeqPlan]:
    lens = wt.rng_for("batch", 4, 0).integers(lo, hi + 1, size=n_seqs)
    kr = wt.rng_for("batch", 4, 1)
    out = []
    for b in range(n_seqs):
        ar = wt.rng_for("accept", 4, b)
        if b < n_seqs // 2:
            k = 8
            a = wt.geometric_accept(ar, 0.4, k)
            kind = "model"
        else:
            k = int(kr.integers(16, 65))
            a = wt.uniform_accept(ar, k)
            kind = "cache"
        out.append(SeqPlan(b, int(lens[b]), kind, k, a))
    return out


def mixed_batch_context(plan: SeqPlan, vocab: int):
    return wt.zipf_context(wt.rng_for("context", 4, plan.seq), plan.ctx_len, vocab)


def mixed_batch_draft(plan: SeqPlan, context, greedy, vocab: int):
    rng = wt.rng_for("draft", 4, plan.seq)
    if plan.kind == "model":
        return wt.plant_chain(rng, greedy, plan.accept, plan.k, vocab)
    return wt.plant_cache_draft(rng, context, greedy, plan.accept, plan.k, vocab)


def mixed_batch_sampled(plans: List[SeqPlan]) -> List[int]:
    """Sequences checked against the oracle: the shortest and longest context
    of each draft kind (so the batch's minimum and maximum are included)."""
    picks = []
    for kind in ("model", "cache"):
        ps = [p for p in plans if p.kind == kind]
        picks += [min(ps, key=lambda p: (p.ctx_len, p.seq)).seq, max(ps, key=lambda p: (p.ctx_len, -p.seq)).seq]
    return sorted(set(picks))


def multistep_plan(n_seqs: int = 8, n_steps: int = 16) -> List[List[SeqPlan]]:
    """plans[step][seq] for the 16-step batch at context 8192."""
    out = []
    for s in range(n_steps):
        row = []
        for b in range(n_seqs):
            r = wt.rng_for("batch", 5, b, s)
            k = int(r.integers(4, 65))
            row.append(SeqPlan(b, 8192, "cache", k, wt.uniform_accept(r, k)))
        out.append(row)
    return out


def multistep_context(seq: int, n: int, vocab: int):
    return wt.zipf_context(wt.rng_for("context", 5, seq), n, vocab)


def multistep_draft(seq: int, step: int, k: int, accept: int, context, greedy, vocab: int):
    return wt.plant_cache_draft(wt.rng_for("draft", 5, seq, step), context, greedy, accept, k, vocab)
