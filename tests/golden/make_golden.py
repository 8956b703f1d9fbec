"""Write the oracle's expected values for the full-size parity tests.

Calls only oracle/ and workloads/ (never the GPU library).  For each case the
script regenerates the seeded weights and context, prefills the oracle,
computes the oracle's greedy continuation, plants drafts with the stated
acceptance, runs the oracle's verify and stores a compact record: drafts,
accepted length, next token, per-row argmax and top-2 margin, and logits at a
fixed sample of vocabulary ids plus each row's top-8 ids.

The 8B- and 32B-shaped references use the oracle in float32 (the float64
path of the same code would need twice the memory and time); a reduced-depth
pin (tests/test_oracle_precision.py) bounds the float32/float64 difference.

Usage: python tests/golden/make_golden.py cfg2 [cfg3 cfg4 cfg5]
"""

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from oracle.model import OracleModel  # noqa: E402
from workloads import SHAPE_8B, SHAPE_32B, make_weights, tokens as wt  # noqa: E402

N_SAMPLE = 64
TOP = 8


def log(*a):
    print(time.strftime("%H:%M:%S"), *a, flush=True)


def sample_ids(vocab):
    return np.sort(wt.rng_for("misc", 99).choice(vocab, size=N_SAMPLE, replace=False)).astype(int)


def record(res, ids):
    lg = res.logits
    part = np.partition(lg, -2, axis=-1)
    top = np.argsort(-lg, axis=-1)[:, :TOP]
    return {
        "draft": [int(t) for t in res.draft],
        "accepted": int(res.accepted),
        "next": int(res.next_token),
        "argmax": [int(t) for t in res.argmax],
        "margin": [float(x) for x in (part[:, -1] - part[:, -2])],
        "sample_logits": [[float(x) for x in row] for row in lg[:, ids]],
        "top_ids": [[int(t) for t in row] for row in top],
        "top_logits": [[float(lg[r, t]) for t in top[r]] for r in range(lg.shape[0])],
    }


def fp32_model(cfg, seed=42):
    """float32 oracle whose converted weights are cached (bf16 copies dropped)."""
    w = make_weights(cfg, seed=seed)

    m = OracleModel(cfg, w, dtype=np.float32, cache=True)
    for n in list(w.keys()):
        m.w(n)          # convert once, keep the float32 copy
        w[n] = None     # free the bf16 copy
    return m


def greedy(m, st, n):
    out, _ = oracle.greedy_decode(m, st, n)
    return out


def case_cfg2():
    cfg = SHAPE_8B
    log("cfg2: weights")
    m = fp32_model(cfg)
    ctx = wt.zipf_context(wt.rng_for("context", 2), 2048, cfg.vocab)
    log("cfg2: prefill")
    st = oracle.prefill(m, ctx)
    ids = sample_ids(cfg.vocab)
    arng = wt.rng_for("accept", 20)
    ks = [1, 2, 4, 8, 16]
    plans = [wt.geometric_accept(arng, 0.3, k) for k in ks]
    log("cfg2: greedy continuation")
    g = greedy(m, st, max(a + 1 for a in plans) + 1)
    drng = wt.rng_for("draft", 20)
    steps = []
    for k, a in zip(ks, plans):
        d = wt.plant_chain(drng, g, a, k, cfg.vocab)
        res = oracle.verify(m, st, d)
        log(f"cfg2: k={k} planted={a} accepted={res.accepted}")
        steps.append(record(res, ids))
    return {"config": "8B shape, batch 1, context 2048 Zipf(1.1), chain drafts k in 1,2,4,8,16 planted "
                      "geometric(p=0.3) from the oracle's greedy continuation",
            "model": cfg.as_dict(), "context_seed": ["context", 2], "context_len": 2048,
            "context_kind": "zipf", "sample_ids": [int(i) for i in ids], "steps": steps,
            "oracle_dtype": "float32"}


def case_cfg3():
    cfg = SHAPE_8B
    log("cfg3: weights")
    m = fp32_model(cfg)
    ctx = wt.segment_context(wt.rng_for("context", 3), 16384, cfg.vocab)
    log("cfg3: prefill")
    st = oracle.prefill(m, ctx)
    ids = sample_ids(cfg.vocab)
    arng = wt.rng_for("accept", 30)
    ks = [32, 48, 64]
    plans = [wt.bimodal_accept(arng, k) for k in ks]
    log(f"cfg3: greedy continuation for plans {plans}")
    g = greedy(m, st, max(a + 1 for a in plans) + 1)
    drng = wt.rng_for("draft", 30)
    steps = []
    for k, a in zip(ks, plans):
        d = wt.plant_cache_draft(drng, ctx, g, a, k, cfg.vocab)
        res = oracle.verify(m, st, d)
        log(f"cfg3: k={k} planted={a} accepted={res.accepted}")
        steps.append(record(res, ids))
    return {"config": "8B shape, batch 1, context 16384 built from 64-token segments (16 base segments, 20% "
                      "per-token mutation), cache drafts k in 32,48,64 planted bimodal from the oracle's greedy "
                      "continuation, tail copied from an earlier context span",
            "model": cfg.as_dict(), "context_seed": ["context", 3], "context_len": 16384,
            "context_kind": "segments", "sample_ids": [int(i) for i in ids], "steps": steps,
            "oracle_dtype": "float32"}


def main():
    cases = {"cfg2": case_cfg2, "cfg3": case_cfg3}
    for name in sys.argv[1:]:
        t0 = time.time()
        out = cases[name]()
        path = os.path.join(HERE, f"{name}.json")
        with open(path, "w") as f:
            json.dump(out, f, separators=(",", ":"))
        log(f"{name}: wrote {path} in {time.time() - t0:.0f}s")


if __name__ == "__main__":
    main()
