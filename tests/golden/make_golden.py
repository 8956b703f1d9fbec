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

Usage: python tests/golden/make_golden.py cfg2 [cfg3 cfg4 cfg5 tree2 cfg5_full] [--spill DIR]
       python tests/golden/make_golden.py rows_cfg2 [rows_cfg3 rows_cfg4 rows64_cfg2] --spill DIR
(the rows_ passes add whole logit rows to an existing record, rows64_ the
float64 oracle's rows; see case_rows_8b)
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
from workloads import SHAPE_8B, SHAPE_32B, batches, make_weights, tokens as wt  # noqa: E402

N_SAMPLE = 64
TOP = 8


def log(*a):
    print(time.strftime("%H:%M:%S"), *a, flush=True)


def sample_ids(vocab):
    return np.sort(wt.rng_for("misc", 99).choice(vocab, size=N_SAMPLE, replace=False)).astype(int)


def record(res, ids, top_n=TOP):
    lg = res.logits
    part = np.partition(lg, -2, axis=-1)
    top = np.argsort(-lg, axis=-1)[:, :top_n]
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


def case_cfg4():
    """Mixed batch: the oracle verifies the sampled sequences one by one (a
    batched verify is per-sequence by construction)."""
    cfg = SHAPE_8B
    plans = batches.mixed_batch_plan()
    picks = batches.mixed_batch_sampled(plans)
    log("cfg4: weights")
    m = fp32_model(cfg)
    ids = sample_ids(cfg.vocab)
    seqs = []
    for b in picks:
        p = plans[b]
        ctx = batches.mixed_batch_context(p, cfg.vocab)
        log(f"cfg4: seq {b} prefill {p.ctx_len}")
        st = oracle.prefill(m, ctx)
        g = greedy(m, st, p.accept + 1)
        d = batches.mixed_batch_draft(p, ctx, g, cfg.vocab)
        res = oracle.verify(m, st, d)
        log(f"cfg4: seq {b} ({p.kind}, k={p.k}) planted={p.accept} accepted={res.accepted}")
        rec = record(res, ids)
        rec["seq"] = b
        seqs.append(rec)
    return {"config": "8B shape, 32 sequences with contexts uniform in [1024, 8192] (Zipf tokens); sequences "
                      "0-15 model chains k=8 planted geometric(p=0.4), 16-31 cache drafts k in [16, 64] planted "
                      "uniform in [0, k]; the oracle checks the shortest and longest context of each kind",
            "model": cfg.as_dict(), "sample_ids": [int(i) for i in ids], "sampled": picks, "seqs": seqs,
            "oracle_dtype": "float32"}


CFG5_LAYERS = 4
CFG5_SEQS = (0, 1)


def case_cfg5():
    """32B-shaped widths at reduced depth: two of the eight sequences over the
    16 verify + commit steps (commit keeps the oracle's accepted prefix)."""
    cfg = SHAPE_32B.with_layers(CFG5_LAYERS)
    plans = batches.multistep_plan()
    log("cfg5: weights")
    m = fp32_model(cfg)
    ids = sample_ids(cfg.vocab)[:16]
    out = []
    for b in CFG5_SEQS:
        ctx = batches.multistep_context(b, 8192, cfg.vocab)
        log(f"cfg5: seq {b} prefill")
        st = oracle.prefill(m, ctx)
        steps = []
        for s_, row in enumerate(plans):
            p = row[b]
            g = greedy(m, st, p.accept + 1)
            d = batches.multistep_draft(b, s_, p.k, p.accept, ctx, g, cfg.vocab)
            res = oracle.verify(m, st, d)
            rec = record(res, ids, top_n=4)
            steps.append(rec)
            st = oracle.commit(st, res, res.accepted)
            log(f"cfg5: seq {b} step {s_} k={p.k} planted={p.accept} accepted={res.accepted}")
        out.append({"seq": b, "steps": steps})
    return {"config": "32B widths (64 q / 8 kv heads of 128, SwiGLU 27648, vocab 152064) at 4 layers; 8 "
                      "sequences at context 8192 (Zipf tokens), 16 verify + commit steps with k uniform in "
                      "{4..64} and cache drafts planted uniform in [0, k]; sequences 0 and 1 checked",
            "model": cfg.as_dict(), "n_layers": CFG5_LAYERS, "sample_ids": [int(i) for i in ids],
            "seqs": out, "oracle_dtype": "float32"}


def record_tree(res, ids, top_n=TOP):
    lg = res.logits
    part = np.partition(lg, -2, axis=-1)
    top = np.argsort(-lg, axis=-1)[:, :top_n]
    return {
        "tokens": [int(t) for t in res.tokens],
        "parents": [int(p) for p in res.parents],
        "path": [int(j) for j in res.path],
        "next": int(res.next_token),
        "argmax": [int(t) for t in res.argmax],
        "margin": [float(x) for x in (part[:, -1] - part[:, -2])],
        "sample_logits": [[float(x) for x in row] for row in lg[:, ids]],
        "top_ids": [[int(t) for t in row] for row in top],
        "top_logits": [[float(lg[r, t]) for t in top[r]] for r in range(lg.shape[0])],
    }


def case_tree2():
    """Token trees on the workload-2 context: EAGLE-shaped trees (32 nodes,
    depth 8, top-k 4) with 2, 5 and 8 tokens planted along a deepest path,
    and a 63-node 4-ary tree with 3 planted."""
    from workloads import trees
    cfg = SHAPE_8B
    log("tree2: weights")
    m = fp32_model(cfg)
    ctx = wt.zipf_context(wt.rng_for("context", 2), 2048, cfg.vocab)
    log("tree2: prefill")
    st = oracle.prefill(m, ctx)
    ids = sample_ids(cfg.vocab)
    g = greedy(m, st, 9)
    rng = wt.rng_for("draft", 22)
    shapes = [(trees.eagle_tree(rng, 32, 8, 4), 2), (trees.eagle_tree(rng, 32, 8, 4), 5),
              (trees.eagle_tree(rng, 32, 8, 4), 8), ([-1] + [j // 4 for j in range(62)], 3)]
    steps = []
    for par, a in shapes:
        tok = trees.plant_path(rng, par, g, a, cfg.vocab)
        res = oracle.verify_tree(m, st, tok, par)
        log(f"tree2: {len(par)} nodes planted={a} accepted={res.accepted}")
        steps.append(record_tree(res, ids))
    return {"config": "8B shape, batch 1, context 2048 Zipf(1.1) (workload 2), token trees: three EAGLE-shaped "
                      "(32 nodes, depth 8, top-k 4) with 2, 5, 8 tokens planted along a deepest path from the "
                      "oracle's greedy continuation, and a 63-node 4-ary tree with 3 planted",
            "model": cfg.as_dict(), "context_seed": ["context", 2], "context_len": 2048,
            "context_kind": "zipf", "sample_ids": [int(i) for i in ids], "steps": steps,
            "oracle_dtype": "float32"}


# ---------------------------------------------------------------- full depth

FULL_ROW_STEP = 2.0 ** -11  # logits stored as int16 multiples of this (|error| <= 2.5e-4)


def quantize_rows(rows):
    """Full logit rows stored compactly: int16 multiples of FULL_ROW_STEP
    (range +-16; the script refuses logits outside it)."""
    rows = np.asarray(rows, dtype=np.float64)
    assert np.abs(rows).max() < 32767 * FULL_ROW_STEP, "logit outside the stored range"
    return np.round(rows / FULL_ROW_STEP).astype(np.int16)


class SpillStore:
    """Canonical tensors (bf16 bits) of a model too large for the host's
    memory: the norms, embedding, LM head and the first ``resident`` layers
    stay in memory; the other layers' matrices go once to raw files in
    ``spill_dir`` and are read back on every use (or, without a directory,
    are re-drawn from their seeds on every use)."""

    def __init__(self, cfg, resident, spill_dir=None, seed=42):
        from concurrent.futures import ThreadPoolExecutor
        from workloads.weights import canonical_tensors, default_threads, make_tensor
        self.cfg, self.seed, self.spill_dir = cfg, seed, spill_dir
        self.mem, self.files = {}, {}
        self._make = make_tensor
        self._pool = ThreadPoolExecutor(max_workers=default_threads())
        for name, shape, layer, kind in canonical_tensors(cfg):
            if layer < resident or kind == "norm":
                self.mem[name] = make_tensor(cfg, name, seed=seed, pool=self._pool)
                continue
            if spill_dir is None:
                self.files[name] = (None, shape)
                continue
            path = os.path.join(spill_dir, f"{cfg.name}.{name}.bf16")
            nbytes = int(np.prod(shape)) * 2
            if not (os.path.exists(path) and os.path.getsize(path) == nbytes):
                make_tensor(cfg, name, seed=seed, pool=self._pool).tofile(path + ".tmp")
                os.replace(path + ".tmp", path)
            self.files[name] = (path, shape)
        log(f"{cfg.name}: {len(self.mem)} tensors in memory, {len(self.files)} streamed")

    def __getitem__(self, name):
        if name in self.mem:
            return self.mem[name]
        path, shape = self.files[name]
        if path is None:
            return self._make(self.cfg, name, seed=self.seed, pool=self._pool)
        return np.fromfile(path, dtype=np.uint16).reshape(shape)

    def keys(self):
        return list(self.mem) + list(self.files)


def _save_progress(ckpt, b, st, steps, rows):
    tmp = f"{ckpt}/cfg5f_seq{b}"
    np.save(tmp + "_K.npy.tmp.npy", np.stack(st.K))
    np.save(tmp + "_V.npy.tmp.npy", np.stack(st.V))
    np.savez(tmp + "_rows.tmp.npz", **rows)
    with open(tmp + ".json.tmp", "w") as f:
        json.dump({"tokens": [int(t) for t in st.tokens], "steps": steps}, f)
    os.replace(tmp + "_K.npy.tmp.npy", tmp + "_K.npy")
    os.replace(tmp + "_V.npy.tmp.npy", tmp + "_V.npy")
    os.replace(tmp + "_rows.tmp.npz", tmp + "_rows.npz")
    os.replace(tmp + ".json.tmp", tmp + ".json")


def _load_progress(ckpt, b):
    from oracle.model import SeqState
    base = f"{ckpt}/cfg5f_seq{b}"
    if ckpt is None or not os.path.exists(base + ".json"):
        return None
    with open(base + ".json") as f:
        meta = json.load(f)
    K, V = np.load(base + "_K.npy"), np.load(base + "_V.npy")
    rows = dict(np.load(base + "_rows.npz"))
    st = SeqState(tokens=meta["tokens"], K=[K[l] for l in range(K.shape[0])], V=[V[l] for l in range(V.shape[0])])
    return st, meta["steps"], rows


CFG5F_SEQS = (0, 1)


def case_cfg5_full(spill=None, n_steps=4, resident=38):
    """Workload 5 at its full depth (64 layers of the 32B shape): sequences 0
    and 1 over the first n_steps verify + commit steps, from a float32
    oracle that streams the weights (oracle/streamed.py).  Besides the
    compact record, rows 0 and k of every verify are kept whole (int16
    multiples of FULL_ROW_STEP) in cfg5_full_rows.npz."""
    from oracle.streamed import StreamedOracleModel
    cfg = SHAPE_32B
    plans = batches.multistep_plan()
    store = SpillStore(cfg, resident, spill)
    m = StreamedOracleModel(cfg, store)
    ids = sample_ids(cfg.vocab)
    out, all_rows = [], {}
    for b in CFG5F_SEQS:
        ctx = batches.multistep_context(b, 8192, cfg.vocab)
        got = _load_progress(spill, b)
        if got is None:
            log(f"cfg5_full: seq {b} prefill")
            st = oracle.prefill(m, ctx, row_block=8192)
            steps, rows = [], {}
            if spill:
                _save_progress(spill, b, st, steps, rows)
        else:
            st, steps, rows = got
            log(f"cfg5_full: seq {b} resumed after {len(steps)} steps")
        for s_ in range(len(steps), n_steps):
            p = plans[s_][b]
            t0 = time.time()
            g = greedy(m, st, p.accept + 1)
            d = batches.multistep_draft(b, s_, p.k, p.accept, ctx, g, cfg.vocab)
            res = oracle.verify(m, st, d)
            steps.append(record(res, ids, top_n=4))
            rows[f"seq{b}_step{s_}"] = quantize_rows(res.logits[[0, len(d)]])
            st = oracle.commit(st, res, res.accepted)
            log(f"cfg5_full: seq {b} step {s_} k={p.k} planted={p.accept} accepted={res.accepted} "
                f"({time.time() - t0:.0f}s)")
            if spill:
                _save_progress(spill, b, st, steps, rows)
        out.append({"seq": b, "steps": steps})
        all_rows.update(rows)
        del st
    np.savez_compressed(os.path.join(HERE, "cfg5_full_rows.npz"), step=np.float64(FULL_ROW_STEP), **all_rows)
    return {"config": "32B shape at full depth (64 layers, 64 q / 8 kv heads of 128, SwiGLU 27648, vocab 152064); "
                      "8 sequences at context 8192 (Zipf tokens), verify + commit steps with k uniform in {4..64} "
                      "and cache drafts planted uniform in [0, k]; sequences 0 and 1 checked over the first "
                      f"{n_steps} steps; rows 0 and k of every verify stored whole in cfg5_full_rows.npz",
            "model": cfg.as_dict(), "n_layers": cfg.n_layers, "n_steps": n_steps,
            "sample_ids": [int(i) for i in ids], "seqs": out, "oracle_dtype": "float32 (bf16 weights streamed)",
            "full_rows": "cfg5_full_rows.npz", "full_row_step": FULL_ROW_STEP}


def _rows_8b_verifies(name):
    """(key, context, draft, stored step record) of every verify of an 8B
    record whose rows 0 and k are kept whole."""
    cfg = SHAPE_8B
    with open(os.path.join(HERE, f"{name}.json")) as f:
        gold = json.load(f)
    if name in ("cfg2", "cfg3"):
        make = wt.zipf_context if gold["context_kind"] == "zipf" else wt.segment_context
        ctx = make(wt.rng_for(*gold["context_seed"]), gold["context_len"], cfg.vocab)
        return gold, [(f"step{i}", ctx, st) for i, st in enumerate(gold["steps"])]
    assert name == "cfg4"
    plans = batches.mixed_batch_plan()
    return gold, [(f"seq{r['seq']}", batches.mixed_batch_context(plans[r["seq"]], cfg.vocab), r)
                  for r in gold["seqs"]]


def case_rows_8b(name, spill=None, dtype=np.float32):
    """Whole logit rows for an existing 8B record (cfg2, cfg3 or cfg4): the
    oracle with streamed bf16 weights re-runs the verify of every stored draft
    on the same context and keeps rows 0 and k whole (int16 multiples of
    FULL_ROW_STEP).  In float32 (oracle/streamed.py; <name>_rows.npz) the
    re-run must reproduce the stored record: sampled logits within 2e-3 (the
    two float32 oracles differ only in summation order) and the same argmax,
    accepted length and next token away from near ties.  In float64 (the
    plain OracleModel widening each streamed matrix; <name>_rows_f64.npz)
    nothing is asserted: tests/test_oracle_precision.py bounds the float32
    drift at full depth from the two files."""
    from oracle.streamed import StreamedOracleModel
    cfg = SHAPE_8B
    f64 = np.dtype(dtype) == np.float64
    gold, items = _rows_8b_verifies(name)
    ids = np.asarray(gold["sample_ids"])
    store = SpillStore(cfg, 0, spill)
    m = OracleModel(cfg, store, dtype=np.float64, cache=False) if f64 else StreamedOracleModel(cfg, store)
    rows, worst, last_ctx, st = {}, 0.0, None, None
    for key, ctx, rec in items:
        if ctx is not last_ctx:
            log(f"rows {name}: {key} prefill {len(ctx)}")
            st = oracle.prefill(m, ctx)
            last_ctx = ctx
        d = np.asarray(rec["draft"], dtype=np.int64)
        res = oracle.verify(m, st, d)
        dev = float(np.abs(res.logits[:, ids] - np.asarray(rec["sample_logits"])).max())
        worst = max(worst, dev)
        if not f64:
            assert dev <= 2e-3, f"{name} {key}: re-run differs from the stored record by {dev:.2e}"
            clear = np.asarray(rec["margin"]) >= 2e-3
            assert np.array_equal(np.asarray(res.argmax)[clear], np.asarray(rec["argmax"])[clear]), key
            if clear[:rec["accepted"] + 1].all():
                assert res.accepted == rec["accepted"] and res.next_token == rec["next"], key
        rows[key] = quantize_rows(res.logits[[0, len(d)]])
        log(f"rows {name}: {key} k={len(d)} accepted={res.accepted} re-run vs record {dev:.2e}")
    out = f"{name}_rows_f64.npz" if f64 else f"{name}_rows.npz"
    np.savez_compressed(os.path.join(HERE, out), step=np.float64(FULL_ROW_STEP), **rows)
    log(f"rows {name}: wrote {out} ({len(rows)} verifies), worst re-run vs record {worst:.2e}")


def main():
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("cases", nargs="+")
    ap.add_argument("--spill", default=None, help="directory for streamed weights and resume state (cfg5_full)")
    ap.add_argument("--steps", type=int, default=4, help="verify + commit steps of cfg5_full")
    ap.add_argument("--resident", type=int, default=38, help="32B layers held in memory (cfg5_full)")
    args = ap.parse_args()
    cases = {"cfg2": case_cfg2, "cfg3": case_cfg3, "cfg4": case_cfg4, "cfg5": case_cfg5, "tree2": case_tree2,
             "cfg5_full": lambda: case_cfg5_full(args.spill, args.steps, args.resident)}
    for name in args.cases:
        if name.startswith("rows_") or name.startswith("rows64_"):  # whole rows of an existing record
            tag, rec = name.split("_", 1)
            case_rows_8b(rec, args.spill, np.float64 if tag == "rows64" else np.float32)
            continue
        t0 = time.time()
        out = cases[name]()
        path = os.path.join(HERE, f"{name}.json")
        with open(path, "w") as f:
            json.dump(out, f, separators=(",", ":"))
        log(f"{name}: wrote {path} in {time.time() - t0:.0f}s")


if __name__ == "__main__":
    main()
