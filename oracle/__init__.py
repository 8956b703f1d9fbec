"""CPU oracle for the target-model verification step of Hybrid Verified Decoding.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import or run anything in this
package.  The GPU library never calls it and shares no code with it.

What it computes (Verify in §3.1 and §3.4, Alg. 1 "Verify" step): one forward
of the unchanged target model over the pending token plus a chain draft, the
greedy accepted length (the longest draft prefix equal to the target's argmax
continuation, the same quantity as the label equation of §3.3 and App. B),
and the committed block of accepted tokens plus one target token; the same
rule over a token tree (the tree-shaped model drafts of App. A), where each
node sees its own path and the accepted path follows the target's argmax.  At
temperature 0 (App. A generation table) greedy speculative verification is
lossless, so the oracle is the plain definition: a Llama-style decoder forward
in float64 (or float32 on request) over bf16-valued weights, and the prefix
match written out.

Parity pins (tests/test_oracle_*.py): brute-force no-cache greedy decoding,
the k = 0 greedy step, full acceptance of the oracle's own greedy
continuation, planted mismatches, causality, rotary-embedding invariants,
textbook softmax attention, Hkv = Hq, a library cross-check against
``transformers.LlamaForCausalLM``, hand-built accept cases and the
cycles-per-1K identity printed in the paper's App. C and Table 4.
"""

from .model import (  # noqa: F401
    OracleModel,
    SeqState,
    VerifyResult,
    TreeVerifyResult,
    accept_length,
    argmax_lowest,
    brute_force_greedy,
    commit,
    commit_tree,
    greedy_decode,
    prefill,
    tree_accept,
    tree_ancestors,
    tree_depths,
    verify,
    verify_tree,
)
