/*
 * hvd.h -- C ABI of the target-model verification step of Hybrid Verified
 * Decoding (arxiv 2606.01019) on one AMD Instinct MI355X (gfx950).
 *
 * The paper's interface (section 3.1, "Verified Drafting as a Common
 * Interface"; section 3.4 and Alg. 1, Verify step) is
 *     (a_t, z_t) = Verify(x_{1:t}, d_t; M)
 * for a prefix x_{1:t}, a chain draft d_t of k tokens and the unchanged target
 * model M: a_t in {0..k} is the number of accepted draft tokens and z_t, the
 * committed block, is the accepted draft prefix followed by one target token
 * (the correction token when the draft is rejected early, the bonus token when
 * all k are accepted).  Alg. 1 then appends z_t to the prefix.
 *
 * Under greedy decoding (temperature 0, App. A generation table) the target
 * token after the accepted prefix is the argmax of the model's logits, and the
 * accepted length is the longest draft prefix that equals the target's own
 * argmax continuation (the label equation of section 3.3 / App. B).
 *
 * Model: Llama-style decoder (RMSNorm, rotary embedding with rotate-half
 * pairing, grouped-query attention, SwiGLU MLP, untied LM head), bf16 weights.
 * The KV cache holds fp16 (the paper's data type, App. A) in 16-token pages.
 *
 * The paper defines only Verify and the commit of its block (Alg. 1).  The
 * other calls -- model loading, KV cache creation, prefill, truncate,
 * sequence free, the device-resident loop, options, profiling and
 * diagnostics -- are this library's own plumbing around them.
 *
 * Conventions for every call:
 *  - Host pointers (const T* / T*) are owned by the caller and read or written
 *    only during the call.  "device" pointers point to GPU memory.
 *  - A borrowed device buffer (dev_buf != NULL) stays owned by the caller; it
 *    must outlive the handle and is never freed by the library.  With
 *    dev_buf == NULL the library allocates (hipMalloc) and frees the memory.
 *  - Work is queued on the HIP stream given at load/alloc time (the caller's
 *    torch stream), and every call returns only after its results are in host
 *    memory (synchronous).  A handle is not thread-safe.
 *  - Every call returns an hvd_status.  On any error the library state is left
 *    unchanged (no partial page allocation, no partial commit) and
 *    hvd_last_error() describes the failure.
 */
#ifndef HVD_H
#define HVD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HVD_OK = 0,
  HVD_ERR_ARG = -1,    /* bad pointer/size, unknown or duplicate seq id, keep > accepted */
  HVD_ERR_STATE = -2,  /* ctx_lens disagree with the library, verify pending, commit without verify */
  HVD_ERR_OOM = -3,    /* page pool or row workspace cannot hold the request (checked before any work) */
  HVD_ERR_RANGE = -4,  /* token outside [0, vocab), draft length outside [0, max_draft], position >= max_pos */
  HVD_ERR_DEVICE = -5  /* a HIP runtime error; message in hvd_last_error() */
} hvd_status;

/* Model shape.  Requirements (HVD_ERR_ARG otherwise): d_model % 64 == 0,
 * ffn_dim % 32 == 0, vocab % 64 == 0, head_dim in {64, 128},
 * n_q_heads % n_kv_heads == 0, page_size == 16, 0 <= max_draft <= 64,
 * max_pos >= 32. */
typedef struct {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t ffn_dim;
  int32_t vocab;
  int32_t max_draft;   /* longest chain draft hvd_verify accepts */
  int32_t page_size;   /* tokens per KV page (16) */
  int32_t max_pos;     /* rotary table length: every position must be < max_pos */
  float rope_theta;
  float rms_eps;
} hvd_config;

typedef struct hvd_model_s* hvd_model;
typedef struct hvd_kv_s* hvd_kv;

/* Device bytes needed by hvd_model_load for this config (packed weights,
 * gains, rotary table). */
size_t hvd_model_bytes(const hvd_config* cfg);

/* Upload and pack the weights.  tensors[i] are host bf16 bit patterns
 * (uint16) in canonical order, each row-major with torch Linear layout
 * [out_features, in_features]:
 *   embed [V, D];
 *   for each layer: attn_norm [D], wq [Hq*dh, D], wk [Hkv*dh, D],
 *     wv [Hkv*dh, D], wo [D, Hq*dh], mlp_norm [D], wg [F, D], wu [F, D],
 *     wd [D, F];
 *   final_norm [D], lm_head [V, D].
 * Count = 3 + 9 * n_layers.  Matrices are stored on the device as fp16
 * (exact for every bf16 value of magnitude >= 2^-17; smaller ones round with
 * an error below 2^-25), the embedding and gains as given.
 * dev_buf (nullable) must hold hvd_model_bytes.
 * stream is a hipStream_t (NULL = default stream).  Temporary staging memory
 * is allocated and freed inside the call. */
hvd_status hvd_model_load(const hvd_config* cfg, const uint16_t* const* tensors, void* dev_buf,
                          size_t dev_bytes, void* stream, hvd_model* out);
void hvd_model_free(hvd_model m);

/* Device bytes for a KV pool of n_pages pages plus the per-step workspace for
 * up to max_seqs sequences verified together. */
size_t hvd_kv_bytes(const hvd_config* cfg, int32_t max_seqs, int32_t n_pages);

/* Create a KV cache bound to model m.  Sequence ids are 0..max_seqs-1.
 * dev_buf (nullable) must hold hvd_kv_bytes.  Work of this handle runs on
 * stream (hipStream_t, NULL = default stream). */
hvd_status hvd_kv_alloc(hvd_model m, int32_t max_seqs, int32_t n_pages, void* dev_buf,
                        size_t dev_bytes, void* stream, hvd_kv* out);
void hvd_kv_free(hvd_kv kv);

/* Start sequence seq_id from a prompt of n >= 1 tokens: caches K/V of
 * tokens[0..n-2] (positions 0..n-2) and makes tokens[n-1] the pending token,
 * so ctx_len = n - 1.  No logits are produced.  seq_id must be free. */
hvd_status hvd_prefill(hvd_model m, hvd_kv kv, int32_t seq_id, const int32_t* tokens, int32_t n);

/* One verification step for `batch` distinct sequences (section 3.1 Verify).
 * Sequence b (id seq_ids[b], current length ctx_lens[b], which must equal the
 * library's) contributes k_b = draft_lens[b] draft tokens, packed in
 * draft_tokens in batch order (sum k_b entries).  One forward covers, for each
 * b, the pending token and the draft at positions ctx_b..ctx_b+k_b.
 * Outputs (host, [batch]): accepted_len[b] = a_b in [0, k_b]; next_token[b] =
 * the target's argmax after the accepted prefix (lowest id on ties).  The
 * committed block is draft[0:a_b] followed by next_token[b].
 * logits (nullable, DEVICE pointer) receives fp32 logits [sum(k_b+1)][vocab],
 * rows packed by sequence -- for parity checks only (extra HBM writes).
 * K/V of all k_b + 1 rows is written tentatively; hvd_commit decides how many
 * stay.  A second verify of a sequence before its commit is HVD_ERR_STATE. */
hvd_status hvd_verify(hvd_model m, hvd_kv kv, int32_t batch, const int32_t* seq_ids,
                      const int32_t* ctx_lens, const int32_t* draft_tokens, const int32_t* draft_lens,
                      int32_t* accepted_len, int32_t* next_token, float* logits);

/* hvd_verify for callers that cannot allocate device memory (tight serving
 * loops, harnesses that forbid hipMalloc after set-up): same arguments,
 * results and errors as hvd_verify, but the step's scratch (split-K partial
 * tiles, attention split-KV partials, LM-head argmax partials, per-row
 * argmax, the results block and the accept kernel's arrival counter) lives
 * in a static device array of 64 MiB that each GPU the library runs on holds
 * until the process ends, instead of the KV handle's workspace.  The call
 * makes no hipMalloc / hipFree and creates no HIP graph or event (kernels are
 * launched one by one; profiling is suspended for the call).  A step whose
 * fixed scratch (about rows * vocab / 2 bytes of LM-head partials plus 8 MiB)
 * does not fit is refused with HVD_ERR_RANGE before any state changes; one
 * whose attention partials do not fit the rest is HVD_ERR_OOM.  All calls on
 * one GPU share that GPU's array, which keeps the last call's contents: calls
 * that overlap on one GPU (two host threads, or two streams) race. */
hvd_status hvd_verify_noalloc(hvd_model m, hvd_kv kv, int32_t batch, const int32_t* seq_ids,
                              const int32_t* ctx_lens, const int32_t* draft_tokens, const int32_t* draft_lens,
                              int32_t* accepted_len, int32_t* next_token, float* logits);

/* One verification step over token trees (the tree-shaped drafts of the
 * model drafter, App. A: EAGLE3 with tree depth 8 and top-k 4), under the
 * same rule: for sequence b, node_counts[b] = n_b <= 63 nodes, packed in
 * batch order in node_tokens and node_parents (sum n_b entries each).  Node
 * j's parent is node_parents[j] = -1 (the pending token) or an earlier node
 * of the same tree (< j).  One forward covers the pending token (rotary
 * position ctx_b) and every node (rotary position ctx_b + depth, depth 1 for
 * children of the pending token); each row attends to the cached context
 * and to the rows on its own path.  The accepted path starts at the pending
 * token and moves to the child whose token is the target's argmax of the
 * current row (the lowest node index if several), while one exists.
 * Outputs (host): accepted_len[b] = a_b, the path length; next_token[b] =
 * the argmax of the path's last row; accepted_nodes (nullable, [batch][63])
 * receives the path's node indices in order.  The K/V of the path is moved
 * to positions ctx_b + 1 .. ctx_b + a_b before the call returns, so
 * hvd_commit keeps a prefix of the path exactly as for a chain draft (the
 * pending token after keep < a_b is the token of path node keep).  logits
 * (nullable, DEVICE) receives fp32 logits [sum(n_b + 1)][vocab], row 0 of
 * each sequence the pending token, row j + 1 node j.  Errors as hvd_verify;
 * a node count outside [0, 63] is HVD_ERR_RANGE, a parent that is not -1 or
 * an earlier node HVD_ERR_ARG. */
hvd_status hvd_verify_tree(hvd_model m, hvd_kv kv, int32_t batch, const int32_t* seq_ids,
                           const int32_t* ctx_lens, const int32_t* node_tokens, const int32_t* node_parents,
                           const int32_t* node_counts, int32_t* accepted_len, int32_t* next_token,
                           int32_t* accepted_nodes, float* logits);

/* Commit the last verify of each listed sequence (Alg. 1: append z_t).
 * keep_lens (nullable = the accepted lengths) keeps 0 <= keep <= a_b draft
 * tokens: ctx_len += keep + 1 and the new pending token is the target's argmax
 * after draft[0:keep] (which equals draft[keep] when keep < a_b).  K/V rows of
 * the rejected suffix are dropped by metadata only; pages wholly past the new
 * end return to the pool. */
hvd_status hvd_commit(hvd_model m, hvd_kv kv, int32_t batch, const int32_t* seq_ids,
                      const int32_t* keep_lens);

/* Device-resident verify loop: Alg. 1's Verify followed by the commit of
 * the whole accepted block (append z_t with keep = a_t), repeated on the GPU
 * with the drafts read from device memory and no host round trip per step.
 * Each step is one replay of a HIP graph captured here, so a drafter running
 * on the GPU (writing `drafts` on the same stream between steps) can feed
 * verification directly, and the host only enqueues.
 *
 * hvd_async_begin opens a loop of at most max_steps >= 1 steps over `batch`
 * sequences with fixed draft lengths draft_lens[b] in [0, max_draft]
 * (ctx_lens as in hvd_verify).  It reserves the pages of the longest
 * possible outcome, ctx_b + max_steps * (k_b + 1) + 1 positions
 * (HVD_ERR_OOM if the pool cannot; HVD_ERR_RANGE past the rotary table), and
 * while the loop is open every other call on these sequences is
 * HVD_ERR_STATE.  The model and KV handles must outlive the loop.
 * Caller-owned DEVICE buffers (int32, kept alive until hvd_async_end):
 *   drafts  [sum k_b]   draft tokens of step s, packed in batch order; read
 *                       by every step (may be NULL when every k_b = 0).  A
 *                       token outside [0, vocab) is never accepted.
 *   state   [2 batch + 1]  ctx[b], pending token[b], steps done; written
 *                       here, then advanced by every step on the device.
 *   history [max_steps][batch][2]  (accepted a_b, next token) of each step.
 * Copy drafter (optional, the cache drafts of section 3.2 in their simplest
 * device form): with ref_tokens (DEVICE, [batch][ref_len]) non-NULL, each
 * step first fills sequence b's drafts with the stream tokens at positions
 * ctx_b + 1 .. ctx_b + k_b, where ref_tokens[b][j] stands at position
 * ref_start[b] + j (ref_start: host, [batch]) and positions outside the
 * stream give -1; the drafts buffer then receives them too.
 * hvd_async_step enqueues n_steps >= 0 steps and returns without waiting
 * (HVD_ERR_RANGE past max_steps in total).  hvd_async_end waits for them,
 * takes ctx and the pending token from `state` into the library's sequence
 * state, releases the pages past each new end and frees the loop (also on
 * error: then the sequences keep their state from before the loop).
 * steps_done (nullable) receives the number of steps run.  The results
 * equal those of hvd_verify + hvd_commit with the same drafts, up to the
 * rounding of attention sums split at other chunk boundaries. */
typedef struct hvd_async_s* hvd_async;
hvd_status hvd_async_begin(hvd_model m, hvd_kv kv, int32_t batch, const int32_t* seq_ids,
                           const int32_t* ctx_lens, const int32_t* draft_lens, int32_t max_steps,
                           int32_t* drafts, int32_t* state, int32_t* history, const int32_t* ref_tokens,
                           int32_t ref_len, const int32_t* ref_start, hvd_async* out);
hvd_status hvd_async_step(hvd_async loop, int32_t n_steps);
hvd_status hvd_async_end(hvd_async loop, int32_t* steps_done);

/* Roll sequence seq_id back to an earlier committed length: 0 <= new_ctx_len
 * <= ctx_len, pending_token is the committed token at position new_ctx_len.
 * Cancels an uncommitted verify. */
hvd_status hvd_truncate(hvd_kv kv, int32_t seq_id, int32_t new_ctx_len, int32_t pending_token);

/* Release a sequence and its pages. */
hvd_status hvd_seq_free(hvd_kv kv, int32_t seq_id);

/* Query a sequence: ctx_len, pending token, 1 if a verify awaits commit.
 * Any output pointer may be NULL. */
hvd_status hvd_seq_info(hvd_kv kv, int32_t seq_id, int32_t* ctx_len, int32_t* pending_token,
                        int32_t* verify_pending);

/* Number of free pages in the pool. */
int32_t hvd_kv_free_pages(hvd_kv kv);

/* Per-kernel timing: while enabled, every launch of a kernel family is
 * bracketed by HIP events on the handle's stream and its algorithmic HBM bytes
 * (weights streamed, KV read) are accumulated.  family: 0 = QKV GEMM,
 * 1 = O GEMM, 2 = gate/up GEMM, 3 = down GEMM, 4 = LM-head GEMM, 5 = verify
 * attention, 6 = attention combine, 7 = everything else, 8 = the one-launch
 * verify step (HVD_OPT_FLOW: the whole forward, its bytes the step's weights
 * and K/V), 9 = the attention + O launch (HVD_OPT_ATTN_O: its bytes the K/V
 * and the O weights).  hvd_profile_read returns the
 * summed event time (ms), launch count and algorithmic bytes since the last
 * enable.  The events add a little time to every bracketed launch. */
hvd_status hvd_profile_enable(hvd_kv kv, int32_t enable);
hvd_status hvd_profile_read(hvd_kv kv, int32_t family, double* ms, int64_t* launches, double* bytes);

/* Handle options.
 * HVD_OPT_GRAPHS (default 0): 1 replays each step's kernel sequence from a
 *   HIP graph cached per step shape (rows, sequences, attention work
 *   buckets, logits pointer); 0 launches the kernels one by one, which
 *   measured slightly faster for single-sequence verifies.  Results are
 *   identical either way.  Profiling (hvd_profile_enable) always launches
 *   eagerly.
 * HVD_OPT_MLP_SINGLE (default 2 up to 32 layers, 0 above): in verify
 *   forwards the gate/up GEMM (2), the down GEMM (3) or both (1) take the
 *   fp16 activation alone (11 bits) instead of the fp16 hi + lo pair (~22
 *   bits), halving their activation traffic and MFMA work; 0 keeps the pair
 *   for both.  Prefill always uses the pair.  Either GEMM's single pass
 *   moves logits (gate/up's input rounding about twice as much as down's),
 *   and the error grows with depth: the default keeps the pair where it is
 *   cheaper, in the down GEMM, and for models deeper than 32 layers in both.
 * HVD_OPT_LM_SINGLE (default 1): likewise for the LM-head GEMM of verify
 *   forwards (its rounding error, ~1e-4 on the logits, is far below the
 *   tolerance); 0 keeps the pair.
 * HVD_OPT_FLOW (default 0): 1 runs verify steps of at most 32 rows (head dim
 *   128, at most 128 query rows per kv head per sequence, chain drafts) as
 *   one kernel launch in which each phase's workgroups request their weights
 *   before waiting for the previous phase; 0 launches one kernel per GEMM /
 *   attention pass (measured faster at batch 1).  Results agree within
 *   rounding (the attention split may differ).
 * HVD_OPT_FLOW_ITEMS (default 128): attention work items the one-launch step
 *   aims for (longer KV chunks when fewer); a tuning knob.
 * HVD_OPT_ATTN_O (default 0): 1 runs each layer's attention, split-KV merge
 *   and O projection of verify forwards of at most 32 rows as one launch
 *   whose workgroups hold their O weight strip in registers while the
 *   attention runs (head dim 128, K = 4096 and at most one 16-column strip
 *   per compute unit); results agree with the separate launches within
 *   rounding (the KV chunking may differ).
 *
 * Tuning overrides of the launch policy (for measurements and tests; results
 * stay within the verify step's tolerance whatever they are set to):
 * HVD_OPT_GEMM_MIN_BLOCKS (192): GEMM workgroups below which the skinny GEMM
 *   changes shape.  HVD_OPT_ATTN_MIN_ITEMS (256): attention items a launch
 *   aims for.  HVD_OPT_ATTN_MAX_NP (16): most KV pages one attention
 *   sub-chunk stages (power of two, 2..16).  HVD_OPT_SKINNY_MAX_MT (8): row
 *   tiles above which GEMMs take the MFMA-tiled kernel.  HVD_OPT_NS8_MT3 (1):
 *   8-strip skinny blocks at three and four single-pass row tiles.
 *   HVD_OPT_PREFILL_ROWS (0 = policy): prefill chunk rows, a multiple of 16.
 * HVD_OPT_GEMM_SHAPE + f, f = 0 QKV, 1 O, 2 gate/up, 3 down, 4 LM head:
 *   skinny GEMM shape of that GEMM, strips * 100 + K splits (0 = policy).
 * HVD_OPT_TILED_SHAPE + f: tiled GEMM shape, (tile + 1) * 100 + K splits
 *   (tile 0 = 128x128, 1 = 128x256, 2 = 256x256 / 8 waves, 3 = 256x256 / 4
 *   waves, 4 = 128x256 / 8 waves; 0 = policy). */
enum {
  HVD_OPT_GRAPHS = 1, HVD_OPT_MLP_SINGLE = 2, HVD_OPT_LM_SINGLE = 3, HVD_OPT_FLOW = 4, HVD_OPT_FLOW_ITEMS = 5,
  HVD_OPT_ATTN_O = 6,
  HVD_OPT_GEMM_MIN_BLOCKS = 10, HVD_OPT_ATTN_MIN_ITEMS = 11, HVD_OPT_ATTN_MAX_NP = 12, HVD_OPT_SKINNY_MAX_MT = 13,
  HVD_OPT_NS8_MT3 = 14, HVD_OPT_PREFILL_ROWS = 15, HVD_OPT_GEMM_SHAPE = 16, HVD_OPT_TILED_SHAPE = 24
};
hvd_status hvd_kv_set_option(hvd_kv kv, int32_t option, int32_t value);

/* Diagnostics of the one-launch step (HVD_OPT_FLOW): while dev_buf (DEVICE,
 * caller-owned, n_words uint64) is set, each such step whose workgroups fit
 * (4 words each) writes, for workgroup w in launch order, words 4w..4w+3:
 * its start, the time it found its inputs complete, its end (a 100 MHz
 * constant-rate device clock) and the hardware id it ran on (XCD << 32 |
 * HW_ID).  The attention + O launches (HVD_OPT_ATTN_O) of a step whose
 * stamps fit write, for layer l and workgroup w, 8 words at
 * 8 * (l * workgroups + w): the workgroup's start, its attention items done,
 * counted, all items seen, its merges done, counted, all merges seen, and
 * its end.  dev_buf NULL stops tracing.  Not needed for results. */
hvd_status hvd_flow_trace(hvd_kv kv, uint64_t* dev_buf, int64_t n_words);

/* Measure the dense fp16 MFMA rate of the current GPU (not a step of the
 * verify path; a reference for the MFMA fractions the benchmark quotes):
 * every SIMD runs waves of register-only MFMA 32x32x16 f16 chains on
 * stream (hipStream_t, NULL = default) for a few milliseconds; *tflops
 * receives the best of three timed launches.  Returns 0, or a negative
 * hvd_status. */
int hvd_measure_mfma_peak(void* stream, double* tflops);

/* Message of the last failing call on this thread ("" if none). */
const char* hvd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* HVD_H */
