// Kernel argument blocks and host-side launchers of libhvd (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

namespace hvd {

// Per-role kernel timing (profiling only): while a role's scope is open, its
// launches go through hipExtLaunchKernel with these events, so `start` marks
// the start of the role's first kernel and `stop` the end of its last one
// (kernel execution only, as a kernel trace measures it).
struct LaunchTiming {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local LaunchTiming tl_timing;

template <typename F, typename... Args>
inline void hvd_launch(F kernel, const dim3& grid, const dim3& block, uint32_t lds, hipStream_t s, Args... args) {
  if (tl_timing.start != nullptr || tl_timing.stop != nullptr) {
    hipExtLaunchKernelGGL(kernel, grid, block, lds, s, tl_timing.start, tl_timing.stop, 0u, args...);
    tl_timing.start = nullptr;
  } else {
    hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
  }
}

constexpr int kPage = 16;        // tokens per KV page
constexpr int kAttnChunk = 256;  // most KV positions one attention workgroup stages in LDS

// Row metadata of one forward: token, sequence slot, rotary position, and
// where the row's K/V goes: kvs = pool page * kPage + offset in the page.
// (For a chain row the K/V position is its rotary position; a tree node at
// depth d sits at rotary position ctx + d and K/V position ctx + 1 + node.)
struct RowMeta {
  int32_t tok, slot, pos, kvs;
};
// Sequence metadata of one forward: slot, cached length, draft length k (or
// tree node count), first row (rows cu .. cu+k), tree = 1 for a token tree.
struct SeqMeta {
  int32_t slot, ctx, k, cu;
  int32_t tree, pad0, pad1, pad2;
};
// Token trees: at most this many nodes, so a row's ancestor set over the
// pending token and the nodes fits one 64-bit mask (bit 0 = pending row).
constexpr int kMaxTreeNodes = 63;
// One attention work item, self-contained so a workgroup needs no other
// metadata: sequence slot, cached length ctx, draft length k, first row cu;
// kv head g; KV chunk c of nch covering positions [p_begin, p_end); the row
// group rg (rows [rg*128, rg*128+128) of the (k+1)*group query rows); for
// multi-chunk items, the partial slot `part` (combine heads: first slot); and
// the pool pages holding the first kAttnChunk positions of the chunk, so the
// KV loads need not wait for a page-table read.
constexpr int kItemPages = 16;  // kAttnChunk / kPage
struct AttnItem {
  int32_t slot, ctx, k, cu;
  int32_t g, c, nch, rg;
  int32_t part, p_begin, p_end, tree;
  int32_t pad1, pad2, pad3, pad4;
  int32_t pages[kItemPages];
};
static_assert(kItemPages * kPage == kAttnChunk, "item page list covers one LDS sub-chunk");

enum Epilogue { EPI_QKV = 0, EPI_RESID = 1, EPI_SILU = 2, EPI_LM = 3 };

struct GemmArgs {
  const uint4* W;    // packed weights: 1 KB fragment of strip s, K step kt at
                     // (s/4)*wg + (s%4)*64 + kt*wk (16-byte units)
  size_t wg, wk;     // group and K-step strides of the packing (see pack_weight)
  const uint4* Ahi;  // packed activations (hi part), fragment (kt, mt) at (kt*MTtot + mt)*64
  const uint4* Alo;  // packed activations (lo part)
  int KT, NT, MTtot, M;
  // inverse RMS of the GEMM's input rows, from per-16-column sums of squares
  const float* ss;   // [MTtot*16][ss_n] (null: no row scaling)
  int ss_n;
  float inv_dim, eps;
  // EPI_QKV
  _Float16* Q;       // [M][Hq*dh], d in rotary-pair order
  _Float16* kv;      // this layer's KV pool: page p, K at p*page_stride, V at +Hkv*16*dh
  size_t page_stride;
  int q_cols, kv_cols, Hkv, dh;
  const int32_t* pt;  // page table [max_seqs][pt_stride]
  int pt_stride;
  const RowMeta* rows;
  const float2* rope;  // [max_pos][dh/2] (cos, sin)
  // EPI_RESID
  float* X;            // residual stream [MTtot*16][D] fp32
  float* X_out;        // nullable: the updated stream goes here instead of X
  int D;
  const float* gain_next;  // gain of the norm that consumes X next
  uint16_t* Nhi;       // next GEMM's A operand (hi), K = D
  uint16_t* Nlo;
  float* ss_out;       // [MTtot*16][D/16]
  // EPI_SILU
  uint16_t* act_hi;    // down GEMM's A operand, K = F
  uint16_t* act_lo;
  // EPI_LM
  float* logits;       // [M][vocab] or null
  int vocab;
  float* part_val;     // [M][n_part]
  int32_t* part_idx;
  int n_part;
  // K split across workgroups: partial tiles [mblocks][NT/ns][splits][rows][cols]
  // and one arrival counter per (row block, column block), zero between launches
  float* part;
  uint32_t* cnt;
};

struct AttnArgs {
  const _Float16* Q;
  const _Float16* kv;  // this layer's pool
  size_t page_stride;
  int Hq, Hkv, dh, group;
  const int32_t* pt;
  int pt_stride;
  const AttnItem* items;
  float scale_log2;    // log2(e) / sqrt(dh)
  uint16_t* Ohi;       // O GEMM A operand (K = Hq*dh)
  uint16_t* Olo;
  int MTtot;
  float* part_o;       // [slots][rows per item][dh] fp32 unnormalized output of one chunk
  float* part_ml;      // [slots][rows per item][2] running max (base 2) and sum
  const uint64_t* tree_mask;  // [rows]: tree rows' ancestor sets over positions ctx.. (bit j = ctx + j)
};

struct CombineArgs {
  const AttnItem* heads;  // one entry per (b, g, rg) whose nch > 1; part = first slot
  int Hq, Hkv, dh, group;
  const float* part_o;
  const float* part_ml;
  uint16_t* Ohi;
  uint16_t* Olo;
  int MTtot;
  int rpi;       // query rows per work item (partial slot stride)
  int max_rows;  // most rows of any head entry (1..rpi): sizes the grid
};

struct EmbedArgs {
  const uint16_t* E;   // embedding [V][D] bf16
  const RowMeta* rows;
  int M, Mpad, D;
  const float* gain;
  float* X;
  uint16_t* Nhi;
  uint16_t* Nlo;
  float* ss_out;
  int MTtot;
  // page-table updates applied before any KV write of this step
  const int32_t* upd;    // [n_upd][3]: slot, index, page
  const int32_t* n_upd;  // device count (metadata header) so the launch is shape-only
  int32_t* pt;
  int pt_stride;
  int V;  // token ids outside [0, V) gather row 0 (they can never be accepted)
  uint32_t* zero;  // nullable: n_zero words cleared before the step (one-launch step counters)
  int n_zero;
};

struct AcceptArgs {
  const float* part_val;
  const int32_t* part_idx;
  int n_part;
  int M;
  int32_t* g;          // [M] argmax per row
  const SeqMeta* seqs;
  const RowMeta* rows;
  int B;
  int32_t* out;        // [B][2]: accepted, next
  uint32_t* counter;   // one uint32, zero between launches
  const int32_t* tree_parent;  // [rows]: parent node of a tree row (-1 = the pending token)
  int32_t* path;       // [B][kMaxTreeNodes]: accepted node indices of tree sequences
  // device-resident loop (null otherwise): the commit of the accepted block is
  // applied here, state = ctx[B], pending[B], steps done; each step's
  // (accepted, next) pairs go to hist[step][B][2] while step < hist_cap
  int32_t* astate;
  int32_t* hist;
  int hist_cap;
  const uint32_t* err_word;  // nullable: the step's error word of bounded in-kernel waits, copied to out[err_index]
  int err_index;             // after the results (and a tree step's paths)
};
// Moves the K/V of each tree sequence's accepted path from the nodes'
// positions (ctx + 1 + node) to the chain positions ctx + 1 .. ctx + a.
struct CompactArgs {
  _Float16* pool;      // all layers
  size_t page_stride, layer_stride;
  int n_layers, Hkv, dh;
  const int32_t* pt;
  int pt_stride;
  const SeqMeta* seqs;
  const int32_t* out;  // [B][2] accepted, next
  const int32_t* path; // [B][kMaxTreeNodes]
};

// Device-resident verify loop: one workgroup rebuilds a step's row and
// attention metadata from the device state (ctx and pending token per
// sequence) and the draft buffer, so the step's captured launches need no
// host staging.  The attention items were planned on the host for the longest
// context the loop can reach; here each item takes the current ctx, its chunk
// end, and whether it still has keys (chunks past the keys become no-ops and
// the combine entries count only the live chunks).
struct AsyncPlanArgs {
  const int32_t* state;      // ctx[B], pending[B]
  int32_t* drafts;           // [sum k]: draft tokens of sequence b from seq_static[b].cu - b
  const int32_t* ref;        // nullable: [B][ref_len] token stream of the copy drafter
  int ref_len;
  const int32_t* ref_start;  // [B]: position of ref[b][0]
  const SeqMeta* seq_static; // [B] (ctx unused)
  const int32_t* page_off;   // [B + 1]: offsets of each sequence's page list in pages
  const int32_t* pages;      // reserved pages of every sequence, concatenated
  const int32_t* row_seq;    // [M]: sequence of each row
  RowMeta* rows;             // [M] out
  SeqMeta* seqs;             // [B] out
  const AttnItem* items_static;  // [n_items]: pad1 = sequence, pad2 = the unit's last row index,
  AttnItem* items;               //   pad3 = its plan's chunk length
  int n_items;
  const AttnItem* heads_static;  // [n_heads], same extra fields
  AttnItem* heads;
  int n_heads;
  int M, B;
};

// One-launch verify step (flow.hip): every layer's QKV GEMM, attention,
// split-KV merge, O, gate/up and down GEMMs, then the LM head, as one grid.
// Workgroup w takes the role its index gives (layer, phase, unit); roles of
// later phases have larger indices, so a workgroup only ever waits for work
// of smaller indices, which the in-order dispatch has already started.
// Finished output blocks are counted per layer and phase; a consumer
// requests its weights (and cached K/V) first, waits (bounded, see err)
// until its inputs are complete, then reads them with device-scope loads.
// One layer's weights, KV pool and activation buffers.  In the one-launch
// step every activation buffer is written once per launch and read only
// after its producers are complete, so readers use ordinary (L2-cached)
// loads: no buffer is shared by two layers.
struct FlowLayer {
  const uint4 *qkv, *o, *gu, *down;  // packed weights
  const float *g_attn, *g_mlp;        // norm gains
  _Float16* kv;                        // this layer's KV pool
  // input: residual stream, next norm's operand (hi, lo), sums of squares
  // (the previous layer's output; the embedding's for layer 0)
  const float* x_in;
  const uint16_t *n_in_hi, *n_in_lo;
  const float* ss_in;
  float* x_mid;  // after attention + O
  uint16_t *n_mid_hi, *n_mid_lo;
  float* ss_mid;
  float* x_out;  // after the MLP
  uint16_t *n_out_hi, *n_out_lo;
  float* ss_out;
  _Float16* q;                   // rotated queries
  uint16_t *o_hi, *o_lo;         // attention output (O GEMM operand)
  uint16_t *a_hi, *a_lo;         // SiLU(gate) * up (down GEMM operand)
};
enum { FL_QKV = 0, FL_ATTN = 1, FL_MERGE = 2, FL_O = 3, FL_GU = 4, FL_DOWN = 5, FL_PHASES = 6 };
enum { FG_QKV = 0, FG_O = 1, FG_GU = 2, FG_DOWN = 3, FG_LM = 4, FG_N = 5 };
struct FlowArgs {
  const FlowLayer* layers;  // [L] (device)
  int L;
  GemmArgs g[FG_N];         // per GEMM role; W / kv / gains / counters set per layer in the kernel
  int ns[FG_N], splits[FG_N], n_cb[FG_N];
  const float* g_final;     // gain of the final norm (read by the last down GEMM's epilogue)
  AttnArgs attn;            // kv set per layer
  CombineArgs comb;
  int np;                   // attention pages per sub-chunk
  int per_layer;            // workgroups of one layer
  int ph[FL_PHASES + 1];    // first workgroup of each phase within a layer (ph[FL_PHASES] = per_layer)
  int n_lm;                 // LM-head workgroups after the layers
  const AttnItem* items;    // attention items of one layer (pad4: merge unit of a multi-chunk item)
  const AttnItem* heads;    // merge entries (pad4: merge unit)
  int merge_spb;            // row slices per merge entry
  // counters, `cstride` per layer: [0, Hkv) finished QKV blocks per kv-head
  // group; [c_unit, +units) finished chunks per merge unit; then 8-way split
  // counters (indexed by block & 7) of O inputs (single-chunk items and merge
  // slices), O, gate/up and down output blocks
  uint32_t* cnt;
  int cstride, c_unit, c_oin, c_o, c_gu, c_down;
  uint32_t qkv_group_target;  // QKV output blocks per kv-head group
  uint32_t oin_target;        // single-chunk items + merge slices per layer
  uint32_t* err;              // set (bit 0) if a wait gave up: results are then invalid
  int G, dh;
  // nullable diagnostics: per workgroup {start, inputs ready, end} in the
  // 100 MHz constant clock and the hardware id (XCD, CU) it ran on
  uint64_t* trace;
};

// Attention, its split-KV merge and the O GEMM of one layer as one launch
// of n_attn + go.NT co-resident 256-thread workgroups (attn_o.hip).
struct AttnOArgs {
  AttnArgs at;              // items: n_items (attention workgroup r takes items r, r + n_attn, ...)
  CombineArgs cb;           // merge entries: n_heads, merge_spb row slices each
  GemmArgs go;              // the O GEMM: one 16-column strip per O workgroup
  int n_attn;               // attention workgroups (the first of the grid)
  int n_items, n_heads, merge_spb;
  // [2][kAoSlots] counters kAoSlotWords apart (items done, merges done),
  // zeroed once per step; layer l waits for (l + 1) * n_attn arrivals
  uint32_t* cnt;
  uint32_t target;          // (layer + 1) * n_attn
  uint32_t* err;            // bit 0 set if a wait gave up (results then invalid)
  // nullable diagnostics: per workgroup kAoTraceWords constant-clock stamps
  // (attention: start, items done, counted, all items seen, merges done,
  // counted; O: start, strip requested, all merges seen, end at 0, 1, 6, 7)
  uint64_t* trace;
};
constexpr int kAoTraceWords = 8;
constexpr int kAoSlots = 32;
constexpr int kAoSlotWords = 32;  // one 128-byte line per counter slot
constexpr int kAoMergeRows = 2;   // rows per merge slice (256 threads, 8 lanes per (row, 8 dims))

// Launchers: all enqueue on `s` and return the launch status.
hipError_t launch_pack(const uint16_t* src, const int32_t* rowmap, uint16_t* dst, int N, int K,
                       hipStream_t s);
hipError_t launch_embed(const EmbedArgs& a, hipStream_t s);
// ns: 16-column strips per workgroup (1, 2, 4; >= 2 for EPI_SILU); grid.x = NT / ns.
// splits > 1 splits K across workgroups; the last split of each output block
// to finish reduces (a.part, a.cnt).
// hi_lo false: the hi activation part alone (honoured for the residual and
// SiLU GEMMs at 3-4 row tiles; other shapes keep the pair)
hipError_t launch_gemm(int epi, const GemmArgs& a, int ns, int splits, int mblocks, int mt_block, bool hi_lo,
                       hipStream_t s);
// Large-batch GEMM (gemm_tiled.hip): tile 0 = 128 x 128, 1 = 128 x 256,
// 2 = 256 x 256 (8 waves), 3 = 256 x 256 (4 waves), 4 = 128 x 256 (8 waves)
// (rows x columns); hi_lo false = the hi activation part
// alone; K split `splits` ways; inv_rms is a per-row scratch vector
// (computed here for normalised inputs).
hipError_t launch_gemm_tiled(int epi, const GemmArgs& a, int tile, bool hi_lo, int splits, float* inv_rms,
                             hipStream_t s);
// chunk: the plan's KV chunk length (picks the pages staged per sub-chunk);
// rows_per_item: 64, 128 or 256 (256 for head_dim 128 only)
// max_np caps the pages staged per sub-chunk (longer chunks loop over sub-chunks)
hipError_t launch_attn(const AttnArgs& a, int n_items, int chunk, int rows_per_item, int max_np, hipStream_t s);
hipError_t attn_set_lds_limit();  // once per process, before the first launch
int attn_pages_per_sub(int chunk);        // pages one sub-chunk stages for a chunk length
size_t attn_lds_bytes(int dh, int np);    // LDS of a workgroup staging np-page sub-chunks
hipError_t launch_combine(const CombineArgs& a, int n_heads, hipStream_t s);
hipError_t launch_accept(const AcceptArgs& a, hipStream_t s);
hipError_t launch_compact(const CompactArgs& a, int B, hipStream_t s);
hipError_t launch_async_plan(const AsyncPlanArgs& a, hipStream_t s);
hipError_t launch_pt_update(const int32_t* upd, const int32_t* n_upd, int32_t* pt, int pt_stride, hipStream_t s);
// n 32-bit words from src (device-accessible, e.g. pinned host memory) to dst
// (device); both 16-byte aligned.
hipError_t launch_copy_words(int32_t* dst, const int32_t* src, size_t n, hipStream_t s);
// One-launch verify step over MT (1 or 2) row tiles; false if this shape has
// no compiled variant (head dim, strips per workgroup, pages per sub-chunk).
bool flow_supported(int MT, int dh, int np, const int* ns);
hipError_t launch_flow(const FlowArgs& f, int MT, hipStream_t s);
hipError_t flow_set_lds_limit();  // once per process, before the first launch
// Whether the fused attention + O launch handles this shape (head dim, pages
// per sub-chunk, row tiles, K steps and strips of the O GEMM) and fits
// `n_cus` compute units.
bool attn_o_supported(int dh, int np, int MT, int KT, int NT, int n_cus);
hipError_t launch_attn_o(const AttnOArgs& a, int np, int rows_per_item, int MT, hipStream_t s);
hipError_t attn_o_set_lds_limit();

constexpr int kGemmMaxMT = 4;  // 16-row tiles of one GEMM workgroup (5 for single-pass GEMMs of 65-80 rows)
constexpr int kGemmPadMT = 5;  // row tiles of padding after every GEMM operand

// Static per-device scratch of hvd_verify_noalloc (scratch.hip): its device
// address on the current device, taken once per device.
constexpr size_t kStaticScratchBytes = 64u << 20;
hipError_t static_scratch(void** ptr, size_t* bytes);

}  // namespace hvd
