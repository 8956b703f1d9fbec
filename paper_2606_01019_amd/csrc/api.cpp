// C ABI of libhvd: model loading and packing, the KV cache handle, and the
// verify / commit / prefill drivers that enqueue the gfx950 kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/hvd.h"
#include "host_state.h"
#include "kernels.h"

using namespace hvd;

namespace {

thread_local std::string g_err;

hvd_status set_err(hvd_status s, const std::string& m) {
  g_err = m;
  return s;
}

#define HIP_TRY(expr)                                                                          \
  do {                                                                                         \
    hipError_t e_ = (expr);                                                                    \
    if (e_ != hipSuccess) return set_err(HVD_ERR_DEVICE, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr size_t kAlign = 256;
// Prefill chunk: rows whose query rows per kv head (rows x group) come to
// 2048, between 128 and 512 rows (measured: 512 rows for the 8B shape,
// group 4, above 256 and 1024; 256 for the 32B shape, group 8, above 512).
// HVD_OPT_PREFILL_ROWS overrides it per handle (up to this size).
int prefill_rows(const hvd_config& c) {
  const int G = c.n_q_heads / c.n_kv_heads;
  return std::max(128, std::min(512, 2048 / G));
}
// Up to 8 row tiles (128 rows) the skinny kernel in row blocks of <= 4
// tiles beats the tiled kernel (measured: 65-row verifies and 128-row
// prefill chunks of the 8B shape)
constexpr int kSkinnyMaxMT = 8;
constexpr int kMlpSingleMaxLayers = 32;      // deepest model whose verify gate/up GEMM runs single-pass by default
constexpr int kGemmMinBlocks = 192;          // GEMM workgroups below which the shape changes
constexpr int kGemmSplitTarget = 256;        // workgroups a K split aims for (one per CU)
constexpr int kGemmLongK = 256;              // K steps above which a K split pays for its reduction
constexpr size_t kGemmPartBytes = 64u << 20;  // split-K partial tiles of one GEMM launch
constexpr int kGemmCounters = 16384;          // split-K arrival counters (output blocks of one launch)
constexpr int kFlowCounterWords = 1 << 17;    // one-launch step: error word and per-layer counters
constexpr int kAoCounterBase = 64;             // attention + O launches: their counters after the error word
constexpr int kFlowAttnItems = 128;           // attention items the one-launch step aims for
constexpr int kFlowRows = 32;                 // rows of the one-launch step (two 16-row tiles)
constexpr int kAttnMinItems = 256;            // attention workgroups wanted per launch
constexpr int kCUs = 256;                     // compute units of the MI355X
constexpr int kAttnRows = 128;     // query rows per attention work item
constexpr int kAttnClasses = 4;    // attention row classes: items of 64, 128, 256 and 384 rows
constexpr int kPartSlots = 4096;   // attention partial slots (multi-chunk items)
constexpr size_t kMaxGraphs = 64;  // cached step graphs per KV handle
// profiling families: GEMM by role, attention, combine, everything else
enum { PF_QKV = 0, PF_O = 1, PF_GATEUP = 2, PF_DOWN = 3, PF_LM = 4, PF_ATTN = 5, PF_COMBINE = 6, PF_OTHER = 7,
       PF_FLOW = 8, PF_ATTN_O = 9, kProfFamilies = 10 };

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Bump allocator over one device buffer.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  template <class T>
  T* take(size_t n) {
    T* p = base ? (T*)(base + off) : nullptr;
    off = align_up(off + n * sizeof(T));
    return p;
  }
};

hvd_status check_config(const hvd_config* c) {
  if (!c) return set_err(HVD_ERR_ARG, "null config");
  if (c->n_layers < 1 || c->d_model < 64 || c->d_model % 64) return set_err(HVD_ERR_ARG, "d_model must be a positive multiple of 64");
  if (c->head_dim != 64 && c->head_dim != 128) return set_err(HVD_ERR_ARG, "head_dim must be 64 or 128");
  if (c->n_kv_heads < 1 || c->n_q_heads < 1 || c->n_q_heads % c->n_kv_heads) return set_err(HVD_ERR_ARG, "n_q_heads must be a multiple of n_kv_heads");
  if (c->ffn_dim < 32 || c->ffn_dim % 32) return set_err(HVD_ERR_ARG, "ffn_dim must be a positive multiple of 32");
  if (c->vocab < 64 || c->vocab % 64) return set_err(HVD_ERR_ARG, "vocab must be a positive multiple of 64");
  if (c->page_size != kPage) return set_err(HVD_ERR_ARG, "page_size must be 16");
  if (c->max_draft < 0 || c->max_draft > 64) return set_err(HVD_ERR_ARG, "max_draft must be in [0, 64]");
  if (c->max_pos < 32) return set_err(HVD_ERR_ARG, "max_pos must be >= 32");
  if (!(c->rope_theta > 0.f) || !(c->rms_eps > 0.f)) return set_err(HVD_ERR_ARG, "rope_theta and rms_eps must be > 0");
  return HVD_OK;
}

struct LayerW {
  uint16_t *qkv, *o, *gu, *down;
  float *g_attn, *g_mlp;
};

}  // namespace

struct hvd_model_s {
  hvd_config cfg;
  void* base = nullptr;
  bool owned = false;
  size_t bytes = 0;
  uint16_t* embed = nullptr;
  std::vector<LayerW> layers;
  float* g_final = nullptr;
  uint16_t* lm = nullptr;
  float2* rope = nullptr;
  hipStream_t stream = nullptr;
};

namespace {

// Lay out (or size, with base == null) the model buffer.
size_t carve_model(hvd_model_s* m, void* base) {
  const hvd_config& c = m->cfg;
  Carver cv(base);
  const size_t D = c.d_model, F = c.ffn_dim, V = c.vocab, qd = (size_t)c.n_q_heads * c.head_dim,
               kd = (size_t)c.n_kv_heads * c.head_dim;
  m->embed = cv.take<uint16_t>(V * D);
  m->layers.resize(c.n_layers);
  for (auto& L : m->layers) {
    L.qkv = cv.take<uint16_t>((qd + 2 * kd) * D);
    L.o = cv.take<uint16_t>(D * qd);
    L.gu = cv.take<uint16_t>(2 * F * D);
    L.down = cv.take<uint16_t>(D * F);
    L.g_attn = cv.take<float>(D);
    L.g_mlp = cv.take<float>(D);
  }
  m->g_final = cv.take<float>(D);
  m->lm = cv.take<uint16_t>(V * D);
  m->rope = cv.take<float2>((size_t)c.max_pos * (c.head_dim / 2));
  return cv.off;
}

}  // namespace

extern "C" size_t hvd_model_bytes(const hvd_config* cfg) {
  if (check_config(cfg) != HVD_OK) return 0;
  hvd_model_s tmp;
  tmp.cfg = *cfg;
  return carve_model(&tmp, nullptr);
}

namespace {

float bf16_bits_to_float(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

hvd_status upload_gain(const uint16_t* src, float* dst, int n, hipStream_t s) {
  std::vector<float> g(n);
  for (int i = 0; i < n; ++i) g[i] = bf16_bits_to_float(src[i]);
  HIP_TRY(hipMemcpyAsync(dst, g.data(), n * sizeof(float), hipMemcpyHostToDevice, s));
  HIP_TRY(hipStreamSynchronize(s));
  return HVD_OK;
}

// Copy rows of host tensors into the staging buffer back to back, then pack
// them into fragment order through rowmap.
hvd_status pack_group(const std::vector<std::pair<const uint16_t*, size_t>>& parts, const std::vector<int32_t>& rowmap,
                      int K, uint16_t* staging, int32_t* dmap, uint16_t* dst, hipStream_t s) {
  size_t off = 0;
  for (auto& p : parts) {
    HIP_TRY(hipMemcpyAsync(staging + off, p.first, p.second * sizeof(uint16_t), hipMemcpyHostToDevice, s));
    off += p.second;
  }
  HIP_TRY(hipMemcpyAsync(dmap, rowmap.data(), rowmap.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
  HIP_TRY(launch_pack(staging, dmap, dst, (int)rowmap.size(), K, s));
  HIP_TRY(hipStreamSynchronize(s));
  return HVD_OK;
}

}  // namespace

extern "C" hvd_status hvd_model_load(const hvd_config* cfg, const uint16_t* const* t, void* dev_buf, size_t dev_bytes,
                                     void* stream, hvd_model* out) {
  if (hvd_status st = check_config(cfg); st != HVD_OK) return st;
  if (!t || !out) return set_err(HVD_ERR_ARG, "null tensors or out");
  const hvd_config& c = *cfg;
  const int n_t = 3 + 9 * c.n_layers;
  for (int i = 0; i < n_t; ++i)
    if (!t[i]) return set_err(HVD_ERR_ARG, "null tensor pointer");
  auto* m = new hvd_model_s();
  m->cfg = c;
  m->stream = (hipStream_t)stream;
  const size_t need = carve_model(m, nullptr);
  if (dev_buf) {
    if (dev_bytes < need) {
      delete m;
      return set_err(HVD_ERR_ARG, "dev_buf smaller than hvd_model_bytes");
    }
    m->base = dev_buf;
  } else {
    if (hipMalloc(&m->base, need) != hipSuccess) {
      delete m;
      return set_err(HVD_ERR_OOM, "hipMalloc of model weights failed");
    }
    m->owned = true;
  }
  m->bytes = need;
  carve_model(m, m->base);
  hipStream_t s = m->stream;

  const size_t D = c.d_model, F = c.ffn_dim, V = c.vocab, dh = c.head_dim, qd = (size_t)c.n_q_heads * dh,
               kd = (size_t)c.n_kv_heads * dh;
  size_t stage_elems = std::max({(qd + 2 * kd) * D, 2 * F * D, D * F, V * D, D * qd});
  size_t map_elems = std::max({qd + 2 * kd, 2 * F, V, D});
  uint16_t* staging = nullptr;
  int32_t* dmap = nullptr;
  hvd_status st = HVD_OK;
  auto fail = [&](hvd_status e) {
    if (staging) (void)hipFree(staging);
    if (dmap) (void)hipFree(dmap);
    if (m->owned) (void)hipFree(m->base);
    delete m;
    return e;
  };
  hipError_t ea = hipMalloc(&staging, stage_elems * 2);
  if (ea == hipSuccess) ea = hipMalloc(&dmap, map_elems * 4);
  if (ea != hipSuccess) {
    size_t free_b = 0, total_b = 0;
    (void)hipMemGetInfo(&free_b, &total_b);
    return fail(set_err(HVD_ERR_OOM, std::string("hipMalloc of load staging (") + std::to_string(stage_elems * 2) +
                                         " bytes) failed: " + hipGetErrorString(ea) + "; device memory free " +
                                         std::to_string(free_b) + " of " + std::to_string(total_b) + " bytes"));
  }

  auto ident = [](size_t n) {
    std::vector<int32_t> r(n);
    for (size_t i = 0; i < n; ++i) r[i] = (int32_t)i;
    return r;
  };
  // q and k output rows permuted inside each head so that the rotate-half
  // pairs (j, j + dh/2) become adjacent columns (2j, 2j+1).
  std::vector<int32_t> qkv_map(qd + 2 * kd);
  for (size_t n = 0; n < qd + 2 * kd; ++n) {
    if (n < qd + kd) {
      size_t base = n < qd ? 0 : qd;
      size_t head = (n - base) / dh, dp = (n - base) % dh;
      size_t d = (dp % 2 == 0) ? dp / 2 : dh / 2 + dp / 2;
      qkv_map[n] = (int32_t)(base + head * dh + d);
    } else {
      qkv_map[n] = (int32_t)n;
    }
  }
  // gate/up interleaved by 16-row strips: strip 2s = gate rows 16s.., 2s+1 = up rows.
  std::vector<int32_t> gu_map(2 * F);
  for (size_t n = 0; n < 2 * F; ++n) {
    size_t strip = n / 16;
    gu_map[n] = (int32_t)((strip % 2 ? F : 0) + (strip / 2) * 16 + n % 16);
  }
  const std::vector<int32_t> map_D = ident(D), map_V = ident(V);

  if (hipMemcpyAsync(m->embed, t[0], V * D * 2, hipMemcpyHostToDevice, s) != hipSuccess)
    return fail(set_err(HVD_ERR_DEVICE, "embedding upload failed"));
  for (int l = 0; l < c.n_layers && st == HVD_OK; ++l) {
    const uint16_t* const* lt = t + 1 + 9 * l;
    LayerW& L = m->layers[l];
    if ((st = upload_gain(lt[0], L.g_attn, (int)D, s)) != HVD_OK) break;
    if ((st = pack_group({{lt[1], qd * D}, {lt[2], kd * D}, {lt[3], kd * D}}, qkv_map, (int)D, staging, dmap, L.qkv, s)) != HVD_OK) break;
    if ((st = pack_group({{lt[4], D * qd}}, map_D, (int)qd, staging, dmap, L.o, s)) != HVD_OK) break;
    if ((st = upload_gain(lt[5], L.g_mlp, (int)D, s)) != HVD_OK) break;
    if ((st = pack_group({{lt[6], F * D}, {lt[7], F * D}}, gu_map, (int)D, staging, dmap, L.gu, s)) != HVD_OK) break;
    if ((st = pack_group({{lt[8], D * F}}, map_D, (int)F, staging, dmap, L.down, s)) != HVD_OK) break;
  }
  if (st == HVD_OK) st = upload_gain(t[1 + 9 * c.n_layers], m->g_final, (int)D, s);
  if (st == HVD_OK) st = pack_group({{t[2 + 9 * c.n_layers], V * D}}, map_V, (int)D, staging, dmap, m->lm, s);
  if (st != HVD_OK) return fail(st);

  // rotary table: angle = pos * theta^(-2j/dh) in double, stored as fp32 (cos, sin)
  {
    const int half = c.head_dim / 2;
    std::vector<float2> tab((size_t)c.max_pos * half);
    for (int p = 0; p < c.max_pos; ++p)
      for (int j = 0; j < half; ++j) {
        double ang = (double)p * std::pow((double)c.rope_theta, -(2.0 * j) / c.head_dim);
        tab[(size_t)p * half + j] = float2{(float)std::cos(ang), (float)std::sin(ang)};
      }
    if (hipMemcpyAsync(m->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return fail(set_err(HVD_ERR_DEVICE, "rotary table upload failed"));
  }
  (void)hipFree(staging);
  (void)hipFree(dmap);
  *out = m;
  return HVD_OK;
}

extern "C" void hvd_model_free(hvd_model m) {
  if (!m) return;
  if (m->owned && m->base) (void)hipFree(m->base);
  delete m;
}

// ------------------------------------------------------------------ KV handle

// A captured step is valid for every step with the same launch sequence:
// rows, sequences, attention grid sizes and kernel variants (chunk length,
// rows per item), LM head on/off and the logits pointer.
struct GraphKey {
  int M, B, lm_head, tree;
  std::array<int, 4 * kAttnClasses> attn;  // per row class: items, combine entries, chunk, combine rows
  float* logits;
  bool operator<(const GraphKey& o) const {
    return std::tie(M, B, lm_head, tree, attn, logits) < std::tie(o.M, o.B, o.lm_head, o.tree, o.attn, o.logits);
  }
};

struct ProfRec {
  hipEvent_t a, b;
  int family;
  double bytes;
};

// The per-step scratch of one forward: split-K partial tiles, attention
// split-KV partials, LM-head argmax partials, per-row inverse RMS and argmax,
// the results block and the accept kernel's arrival counter.  hvd_verify takes
// it from the handle's workspace; hvd_verify_noalloc from the library's static
// device array.
struct StepScratch {
  float* gemm_part = nullptr;
  size_t gemm_part_bytes = 0;
  uint32_t* gemm_cnt = nullptr;  // split-K arrival counters (zero between launches)
  uint32_t* flow_cnt = nullptr;  // one-launch step: error word, then per-layer counters (cleared each step)
  float* part_o = nullptr;
  float* part_ml = nullptr;
  size_t part_rows = 0;  // attention partial rows (each dh floats in part_o, 2 in part_ml)
  float* lm_val = nullptr;
  int32_t* lm_idx = nullptr;
  float* inv_rms = nullptr;
  int32_t* g = nullptr;
  int32_t* out = nullptr;
  uint32_t* counter = nullptr;
};

struct hvd_kv_s {
  hvd_model_s* m = nullptr;
  HostState* hs = nullptr;
  void* base = nullptr;
  bool owned = false;
  hipStream_t stream = nullptr;
  int32_t n_pages = 0;
  _Float16* pool = nullptr;
  size_t page_stride = 0;   // halves per (layer, page): K and V of every kv head
  size_t layer_stride = 0;  // halves per layer
  int32_t* pt = nullptr;
  int pt_stride = 0;
  int max_rows = 0, MTmax = 0;
  float* X = nullptr;
  float* ss = nullptr;
  uint16_t *Nhi = nullptr, *Nlo = nullptr;
  _Float16* Q = nullptr;
  uint16_t *Ohi = nullptr, *Olo = nullptr;
  uint16_t *Ahi = nullptr, *Alo = nullptr;
  float* lm_val = nullptr;
  int32_t* lm_idx = nullptr;
  int n_part_lm = 0;
  int gemm_min_blocks = kGemmMinBlocks;
  int prefill_rows = 0;  // prefill chunk rows (0: the policy of prefill_rows())
  bool use_graphs = false;
  std::map<GraphKey, hipGraphExec_t> graphs;
  int attn_min_items = kAttnMinItems;
  int attn_max_np = kItemPages;  // most pages one attention sub-chunk stages
  int skinny_max_mt = kSkinnyMaxMT;   // row tiles above which GEMMs take the MFMA-tiled kernel
  int gemm_force[PF_LM + 1][2] = {};  // per GEMM family: {strips per workgroup, K splits} of the skinny kernel, 0 = policy
  bool ns8_mt3 = true;  // 8-strip skinny blocks at three and four single-pass row tiles
  int tiled_force[PF_LM + 1][2] = {};  // per GEMM family: {tile + 1, K splits} of the tiled kernel, 0 = policy
  float* gemm_part = nullptr;
  uint32_t* gemm_cnt = nullptr;
  float* inv_rms = nullptr;  // per-row inverse RMS for the large-batch GEMMs
  bool mlp_single_gu = true;     // verify gate/up GEMMs on the hi activation part only
  bool mlp_single_down = false;  // verify down GEMMs on the hi + lo pair (the cheaper of the two to keep)
  bool lm_single = true;     // large-batch verify LM head on the hi activation part only
  int32_t* g = nullptr;
  int32_t* out = nullptr;
  uint32_t* counter = nullptr;
  float* part_o = nullptr;
  float* part_ml = nullptr;
  int32_t* meta_dev = nullptr;
  int32_t* meta_host = nullptr;
  const int32_t* meta_host_dev = nullptr;  // meta_host as the device sees it
  size_t meta_ints = 0;
  int32_t* out_host = nullptr;
  StepScratch sx;                 // the handle's own step scratch
  bool use_flow = false;          // one-launch step (flow.hip) where the shape allows it (HVD_OPT_FLOW)
  bool use_attn_o = false;        // attention + merge + O GEMM as one launch (attn_o.hip; HVD_OPT_ATTN_O)
  int n_cus = 0;                  // compute units of the device
  int flow_min_items = kFlowAttnItems;  // attention items the one-launch step aims for
  FlowLayer* flow_layers = nullptr;     // [n_layers] (device)
  std::vector<FlowLayer> flow_host;     // the same table on the host (filled by carve_kv)
  uint64_t* flow_trace = nullptr;       // borrowed diagnostics buffer (hvd_flow_trace), or null
  int64_t flow_trace_words = 0;
  uint32_t* flow_cnt = nullptr;         // [kFlowCounterWords]: err word, then the step's counters
  void* static_base = nullptr;    // this device's static scratch (hipGetSymbolAddress at kv_alloc)
  size_t static_bytes = 0;
  // profiling
  bool prof = false;
  std::vector<ProfRec> prof_pending;
  std::vector<hipEvent_t> ev_pool;
  double prof_ms[kProfFamilies] = {}, prof_bytes[kProfFamilies] = {};
  int64_t prof_n[kProfFamilies] = {};
};

namespace {

// Upper bound of one step's metadata: rows, sequences, attention items and
// combine heads (units = sequence x kv head x row group), page-table updates.
size_t meta_capacity_ints(const hvd_config& c, int max_rows, int max_seqs, int pt_stride) {
  const int G = c.n_q_heads / c.n_kv_heads;
  const size_t rg_verify = ((size_t)(c.max_draft + 1) * G + kAttnRows - 1) / kAttnRows;
  const size_t rg_prefill = ((size_t)prefill_rows(c) * G + kAttnRows - 1) / kAttnRows;
  const size_t units = std::max((size_t)max_seqs * rg_verify, rg_prefill) * c.n_kv_heads;
  // items <= units + partial slots (at most 2 kPartSlots: 64-row items),
  // twice over for the no-op items that keep row groups 8 grid positions
  // apart, and heads <= units, each row class padded up (to 64 and 16
  // entries); header and per-section alignment fit in the last term
  const size_t item_ints = sizeof(AttnItem) / 4;
  return (4 + 3) * (size_t)max_rows + sizeof(SeqMeta) / 4 * (size_t)max_seqs +
         item_ints * (4 * units + 4 * kPartSlots + kAttnClasses * (64 + 16)) + 3 * (size_t)max_seqs * pt_stride + 64;
}

size_t carve_kv(hvd_kv_s* k, const hvd_config& c, int max_seqs, int n_pages, void* base) {
  Carver cv(base);
  const size_t D = c.d_model, F = c.ffn_dim, qd = (size_t)c.n_q_heads * c.head_dim;
  k->page_stride = (size_t)2 * c.n_kv_heads * kPage * c.head_dim;
  k->layer_stride = k->page_stride * n_pages;
  k->pool = cv.take<_Float16>(k->layer_stride * c.n_layers);
  k->pt_stride = (c.max_pos + kPage) / kPage + 1;
  k->pt = cv.take<int32_t>((size_t)max_seqs * k->pt_stride);
  k->max_rows = std::max(max_seqs * (c.max_draft + 1), prefill_rows(c));
  k->MTmax = (k->max_rows + 15) / 16;
  const size_t Mp = (size_t)k->MTmax * 16;
  k->X = cv.take<float>(Mp * D);
  k->ss = cv.take<float>(Mp * (D / 16));
  // GEMM operands carry kGemmMaxMT extra fragments: a workgroup always reads
  // a full block of row tiles and drops the rows past the last tile
  const size_t pad = (size_t)kGemmPadMT * 512;
  k->Nhi = cv.take<uint16_t>(Mp * D + pad);
  k->Nlo = cv.take<uint16_t>(Mp * D + pad);
  k->Q = cv.take<_Float16>(Mp * qd);
  k->Ohi = cv.take<uint16_t>(Mp * qd + pad);
  k->Olo = cv.take<uint16_t>(Mp * qd + pad);
  k->Ahi = cv.take<uint16_t>(Mp * F + pad);
  k->Alo = cv.take<uint16_t>(Mp * F + pad);
  k->n_part_lm = c.vocab / 16;  // LM-head partials per row (upper bound: one per strip)
  k->lm_val = cv.take<float>(Mp * k->n_part_lm);
  k->lm_idx = cv.take<int32_t>(Mp * k->n_part_lm);
  k->gemm_part = cv.take<float>(kGemmPartBytes / 4);
  k->gemm_cnt = cv.take<uint32_t>(kGemmCounters);
  k->inv_rms = cv.take<float>(Mp);
  k->g = cv.take<int32_t>(Mp);
  // [B][2] results, then [B][63] tree paths, then an error word
  k->out = cv.take<int32_t>((2 + kMaxTreeNodes) * (size_t)max_seqs + 1);
  k->counter = cv.take<uint32_t>(64);
  k->part_o = cv.take<float>((size_t)kPartSlots * kAttnRows * c.head_dim);
  k->part_ml = cv.take<float>((size_t)kPartSlots * kAttnRows * 2);
  k->meta_ints = meta_capacity_ints(c, k->max_rows, max_seqs, k->pt_stride);
  k->meta_dev = cv.take<int32_t>(k->meta_ints);
  k->flow_layers = cv.take<FlowLayer>(c.n_layers);
  k->flow_cnt = cv.take<uint32_t>(kFlowCounterWords);
  // the one-launch step's per-layer activations (head dim 128 only), sized
  // for its largest batch: kFlowRows rows
  k->flow_host.assign(c.n_layers, FlowLayer{});
  if (c.head_dim == 128) {
    const size_t R = kFlowRows, fpad = (size_t)kGemmPadMT * 512;
    for (int l = 0; l < c.n_layers; ++l) {
      FlowLayer& f = k->flow_host[l];
      f.x_mid = cv.take<float>(R * D);
      f.x_out = cv.take<float>(R * D);
      f.n_mid_hi = cv.take<uint16_t>(R * D + fpad);
      f.n_mid_lo = cv.take<uint16_t>(R * D + fpad);
      f.n_out_hi = cv.take<uint16_t>(R * D + fpad);
      f.n_out_lo = cv.take<uint16_t>(R * D + fpad);
      f.ss_mid = cv.take<float>(R * (D / 16));
      f.ss_out = cv.take<float>(R * (D / 16));
      f.q = cv.take<_Float16>(R * qd);
      f.o_hi = cv.take<uint16_t>(R * qd + fpad);
      f.o_lo = cv.take<uint16_t>(R * qd + fpad);
      f.a_hi = cv.take<uint16_t>(R * F + fpad);
      f.a_lo = cv.take<uint16_t>(R * F + fpad);
      f.x_in = l ? k->flow_host[l - 1].x_out : k->X;
      f.n_in_hi = l ? k->flow_host[l - 1].n_out_hi : k->Nhi;
      f.n_in_lo = l ? k->flow_host[l - 1].n_out_lo : k->Nlo;
      f.ss_in = l ? k->flow_host[l - 1].ss_out : k->ss;
    }
  }
  k->sx.gemm_part = k->gemm_part;
  k->sx.gemm_part_bytes = kGemmPartBytes;
  k->sx.gemm_cnt = k->gemm_cnt;
  k->sx.flow_cnt = k->flow_cnt;
  k->sx.part_o = k->part_o;
  k->sx.part_ml = k->part_ml;
  k->sx.part_rows = (size_t)kPartSlots * kAttnRows;
  k->sx.lm_val = k->lm_val;
  k->sx.lm_idx = k->lm_idx;
  k->sx.inv_rms = k->inv_rms;
  k->sx.g = k->g;
  k->sx.out = k->out;
  k->sx.counter = k->counter;
  return cv.off;
}

}  // namespace

extern "C" size_t hvd_kv_bytes(const hvd_config* cfg, int32_t max_seqs, int32_t n_pages) {
  if (check_config(cfg) != HVD_OK || max_seqs < 1 || n_pages < 1) return 0;
  hvd_kv_s tmp;
  return carve_kv(&tmp, *cfg, max_seqs, n_pages, nullptr);
}

extern "C" hvd_status hvd_kv_alloc(hvd_model m, int32_t max_seqs, int32_t n_pages, void* dev_buf, size_t dev_bytes,
                                   void* stream, hvd_kv* out) {
  if (!m || !out) return set_err(HVD_ERR_ARG, "null model or out");
  if (max_seqs < 1 || n_pages < 1) return set_err(HVD_ERR_ARG, "max_seqs and n_pages must be >= 1");
  const hvd_config& c = m->cfg;
  auto* k = new hvd_kv_s();
  k->m = m;
  k->stream = (hipStream_t)stream;
  k->n_pages = n_pages;
  // The logit error of the fp16 path grows as the square root of depth;
  // deeper models keep gate/up on the hi + lo pair too (64 layers of the
  // 32B shape: whole-row error 2.7-2.9e-2 with gate/up single, 2.4e-2 with
  // the pair, against a 2.83e-2 bar)
  k->mlp_single_gu = c.n_layers <= kMlpSingleMaxLayers;
  const size_t need = carve_kv(k, c, max_seqs, n_pages, nullptr);
  if (dev_buf) {
    if (dev_bytes < need) {
      delete k;
      return set_err(HVD_ERR_ARG, "dev_buf smaller than hvd_kv_bytes");
    }
    k->base = dev_buf;
  } else {
    if (hipMalloc(&k->base, need) != hipSuccess) {
      delete k;
      return set_err(HVD_ERR_OOM, "hipMalloc of the KV pool failed");
    }
    k->owned = true;
  }
  carve_kv(k, c, max_seqs, n_pages, k->base);
  if (hipHostMalloc((void**)&k->meta_host, k->meta_ints * 4, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&k->out_host, ((2 + kMaxTreeNodes) * (size_t)max_seqs + 1) * 4, hipHostMallocDefault) !=
          hipSuccess) {
    if (k->meta_host) (void)hipHostFree(k->meta_host);
    if (k->owned) (void)hipFree(k->base);
    delete k;
    return set_err(HVD_ERR_OOM, "pinned host staging allocation failed");
  }
  if (hipHostGetDevicePointer((void**)&k->meta_host_dev, k->meta_host, 0) != hipSuccess) {
    (void)hipHostFree(k->meta_host);
    (void)hipHostFree(k->out_host);
    if (k->owned) (void)hipFree(k->base);
    delete k;
    return set_err(HVD_ERR_DEVICE, "device address of the pinned metadata staging failed");
  }
  // Zero the whole workspace once: padding rows of every operand stay finite.
  // (KV pages are zeroed too; their contents are only read once written.)
  if (hipMemsetAsync(k->base, 0, need, k->stream) != hipSuccess || hipStreamSynchronize(k->stream) != hipSuccess) {
    (void)hipHostFree(k->meta_host);
    (void)hipHostFree(k->out_host);
    if (k->owned) (void)hipFree(k->base);
    delete k;
    return set_err(HVD_ERR_DEVICE, "workspace clear failed");
  }
  {
    // the one-launch step's table of per-layer weights, gains and KV pools
    std::vector<FlowLayer>& fl = k->flow_host;
    for (int l = 0; l < c.n_layers; ++l) {
      const LayerW& L = m->layers[l];
      fl[l].qkv = (const uint4*)L.qkv;
      fl[l].o = (const uint4*)L.o;
      fl[l].gu = (const uint4*)L.gu;
      fl[l].down = (const uint4*)L.down;
      fl[l].g_attn = L.g_attn;
      fl[l].g_mlp = L.g_mlp;
      fl[l].kv = k->pool + (size_t)l * k->layer_stride;
    }
    if (hipMemcpyAsync(k->flow_layers, fl.data(), fl.size() * sizeof(FlowLayer), hipMemcpyHostToDevice, k->stream) !=
            hipSuccess ||
        hipStreamSynchronize(k->stream) != hipSuccess) {
      (void)hipHostFree(k->meta_host);
      (void)hipHostFree(k->out_host);
      if (k->owned) (void)hipFree(k->base);
      delete k;
      return set_err(HVD_ERR_DEVICE, "layer table upload failed");
    }
  }
  k->hs = new HostState(max_seqs, n_pages, kPage, c.max_pos, c.max_draft, c.vocab);
  if (hipError_t e = attn_set_lds_limit(); e != hipSuccess) {
    hvd_kv_free(k);
    return set_err(HVD_ERR_DEVICE, std::string("attention LDS limit: ") + hipGetErrorString(e));
  }
  if (hipError_t e = flow_set_lds_limit(); e != hipSuccess) {
    hvd_kv_free(k);
    return set_err(HVD_ERR_DEVICE, std::string("one-launch step LDS limit: ") + hipGetErrorString(e));
  }
  if (hipError_t e = attn_o_set_lds_limit(); e != hipSuccess) {
    hvd_kv_free(k);
    return set_err(HVD_ERR_DEVICE, std::string("attention + O launch LDS limit: ") + hipGetErrorString(e));
  }
  {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      hvd_kv_free(k);
      return set_err(HVD_ERR_DEVICE, "device attribute query failed");
    }
    k->n_cus = cus;
  }

  // this device's static scratch (hvd_verify_noalloc): its address is taken
  // here, once per device, with the device current
  if (hipError_t e = static_scratch(&k->static_base, &k->static_bytes); e != hipSuccess) {
    hvd_kv_free(k);
    return set_err(HVD_ERR_DEVICE, std::string("static scratch address: ") + hipGetErrorString(e));
  }
  *out = k;
  return HVD_OK;
}

extern "C" void hvd_kv_free(hvd_kv k) {
  if (!k) return;
  for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);
  for (auto e : k->ev_pool) (void)hipEventDestroy(e);
  for (auto& r : k->prof_pending) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  if (k->meta_host) (void)hipHostFree(k->meta_host);
  if (k->out_host) (void)hipHostFree(k->out_host);
  if (k->owned && k->base) (void)hipFree(k->base);
  delete k->hs;
  delete k;
}

// ------------------------------------------------------------------ forward

namespace {

hipEvent_t take_event(hvd_kv_s* k) {
  if (!k->ev_pool.empty()) {
    hipEvent_t e = k->ev_pool.back();
    k->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  (void)hipEventCreate(&e);
  return e;
}

// Bracket one launch with events when profiling.
struct ProfScope {
  hvd_kv_s* k;
  ProfRec r{};
  ProfScope(hvd_kv_s* k_, int family, double bytes) : k(k_) {
    if (!k->prof) return;
    r.a = take_event(k);
    r.b = take_event(k);
    r.family = family;
    r.bytes = bytes;
    tl_timing = LaunchTiming{r.a, r.b};  // the role's kernels record the events
  }
  ~ProfScope() {
    if (!k->prof) return;
    tl_timing = LaunchTiming{};
    k->prof_pending.push_back(r);
  }
};

void prof_collect(hvd_kv_s* k) {
  for (auto& r : k->prof_pending) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      k->prof_ms[r.family] += ms;
      k->prof_n[r.family] += 1;
      k->prof_bytes[r.family] += r.bytes;
    }
    k->ev_pool.push_back(r.a);
    k->ev_pool.push_back(r.b);
  }
  k->prof_pending.clear();
}

struct Plan {
  std::vector<AttnItem> items, heads;
  int chunk = 0;
  int rpi = 0;             // query rows per item
  int comb_rows = 1;       // rows of the largest combine entry
  size_t part_rows = 0;    // partial-buffer rows the plan uses
  size_t part_base = 0;    // its first partial-buffer row
  size_t item0 = 0, head0 = 0;  // offsets of its items and entries in the step's lists
  int n_items_real = 0, n_heads_real = 0;  // before grid padding
};

// Split every (sequence, kv head, row group) of the sequences `members` into
// KV chunks of `chunk` positions, chosen so the launch has enough workgroups
// to fill the GPU; at most part_rows_free partial-buffer rows.
bool plan_attention(const hvd_config& c, const HostState& hs, const std::vector<SeqMeta>& seqs,
                    const std::vector<int>& members, int min_items, int rpi, size_t part_rows_free, Plan& p,
                    int max_items = 0) {
  const int G = c.n_q_heads / c.n_kv_heads;
  struct Unit { int b, g, rg, keys; };
  auto item = [&](const Unit& u, int ci, int nch, int part, int chunk) {
    const SeqMeta& s = seqs[u.b];
    AttnItem it{};
    it.slot = s.slot; it.ctx = s.ctx; it.k = s.k; it.cu = s.cu; it.tree = s.tree;
    it.g = u.g; it.c = ci; it.nch = nch; it.rg = u.rg; it.part = part;
    it.p_begin = ci * chunk;
    it.p_end = std::min(s.ctx + s.k + 1, (ci + 1) * chunk);
    it.pad1 = u.b;                // for a device-side re-plan at another ctx:
    it.pad2 = u.keys - s.ctx - 1;  // sequence, last row index of the unit,
    it.pad3 = chunk;               // chunk length
    // pages of the first kAttnChunk positions; entries past the chunk's end
    // repeat its first page (the kernel loads them unconditionally)
    const std::vector<int32_t>& pg = hs.seq(s.slot).pages;
    const int first = it.p_begin / kPage;
    for (int j = 0; j < kItemPages; ++j) {
      const bool in = it.p_begin + j * kPage < it.p_end;
      it.pages[j] = pg[(size_t)(in ? first + j : first)];
    }
    return it;
  };
  std::vector<Unit> units;
  int64_t total_keys = 0;
  for (int b : members) {
    const SeqMeta& s = seqs[b];
    const int R = (s.k + 1) * G;
    const int n_rg = (R + rpi - 1) / rpi;
    for (int g = 0; g < c.n_kv_heads; ++g)
      for (int rg = 0; rg < n_rg; ++rg) {
        const int i_max = std::min(s.k, ((rg + 1) * rpi - 1) / G);
        const int keys = s.ctx + i_max + 1;
        units.push_back({b, g, rg, keys});
        total_keys += keys;
      }
  }
  // chunk: a power-of-two number of positions, the largest that still gives
  // every CU work -- two 64-row items per CU (4 waves: several share a CU),
  // one item of 128 rows or more (8 waves) -- with at least 64 positions for
  // 64-row items and at most 1024 for the others.  Longer chunks loop over
  // LDS-sized sub-chunks.  Measured: 32 sequences of mixed drafts 34.2 ->
  // 33.2 ms per step; context 16384 at k = 16 / 64 from 4.98 / 9.04 to
  // 4.71 / 8.70 ms (chunks of at most 256 before); 1024 instead of 512 for
  // 256- and 384-row items (fewer partials to write and merge): the 848-row
  // batch 32.4 -> 31.9 ms, the 32B multistep step 62.5 -> 61.3 ms (2048 or
  // 4096: 61.9 ms); more workgroups per CU (384 or 512 targets) measured
  // slower
  const int per_cu = rpi <= kAttnRows / 2 ? 2 : 1;
  const int64_t want = (total_keys + (int64_t)min_items * per_cu - 1) / ((int64_t)min_items * per_cu);
  const int cap = rpi <= kAttnRows / 2 ? (1 << 20) : 1024;
  int chunk = rpi <= kAttnRows / 2 ? 64 : 32;
  while (chunk < cap && 2 * chunk <= want) chunk *= 2;
  if (max_items > 0) {
    // the shortest power-of-two chunk that keeps the items within max_items
    auto n_items_at = [&](int ch) {
      int64_t n = 0;
      for (const Unit& u : units) n += (u.keys + ch - 1) / ch;
      return n;
    };
    chunk = 32;
    while (chunk < (1 << 20) && n_items_at(chunk) > max_items) chunk *= 2;
  }
  // Several row groups of one (sequence, kv head) read the same K/V chunks.
  // Their items go 8 grid positions apart, next to each other in dispatch
  // order: the same XCD under round-robin dispatch, at nearly the same time,
  // so a chunk comes from HBM once and from that XCD's L2 for the others.
  // Per (sequence, kv head) with n_rg > 1 row groups, chunks in runs of 8:
  // item (run position j, row group r) at run base + 8r + j, a no-op item
  // (k = -1) where a row group has fewer chunks.  Partial slots and merge
  // entries follow the units in order, as with one row group.
  AttnItem none{};
  none.k = -1;
  std::vector<int> nch_u, slot_u;
  for (;;) {
    p.items.clear();
    p.heads.clear();
    nch_u.assign(units.size(), 0);
    slot_u.assign(units.size(), -1);
    int slots = 0;
    for (size_t i = 0; i < units.size(); ++i) {
      const Unit& u = units[i];
      const int nch = (u.keys + chunk - 1) / chunk;
      nch_u[i] = nch;
      if (nch > 1) {
        slot_u[i] = slots;
        p.heads.push_back(item(u, 0, nch, slots, chunk));
        slots += nch;
      }
    }
    for (size_t i0 = 0; i0 < units.size();) {
      size_t i1 = i0 + 1;  // units [i0, i1): the row groups of one (sequence, kv head)
      while (i1 < units.size() && units[i1].b == units[i0].b && units[i1].g == units[i0].g) ++i1;
      auto emit = [&](size_t i, int ci) {
        const int nch = nch_u[i];
        if (ci >= nch) p.items.push_back(none);
        else p.items.push_back(nch == 1 ? item(units[i], 0, 1, -1, chunk) : item(units[i], ci, nch, slot_u[i] + ci, chunk));
      };
      if (i1 - i0 == 1) {
        for (int ci = 0; ci < nch_u[i0]; ++ci) emit(i0, ci);
      } else {
        int max_nch = 0;
        for (size_t i = i0; i < i1; ++i) max_nch = std::max(max_nch, nch_u[i]);
        for (int c0 = 0; c0 < max_nch; c0 += 8) {
          const int run = std::min(8, max_nch - c0);
          for (size_t i = i0; i < i1; ++i)
            for (int j = 0; j < run; ++j) emit(i, c0 + j);
        }
      }
      i0 = i1;
    }
    if ((size_t)slots * rpi <= part_rows_free) {  // partial buffer rows
      p.part_rows = (size_t)slots * rpi;
      break;
    }
    if (chunk >= (1 << 20)) return false;
    // longer chunks: multiples of kAttnChunk above it (looped in LDS-sized pieces)
    chunk = chunk < kAttnChunk ? std::min(kAttnChunk, chunk * 2) : chunk * 2;
  }
  p.chunk = chunk;
  p.rpi = rpi;
  int max_r = 1;
  for (int b : members) max_r = std::max(max_r, (seqs[b].k + 1) * G);
  p.comb_rows = std::min(rpi, max_r);
  return true;
}

// rows[].kvs holds each row's K/V position on entry; tree (optional): per
// row, the ancestor mask over positions ctx.. and the parent node.
struct TreeRows {
  std::vector<uint64_t> mask;
  std::vector<int32_t> parent;
};

// A device-resident loop's step, captured instead of run: the metadata
// (planned for the longest context the loop reaches) goes once to a device
// block of the loop's own, and the captured launches start with the
// device-side re-plan and end with the on-device commit.
struct AsyncCap {
  int32_t* drafts = nullptr;
  int32_t* state = nullptr;
  int32_t* hist = nullptr;
  int hist_cap = 0;
  const int32_t* ref = nullptr;
  int ref_len = 0;
  std::vector<int32_t> ref_start;  // [B]
  std::vector<int32_t> page_off;   // [B + 1]
  std::vector<int32_t> pages;      // reserved pages, concatenated
  int32_t* meta = nullptr;         // out: device metadata block (hipMalloc)
  hipGraphExec_t graph = nullptr;  // out
};

hvd_status forward(hvd_kv_s* k, const std::vector<SeqMeta>& seqs, std::vector<RowMeta> rows, bool lm_head,
                   float* logits, const TreeRows* tree = nullptr, AsyncCap* acap = nullptr,
                   const StepScratch* scratch = nullptr) {
  const StepScratch& sx = scratch ? *scratch : k->sx;
  const bool eager_only = scratch != nullptr;  // no graph instantiation (it allocates)
  // each row's pool slot: page * kPage + offset (the QKV epilogue writes K/V there)
  for (RowMeta& r : rows) r.kvs = k->hs->seq(r.slot).pages[(size_t)(r.kvs / kPage)] * kPage + r.kvs % kPage;
  hvd_model_s* m = k->m;
  const hvd_config& c = m->cfg;
  hipStream_t s = k->stream;
  const int M = (int)rows.size();
  const int MT = (M + 15) / 16;
  if (MT > k->MTmax) return set_err(HVD_ERR_OOM, "row workspace too small");
  const int B = (int)seqs.size();
  const int D = c.d_model, F = c.ffn_dim, dh = c.head_dim, qd = c.n_q_heads * dh, kvd = c.n_kv_heads * dh;
  const int G = c.n_q_heads / c.n_kv_heads;

  // Attention row classes: each sequence's (k + 1) * group query rows per kv
  // head go to items of 64, 128 or 256 rows (256 for head dim 128 only;
  // longer row sets take several row groups), one launch per class, so a
  // long draft does not put every short one on the large kernel.
  static const int kClassRows[kAttnClasses] = {kAttnRows / 2, kAttnRows, 2 * kAttnRows, 3 * kAttnRows};
  // One-launch step (flow.hip): verify batches of at most two row tiles,
  // head dim 128, every sequence's query rows per kv head in one 128-row
  // attention item; chain drafts only, outside a device-resident loop.
  bool flow = k->use_flow && lm_head && !tree && !acap && MT * 16 <= kFlowRows && dh == 128;
  for (int b = 0; b < B && flow; ++b) flow = (seqs[b].k + 1) * G <= kAttnRows;
  // Attention + merge + O GEMM as one launch (attn_o.hip): up to two row
  // tiles, head dim 128, an O GEMM of K = 4096 with at most one strip per CU;
  // every sequence's rows in 128-row items.
  const bool attn_o = !flow && k->use_attn_o && lm_head && !acap && (MT == 1 || MT == 2) &&
                      attn_o_supported(dh, 2, MT, qd / 32, D / 16, k->n_cus);
  // the attention workgroups of that launch: the CUs' second slots beside the O strips
  const int ao_attn_wgs = attn_o ? std::min(2 * k->n_cus - D / 16, k->n_cus) : 0;
  // Above 256 rows, 384-row items (three row tiles per wave) when 256-row
  // items would leave a last row group of at most 64 rows -- a whole pass
  // over the keys for a few rows -- and the 384-row items need fewer passes
  // (260 rows: one, not two).  Otherwise the 256-row items are faster per
  // row (measured: 32B multistep steps 15.5-17.8 -> 17.1-17.9 ms of
  // attention with 384-row items for every sequence they save a pass on).
  std::vector<int> members[kAttnClasses];
  int ao_rpi = kAttnRows / 2;  // attention + O launch: 64-row items unless a sequence has more rows
  for (int b = 0; b < B; ++b) {
    const int R = (seqs[b].k + 1) * G;
    if (R > kAttnRows / 2) ao_rpi = kAttnRows;
    // head dim 128: up to 128 rows in 64-row items (two row groups at 65-128
    // rows: the 4-wave items share a CU two at a time; measured at k = 16,
    // 68 rows: 12.6 -> 8.6 us per layer against one 128-row item)
    int cl = (R <= kClassRows[0] || (R <= kClassRows[1] && dh == 128)) ? 0 : (R <= kClassRows[1] || dh != 128) ? 1 : 2;
    if (cl == 2 && (R - 1) % kClassRows[2] < kClassRows[0] &&
        (R + kClassRows[3] - 1) / kClassRows[3] < (R + kClassRows[2] - 1) / kClassRows[2])
      cl = 3;
    members[flow || attn_o ? 1 : cl].push_back(b);
  }
  Plan plans[kAttnClasses];
  std::vector<AttnItem> items_all, heads_all;
  std::array<int, 4 * kAttnClasses> attn_key{};
  size_t part_used = 0;
  for (int cl = 0; cl < kAttnClasses; ++cl) {
    if (members[cl].empty()) continue;
    Plan& pl = plans[cl];
    if (!plan_attention(c, *k->hs, seqs, members[cl], flow ? k->flow_min_items : k->attn_min_items,
                        attn_o ? ao_rpi : kClassRows[cl], sx.part_rows - part_used, pl,
                        attn_o ? ao_attn_wgs : 0))
      return set_err(HVD_ERR_OOM, "attention partial slots exhausted");
    pl.part_base = part_used;
    part_used += pl.part_rows;
    pl.n_items_real = (int)pl.items.size();
    pl.n_heads_real = (int)pl.heads.size();
    if (flow) {
      // merge unit of each multi-chunk item: the index of its merge entry
      std::map<int, int> unit_of_slot;
      for (size_t h = 0; h < pl.heads.size(); ++h) {
        pl.heads[h].pad4 = (int32_t)h;
        unit_of_slot[pl.heads[h].part] = (int)h;
      }
      for (AttnItem& it : pl.items)
        if (it.nch > 1) it.pad4 = unit_of_slot[it.part - it.c];
    }
    // Pad the grids to buckets (no-op items have k = -1) so the launch
    // sequence depends only on (rows, sequences, buckets): one cached HIP
    // graph per such shape.
    AttnItem none{};
    none.k = -1;
    pl.items.resize((pl.items.size() + 63) / 64 * 64, none);
    pl.heads.resize((pl.heads.size() + 15) / 16 * 16, none);
    pl.item0 = items_all.size();
    pl.head0 = heads_all.size();
    items_all.insert(items_all.end(), pl.items.begin(), pl.items.end());
    heads_all.insert(heads_all.end(), pl.heads.begin(), pl.heads.end());
    attn_key[4 * cl] = (int)pl.items.size();
    attn_key[4 * cl + 1] = (int)pl.heads.size();
    attn_key[4 * cl + 2] = pl.chunk;
    attn_key[4 * cl + 3] = pl.comb_rows;
  }
  const size_t n_items = items_all.size(), n_heads = heads_all.size();
  std::vector<PageUpdate> upd_raw = k->hs->take_updates();
  // keep the last update of each (slot, index): they are applied in parallel
  std::map<std::pair<int, int>, int> last;
  for (auto& u : upd_raw) last[{u.slot, u.index}] = u.page;

  // pack metadata: header | rows | seqs | items | heads | updates (a
  // device-resident loop adds its static copies after them)
  std::vector<int32_t> ameta;
  if (acap)
    ameta.resize(16 + 4 * (size_t)M + sizeof(SeqMeta) / 4 * 2 * (size_t)B + 64 * (n_items + n_heads) +
                 3 * (size_t)M + 3 * last.size() + M + 2 * B + 1 + acap->pages.size() + 80);
  int32_t* h = acap ? ameta.data() : k->meta_host;
  size_t off = 0;
  auto put = [&](const void* src, size_t ints) {
    if (ints) std::memcpy(h + off, src, ints * 4);
    size_t o = off;
    off += (ints + 3) / 4 * 4;
    return o;
  };
  const size_t need_ints = 16 + 4 * (size_t)M + sizeof(SeqMeta) / 4 * (size_t)B + 32 * (n_items + n_heads) +
                           3 * (size_t)M + 3 * last.size() + 40;
  if (!acap && need_ints > k->meta_ints) {
    k->hs->take_updates();
    return set_err(HVD_ERR_OOM, "metadata buffer too small");
  }
  int32_t header[16] = {(int32_t)last.size()};
  put(header, 16);
  const size_t o_rows = put(rows.data(), 4 * (size_t)M);
  const size_t o_seqs = put(seqs.data(), sizeof(SeqMeta) / 4 * (size_t)B);
  const size_t o_items = put(items_all.data(), sizeof(AttnItem) / 4 * n_items);
  const size_t o_heads = put(heads_all.data(), sizeof(AttnItem) / 4 * n_heads);
  // tree rows (fixed size per M, before the variable-length updates so every
  // offset a captured graph holds depends on the graph key only)
  off = (off + 7) / 8 * 8;  // 8-byte alignment of the masks
  size_t o_mask = 0, o_parent = 0;
  if (tree) {
    o_mask = put(tree->mask.data(), 2 * (size_t)M);
    o_parent = put(tree->parent.data(), (size_t)M);
  }
  std::vector<int32_t> upd;
  for (auto& kv : last) {
    upd.push_back(kv.first.first);
    upd.push_back(kv.first.second);
    upd.push_back(kv.second);
  }
  const size_t o_upd = put(upd.data(), upd.size());
  size_t o_sitems = 0, o_sheads = 0, o_sseqs = 0, o_rowseq = 0, o_pgoff = 0, o_pages = 0, o_rstart = 0;
  if (acap) {
    o_sitems = put(items_all.data(), sizeof(AttnItem) / 4 * n_items);
    o_sheads = put(heads_all.data(), sizeof(AttnItem) / 4 * n_heads);
    o_sseqs = put(seqs.data(), sizeof(SeqMeta) / 4 * (size_t)B);
    std::vector<int32_t> row_seq(M);
    for (int b = 0; b < B; ++b)
      for (int i = 0; i <= seqs[b].k; ++i) row_seq[seqs[b].cu + i] = b;
    o_rowseq = put(row_seq.data(), M);
    o_pgoff = put(acap->page_off.data(), B + 1);
    o_pages = put(acap->pages.data(), acap->pages.size());
    o_rstart = put(acap->ref_start.data(), B);
    if (off > ameta.size()) return set_err(HVD_ERR_OOM, "loop metadata block too small");
    if (hipMalloc((void**)&acap->meta, off * 4) != hipSuccess) {
      acap->meta = nullptr;
      return set_err(HVD_ERR_OOM, "hipMalloc of the loop metadata failed");
    }
  }
  int32_t* const meta_dev = acap ? acap->meta : k->meta_dev;
  if (acap) HIP_TRY(hipMemcpyAsync(meta_dev, h, off * 4, hipMemcpyHostToDevice, s));
  else HIP_TRY(launch_copy_words(meta_dev, k->meta_host_dev, off, s));  // the previous step has finished with it
  if (acap) {
    // the page-table updates are applied once, here; the replays carry none
    // (replaying them could undo later updates of other sequences)
    static const int32_t zero = 0;
    HIP_TRY(launch_pt_update(meta_dev + o_upd, meta_dev, k->pt, k->pt_stride, s));
    HIP_TRY(hipMemcpyAsync(meta_dev, &zero, 4, hipMemcpyHostToDevice, s));
    HIP_TRY(hipStreamSynchronize(s));  // the staging vector goes out of scope
  }
  const RowMeta* d_rows = (const RowMeta*)(meta_dev + o_rows);
  const SeqMeta* d_seqs = (const SeqMeta*)(meta_dev + o_seqs);
  const AttnItem* d_items = (const AttnItem*)(meta_dev + o_items);
  const AttnItem* d_heads = (const AttnItem*)(meta_dev + o_heads);
  const uint64_t* d_mask = tree ? (const uint64_t*)(meta_dev + o_mask) : nullptr;
  const int32_t* d_parent = tree ? meta_dev + o_parent : nullptr;

  // skinny GEMMs: row blocks of at most kGemmMaxMT tiles, balanced
  const int mblocks = (MT + kGemmMaxMT - 1) / kGemmMaxMT;
  const int mt_block = (MT + mblocks - 1) / mblocks;
  // Strips per workgroup and K splits of the weight-streaming GEMM (measured
  // on the 8B verify shapes): 4 strips per workgroup when that alone gives
  // enough workgroups (8 for two row tiles, which halves the activation
  // fragments per weight byte); for long-K GEMMs 4 strips plus a K split
  // (2 strips and a two-way split at up to 8 rows);
  // otherwise 2 strips, or for one row tile 1 strip when that fills the GPU;
  // K-split if still too few.
  auto skinny_shape = [&](int epi, int N, int K, int family, bool single, int mblocks, int mt_block, int& ns,
                          int& splits) {
    const int nb8 = N / 128 * mblocks, nb4 = N / 64 * mblocks, nb2 = N / 32 * mblocks;
    const int KT = K / 32, NT = N / 16;
    const int want = k->gemm_min_blocks;
    ns = 4;
    splits = 1;
    // 8 strips per workgroup halve the activation fragments per weight byte:
    // two row tiles, or three and four on the single-pass activation
    if ((mt_block == 2 || (mt_block >= 3 && (mt_block <= 4 || epi == EPI_SILU || epi == EPI_LM) && single && k->ns8_mt3)) &&
        N % 128 == 0 && nb8 >= want) {
      ns = 8;
    } else if (nb4 >= want) {
      ns = 4;
    } else if (KT >= kGemmLongK && mt_block == 1 && mblocks == 1 && M <= 8 && nb2 * 2 >= want) {
      // up to 8 live rows: each activation fragment reads one line per 16-lane
      // group, so two strips with a two-way split beat four strips with a
      // four-way split (down, 8B shape: 23.1 -> 22.2 us per layer at 2-8
      // rows; at 9-16 rows 24.5 against 23.7, so those keep four strips)
      ns = 2;
      splits = 2;
    } else if (KT >= kGemmLongK) {
      ns = 4;
      splits = std::max(1, std::min((kGemmSplitTarget + nb4 - 1) / nb4, KT / 64));
    } else if (nb2 >= want) {
      ns = 2;
    } else if (mt_block == 1 && epi != EPI_SILU && nb2 * 2 >= want) {
      ns = 1;  // one strip per workgroup beats a K split plus its reduction
    } else {
      ns = 2;
      splits = std::max(1, std::min((kGemmSplitTarget + nb2 - 1) / nb2, KT / 64));
    }
    if (family <= PF_LM && k->gemm_force[family][0]) {
      const int fns = k->gemm_force[family][0];
      const bool ok = NT % fns == 0 && !(fns == 1 && epi == EPI_SILU) && !(fns == 8 && (mt_block > 2 || N % 128));
      if (ok) {
        ns = fns;
        splits = std::min(k->gemm_force[family][1], KT);
      }
    }
    while (splits > 1 && (size_t)(N / 16) * 16 * splits * mt_block * 16 * mblocks * 4 > sx.gemm_part_bytes) --splits;
    if (splits > 1 && (size_t)(NT / ns) * mblocks > (size_t)kGemmCounters) splits = 1;
  };
  // ---------------------------------------------------------------- one-launch step
  // counter layout per layer: QKV groups, merge units, then four 8-way counters
  const Plan& fpl = plans[1];
  const int flow_cstride = flow ? (c.n_kv_heads + 7) / 8 * 8 + (fpl.n_heads_real + 7) / 8 * 8 + 32 : 0;
  const int flow_words = flow ? 8 + c.n_layers * flow_cstride : 0;
  if (flow && flow_words > kFlowCounterWords) flow = false;  // (not reached for the supported shapes)
  auto launch_flow_step = [&]() -> hvd_status {
    const int qd2 = qd + 2 * kvd;
    FlowArgs f{};
    f.layers = k->flow_layers;
    f.L = c.n_layers;
    f.g_final = m->g_final;
    f.G = G;
    f.dh = dh;
    const int Ns[FG_N] = {qd2, D, 2 * F, D, c.vocab}, Ks[FG_N] = {D, qd, D, F, D};
    const int epis[FG_N] = {EPI_QKV, EPI_RESID, EPI_SILU, EPI_RESID, EPI_LM};
    const int fams[FG_N] = {PF_QKV, PF_O, PF_GATEUP, PF_DOWN, PF_LM};
    for (int i = 0; i < FG_N; ++i) {
      GemmArgs& a = f.g[i];
      a.KT = Ks[i] / 32;
      a.NT = Ns[i] / 16;
      a.wg = (size_t)a.KT * 256;
      a.wk = 256;
      a.MTtot = MT;
      a.M = M;
      a.part = sx.gemm_part;
      a.cnt = sx.gemm_cnt;
      int ns = 4, splits = 1;
      skinny_shape(epis[i], Ns[i], Ks[i], fams[i], false, mblocks, mt_block, ns, splits);
      if (ns == 8) ns = 4;  // the one-launch step compiles 1, 2 and 4 strips
      f.ns[i] = ns;
      f.splits[i] = splits;
      f.n_cb[i] = a.NT / ns;
    }
    {
      GemmArgs& a = f.g[FG_QKV];
      a.Ahi = (const uint4*)k->Nhi;
      a.Alo = (const uint4*)k->Nlo;
      a.ss = k->ss;
      a.ss_n = D / 16;
      a.inv_dim = 1.f / D;
      a.eps = c.rms_eps;
      a.Q = k->Q;
      a.page_stride = k->page_stride;
      a.q_cols = qd;
      a.kv_cols = kvd;
      a.Hkv = c.n_kv_heads;
      a.dh = dh;
      a.pt = k->pt;
      a.pt_stride = k->pt_stride;
      a.rows = d_rows;
      a.rope = m->rope;
    }
    for (int i : {FG_O, FG_DOWN}) {
      GemmArgs& a = f.g[i];
      a.Ahi = (const uint4*)(i == FG_O ? k->Ohi : k->Ahi);
      a.Alo = (const uint4*)(i == FG_O ? k->Olo : k->Alo);
      a.X = k->X;
      a.D = D;
      a.Nhi = k->Nhi;
      a.Nlo = k->Nlo;
      a.ss_out = k->ss;
    }
    for (int i : {FG_GU, FG_LM}) {
      GemmArgs& a = f.g[i];
      a.Ahi = (const uint4*)k->Nhi;
      a.Alo = (const uint4*)k->Nlo;
      a.ss = k->ss;
      a.ss_n = D / 16;
      a.inv_dim = 1.f / D;
      a.eps = c.rms_eps;
    }
    f.g[FG_GU].act_hi = k->Ahi;
    f.g[FG_GU].act_lo = k->Alo;
    f.g[FG_LM].W = (const uint4*)m->lm;  // (the layer GEMMs take W from the layer table)
    f.g[FG_LM].logits = logits;
    f.g[FG_LM].vocab = c.vocab;
    f.g[FG_LM].part_val = sx.lm_val;
    f.g[FG_LM].part_idx = sx.lm_idx;
    f.g[FG_LM].n_part = f.n_cb[FG_LM];
    // attention (one 128-row class) and its merge
    AttnArgs& at = f.attn;
    at.Q = k->Q;
    at.page_stride = k->page_stride;
    at.Hq = c.n_q_heads;
    at.Hkv = c.n_kv_heads;
    at.dh = dh;
    at.group = G;
    at.pt = k->pt;
    at.pt_stride = k->pt_stride;
    at.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)dh));
    at.Ohi = k->Ohi;
    at.Olo = k->Olo;
    at.MTtot = MT;
    at.part_o = sx.part_o + fpl.part_base * dh;
    at.part_ml = sx.part_ml + fpl.part_base * 2;
    CombineArgs& cb = f.comb;
    cb.heads = d_heads + fpl.head0;
    cb.Hq = c.n_q_heads;
    cb.Hkv = c.n_kv_heads;
    cb.dh = dh;
    cb.group = G;
    cb.part_o = at.part_o;
    cb.part_ml = at.part_ml;
    cb.Ohi = k->Ohi;
    cb.Olo = k->Olo;
    cb.MTtot = MT;
    cb.rpi = fpl.rpi;
    cb.max_rows = fpl.comb_rows;
    f.np = std::max(2, std::min(4, attn_pages_per_sub(fpl.chunk)));
    f.items = d_items + fpl.item0;
    f.heads = d_heads + fpl.head0;
    constexpr int kMergeRows = 512 / (128 / 8 * 4);  // rows per merge slice (combine_slice<128, 4, 512>)
    f.merge_spb = (fpl.comb_rows + kMergeRows - 1) / kMergeRows;
    int n_single = 0;
    for (int i = 0; i < fpl.n_items_real; ++i) n_single += fpl.items[i].nch == 1;
    f.oin_target = (uint32_t)(n_single + fpl.n_heads_real * f.merge_spb);
    f.qkv_group_target = (uint32_t)((G * dh + 2 * dh) / (16 * f.ns[FG_QKV]));
    // phases of a layer
    f.ph[FL_QKV] = 0;
    f.ph[FL_ATTN] = f.n_cb[FG_QKV] * f.splits[FG_QKV];
    f.ph[FL_MERGE] = f.ph[FL_ATTN] + fpl.n_items_real;
    f.ph[FL_O] = f.ph[FL_MERGE] + fpl.n_heads_real * f.merge_spb;
    f.ph[FL_GU] = f.ph[FL_O] + f.n_cb[FG_O] * f.splits[FG_O];
    f.ph[FL_DOWN] = f.ph[FL_GU] + f.n_cb[FG_GU] * f.splits[FG_GU];
    f.ph[FL_PHASES] = f.ph[FL_DOWN] + f.n_cb[FG_DOWN] * f.splits[FG_DOWN];
    f.per_layer = f.ph[FL_PHASES];
    f.n_lm = f.n_cb[FG_LM] * f.splits[FG_LM];
    f.err = sx.flow_cnt;
    if (k->flow_trace && (int64_t)4 * (c.n_layers * f.per_layer + f.n_lm) <= k->flow_trace_words)
      f.trace = k->flow_trace;
    f.cnt = sx.flow_cnt + 8;
    f.cstride = flow_cstride;
    f.c_unit = (c.n_kv_heads + 7) / 8 * 8;
    f.c_oin = f.c_unit + (fpl.n_heads_real + 7) / 8 * 8;
    f.c_o = f.c_oin + 8;
    f.c_gu = f.c_o + 8;
    f.c_down = f.c_gu + 8;
    {
      double bytes = 2.0 * ((double)c.n_layers * ((double)qd2 * D + (double)D * qd + 2.0 * F * D + (double)D * F) +
                            (double)c.vocab * D);
      for (int b = 0; b < B; ++b) bytes += (double)(seqs[b].ctx + seqs[b].k + 1) * kvd * 2 * 2 * c.n_layers;
      ProfScope ps(k, PF_FLOW, bytes);
      HIP_TRY(launch_flow(f, MT, s));
    }
    AcceptArgs ac{};
    ac.part_val = sx.lm_val;
    ac.part_idx = sx.lm_idx;
    ac.n_part = f.n_cb[FG_LM];
    ac.M = M;
    ac.g = sx.g;
    ac.seqs = d_seqs;
    ac.rows = d_rows;
    ac.B = B;
    ac.out = sx.out;
    ac.counter = sx.counter;
    ac.path = sx.out + 2 * B;
    ac.err_word = sx.flow_cnt;
    ac.err_index = 2 * B;
    ProfScope ps(k, PF_OTHER, 0.0);
    HIP_TRY(launch_accept(ac, s));
    return HVD_OK;
  };

  // ---------------------------------------------------------------- launches
  // Everything below only enqueues kernels whose arguments are fixed by
  // the GraphKey fields: captured once per shape into
  // a HIP graph and replayed (eager while profiling or with graphs off).
  auto launch_all = [&]() -> hvd_status {
  if (acap) {
    AsyncPlanArgs p{};
    p.state = acap->state;
    p.drafts = acap->drafts;
    p.ref = acap->ref;
    p.ref_len = acap->ref_len;
    p.ref_start = meta_dev + o_rstart;
    p.seq_static = (const SeqMeta*)(meta_dev + o_sseqs);
    p.page_off = meta_dev + o_pgoff;
    p.pages = meta_dev + o_pages;
    p.row_seq = meta_dev + o_rowseq;
    p.rows = (RowMeta*)(meta_dev + o_rows);
    p.seqs = (SeqMeta*)(meta_dev + o_seqs);
    p.items_static = (const AttnItem*)(meta_dev + o_sitems);
    p.items = (AttnItem*)(meta_dev + o_items);
    p.n_items = (int)n_items;
    p.heads_static = (const AttnItem*)(meta_dev + o_sheads);
    p.heads = (AttnItem*)(meta_dev + o_heads);
    p.n_heads = (int)n_heads;
    p.M = M;
    p.B = B;
    HIP_TRY(launch_async_plan(p, s));
  }
  {
    EmbedArgs e{};
    e.E = m->embed;
    e.rows = d_rows;
    e.M = M;
    e.Mpad = MT * 16;
    e.D = D;
    e.gain = m->layers[0].g_attn;
    e.X = k->X;
    e.Nhi = k->Nhi;
    e.Nlo = k->Nlo;
    e.ss_out = k->ss;
    e.MTtot = MT;
    e.upd = meta_dev + o_upd;
    e.n_upd = meta_dev;  // header[0]
    e.pt = k->pt;
    e.pt_stride = k->pt_stride;
    e.V = c.vocab;
    if (flow) {  // the one-launch step's error word and counters start at zero
      e.zero = sx.flow_cnt;
      e.n_zero = flow_words;
    } else if (attn_o) {  // likewise the attention + O launches' counters
      e.zero = sx.flow_cnt;
      e.n_zero = kAoCounterBase + 2 * kAoSlots * kAoSlotWords;
    } else {  // the error word alone
      e.zero = sx.flow_cnt;
      e.n_zero = 1;
    }
    ProfScope ps(k, PF_OTHER, 0.0);
    HIP_TRY(launch_embed(e, s));
  }
  if (flow) return launch_flow_step();

  int lm_parts = 0;
  auto gemm = [&](int epi, GemmArgs& a, int N, int K, int family) -> hvd_status {
    a.KT = K / 32;
    a.NT = N / 16;
    a.wg = (size_t)a.KT * 256;  // pack_weight's layout: 4-strip groups, K steps contiguous
    a.wk = 256;
    a.MTtot = MT;
    a.M = M;
    a.part = sx.gemm_part;
    a.cnt = sx.gemm_cnt;
    const int want = k->gemm_min_blocks;
    if (MT > k->skinny_max_mt && N % 128 == 0) {
      // many rows: MFMA-tiled kernel, weights read once per XCD.  Of the
      // tiles that give at least one workgroup per CU, 256 x 256 unless the
      // 128-row tile pads the rows less (the padded rows' MFMA work is
      // wasted: 848 rows run as 1024 or as 896); else 128 x 256 on 8 waves
      // (one workgroup per CU, a six-slot operand ring), K-split to about
      // 7/8 of a workgroup per CU unless 5/8 are there already; else
      // 128 x 128 with a K split when even that leaves CUs idle.  Measured
      // against 128 x 128: the 848-row batch 30.2 -> 29.3 ms (QKV unsplit,
      // O and down split 2), the 32B multistep step 59.3 -> 57.1 ms (QKV
      // split 2, O and down split 4)
      static const int tile_bm[5] = {128, 128, 256, 256, 128}, tile_bn[5] = {128, 256, 256, 256, 256};
      const int want_t = std::max(want, kCUs);
      auto rb_of = [&](int t) { return (MT * 16 + tile_bm[t] - 1) / tile_bm[t]; };
      auto fits = [&](int t) { return N % tile_bn[t] == 0 && N / tile_bn[t] * rb_of(t) >= want_t; };
      const bool mlp = epi == EPI_SILU || family == PF_DOWN;
      const bool single = lm_head && ((mlp && (epi == EPI_SILU ? k->mlp_single_gu : k->mlp_single_down)) ||
                                      (epi == EPI_LM && k->lm_single));
      int tile = 0;
      if (fits(2) && !(fits(1) && rb_of(1) * 128 < rb_of(2) * 256)) tile = 2;
      // the hi + lo pair's 32 KB K steps leave the 4-wave 128 x 256 tile one
      // workgroup per CU and a three-slot ring: the 8-wave tile's four slots
      // serve it better (32B multistep, gate/up on the pair: 69.1 -> 67.3 ms)
      else if (fits(1)) tile = single ? 1 : 4;
      else if (N % tile_bn[4] == 0) tile = 4;
      const bool forced = family <= PF_LM && k->tiled_force[family][0] && N % tile_bn[k->tiled_force[family][0] - 1] == 0;
      if (forced) tile = k->tiled_force[family][0] - 1;
      const int RB = (MT * 16 + tile_bm[tile] - 1) / tile_bm[tile];
      const int nblk = N / tile_bn[tile] * RB;
      int splits = 1;
      if (forced) splits = std::max(1, std::min(k->tiled_force[family][1], a.KT / 32));
      else if (tile == 4) {
        if (nblk * 8 < want_t * 5) splits = std::max(1, std::min({4, (want_t * 7 / 8 + nblk - 1) / nblk, a.KT / 32}));
      } else if (nblk < want_t) splits = std::max(1, std::min({4, (want_t + nblk - 1) / nblk, a.KT / 32}));
      while (splits > 1 && (size_t)splits * RB * tile_bm[tile] * N * 4 > sx.gemm_part_bytes) --splits;
      if (splits > 1 && nblk > kGemmCounters) splits = 1;  // one arrival counter per output tile
      if (epi == EPI_LM) {
        lm_parts = N / tile_bn[tile];
        a.n_part = lm_parts;
      }
      ProfScope ps(k, family, (double)N * K * 2.0);
      HIP_TRY(launch_gemm_tiled(epi, a, tile, !single, splits, sx.inv_rms, s));
      return HVD_OK;
    }
    // verify forwards: MLP and LM-head GEMMs on the hi activation part (as the
    // tiled path); measured at batch 1, context 2048: 3.48 -> 3.39 ms per step at
    // k = 8 (gate/up 38.3 -> 36.0 us, down 23.9 -> 22.9 us per layer)
    const bool single = lm_head &&
                        ((epi == EPI_SILU && k->mlp_single_gu) || (family == PF_DOWN && k->mlp_single_down) ||
                         (k->lm_single && epi == EPI_LM));
    // five row tiles (65-80 rows): one block, so the weights are read once --
    // single-pass GEMMs, and the residual GEMMs (O, down) on the hi + lo pair
    const bool five = MT == 5 && (single || epi == EPI_RESID);
    const int mblocks_g = five ? 1 : mblocks, mt_block_g = five ? 5 : mt_block;
    int ns = 4, splits = 1;
    skinny_shape(epi, N, K, family, single, mblocks_g, mt_block_g, ns, splits);
    if (epi == EPI_LM) {
      lm_parts = a.NT / ns;
      a.n_part = lm_parts;
    }
    ProfScope ps(k, family, (double)N * K * 2.0);
    HIP_TRY(launch_gemm(epi, a, ns, splits, mblocks_g, mt_block_g, !single, s));
    return HVD_OK;
  };
  double kv_bytes_cl[kAttnClasses] = {};  // KV bytes each attention launch reads
  for (int cl = 0; cl < kAttnClasses; ++cl)
    for (int b : members[cl]) kv_bytes_cl[cl] += (double)(seqs[b].ctx + seqs[b].k + 1) * kvd * 2 * 2;

  for (int l = 0; l < c.n_layers; ++l) {
    const LayerW& L = m->layers[l];
    _Float16* kvl = k->pool + (size_t)l * k->layer_stride;
    {
      GemmArgs a{};
      a.W = (const uint4*)L.qkv;
      a.Ahi = (const uint4*)k->Nhi;
      a.Alo = (const uint4*)k->Nlo;
      a.ss = k->ss;
      a.ss_n = D / 16;
      a.inv_dim = 1.f / D;
      a.eps = c.rms_eps;
      a.Q = k->Q;
      a.kv = kvl;
      a.page_stride = k->page_stride;
      a.q_cols = qd;
      a.kv_cols = kvd;
      a.Hkv = c.n_kv_heads;
      a.dh = dh;
      a.pt = k->pt;
      a.pt_stride = k->pt_stride;
      a.rows = d_rows;
      a.rope = m->rope;
      if (hvd_status st = gemm(EPI_QKV, a, qd + 2 * kvd, D, PF_QKV); st != HVD_OK) return st;
    }
    if (attn_o) {
      const Plan& pl = plans[1];
      AttnOArgs ao{};
      AttnArgs& a = ao.at;
      a.Q = k->Q;
      a.kv = kvl;
      a.page_stride = k->page_stride;
      a.Hq = c.n_q_heads;
      a.Hkv = c.n_kv_heads;
      a.dh = dh;
      a.group = G;
      a.pt = k->pt;
      a.pt_stride = k->pt_stride;
      a.items = d_items + pl.item0;
      a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)dh));
      a.Ohi = k->Ohi;
      a.Olo = k->Olo;
      a.MTtot = MT;
      a.tree_mask = d_mask;
      a.part_o = sx.part_o + pl.part_base * dh;
      a.part_ml = sx.part_ml + pl.part_base * 2;
      CombineArgs& cb = ao.cb;
      cb.heads = d_heads + pl.head0;
      cb.Hq = c.n_q_heads;
      cb.Hkv = c.n_kv_heads;
      cb.dh = dh;
      cb.group = G;
      cb.part_o = a.part_o;
      cb.part_ml = a.part_ml;
      cb.Ohi = k->Ohi;
      cb.Olo = k->Olo;
      cb.MTtot = MT;
      cb.rpi = pl.rpi;
      cb.max_rows = pl.comb_rows;
      ao.n_attn = ao_attn_wgs;
      ao.n_items = pl.n_items_real;
      ao.n_heads = pl.n_heads_real;
      ao.merge_spb = (pl.comb_rows + kAoMergeRows - 1) / kAoMergeRows;
      GemmArgs& g = ao.go;
      g.W = (const uint4*)L.o;
      g.KT = qd / 32;
      g.NT = D / 16;
      g.wg = (size_t)g.KT * 256;
      g.wk = 256;
      g.Ahi = (const uint4*)k->Ohi;
      g.Alo = (const uint4*)k->Olo;
      g.MTtot = MT;
      g.M = M;
      g.X = k->X;
      g.D = D;
      g.gain_next = L.g_mlp;
      g.Nhi = k->Nhi;
      g.Nlo = k->Nlo;
      g.ss_out = k->ss;
      ao.cnt = sx.flow_cnt + kAoCounterBase;
      ao.target = (uint32_t)(l + 1) * (uint32_t)ao_attn_wgs;
      ao.err = sx.flow_cnt;
      const size_t grid = (size_t)ao_attn_wgs + g.NT;
      if (k->flow_trace && (size_t)c.n_layers * grid * kAoTraceWords <= (size_t)k->flow_trace_words)
        ao.trace = k->flow_trace + (size_t)l * grid * kAoTraceWords;
      // 2-page sub-chunks for 128-row items (4 would spill registers)
      const int np = std::min(pl.rpi > kAttnRows / 2 ? 2 : 4, attn_pages_per_sub(pl.chunk));
      ProfScope ps(k, PF_ATTN_O, kv_bytes_cl[1] + (double)qd * D * 2);
      HIP_TRY(launch_attn_o(ao, np, pl.rpi, MT, s));
    } else {
      {
        AttnArgs a{};
        a.Q = k->Q;
        a.kv = kvl;
        a.page_stride = k->page_stride;
        a.Hq = c.n_q_heads;
        a.Hkv = c.n_kv_heads;
        a.dh = dh;
        a.group = G;
        a.pt = k->pt;
        a.pt_stride = k->pt_stride;
        a.items = d_items;
        a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)dh));
        a.Ohi = k->Ohi;
        a.Olo = k->Olo;
        a.MTtot = MT;
        a.tree_mask = d_mask;
        // one launch per row class, then the combine passes
        for (int cl = 0; cl < kAttnClasses; ++cl) {
          const Plan& pl = plans[cl];
          if (pl.items.empty()) continue;
          a.items = d_items + pl.item0;
          a.part_o = sx.part_o + pl.part_base * dh;
          a.part_ml = sx.part_ml + pl.part_base * 2;
          ProfScope ps(k, PF_ATTN, kv_bytes_cl[cl]);
          HIP_TRY(launch_attn(a, (int)pl.items.size(), pl.chunk, pl.rpi, k->attn_max_np, s));
        }
        for (int cl = 0; cl < kAttnClasses; ++cl) {
          const Plan& pl = plans[cl];
          if (pl.heads.empty()) continue;
          CombineArgs cb{};
          cb.heads = d_heads + pl.head0;
          cb.Hq = c.n_q_heads;
          cb.Hkv = c.n_kv_heads;
          cb.dh = dh;
          cb.group = G;
          cb.part_o = sx.part_o + pl.part_base * dh;
          cb.part_ml = sx.part_ml + pl.part_base * 2;
          cb.Ohi = k->Ohi;
          cb.Olo = k->Olo;
          cb.MTtot = MT;
          cb.rpi = pl.rpi;
          cb.max_rows = pl.comb_rows;
          ProfScope ps(k, PF_COMBINE, 0.0);
          HIP_TRY(launch_combine(cb, (int)pl.heads.size(), s));
        }
      }
      {
        GemmArgs a{};
        a.W = (const uint4*)L.o;
        a.Ahi = (const uint4*)k->Ohi;
        a.Alo = (const uint4*)k->Olo;
        a.X = k->X;
        a.D = D;
        a.gain_next = L.g_mlp;
        a.Nhi = k->Nhi;
        a.Nlo = k->Nlo;
        a.ss_out = k->ss;
        if (hvd_status st = gemm(EPI_RESID, a, D, qd, PF_O); st != HVD_OK) return st;
      }
    }
    {
      GemmArgs a{};
      a.W = (const uint4*)L.gu;
      a.Ahi = (const uint4*)k->Nhi;
      a.Alo = (const uint4*)k->Nlo;
      a.ss = k->ss;
      a.ss_n = D / 16;
      a.inv_dim = 1.f / D;
      a.eps = c.rms_eps;
      a.act_hi = k->Ahi;
      a.act_lo = k->Alo;
      if (hvd_status st = gemm(EPI_SILU, a, 2 * F, D, PF_GATEUP); st != HVD_OK) return st;
    }
    {
      GemmArgs a{};
      a.W = (const uint4*)L.down;
      a.Ahi = (const uint4*)k->Ahi;
      a.Alo = (const uint4*)k->Alo;
      a.X = k->X;
      a.D = D;
      a.gain_next = (l + 1 < c.n_layers) ? m->layers[l + 1].g_attn : m->g_final;
      a.Nhi = k->Nhi;
      a.Nlo = k->Nlo;
      a.ss_out = k->ss;
      if (hvd_status st = gemm(EPI_RESID, a, D, F, PF_DOWN); st != HVD_OK) return st;
    }
  }
  if (lm_head) {
    GemmArgs a{};
    a.W = (const uint4*)m->lm;
    a.Ahi = (const uint4*)k->Nhi;
    a.Alo = (const uint4*)k->Nlo;
    a.ss = k->ss;
    a.ss_n = D / 16;
    a.inv_dim = 1.f / D;
    a.eps = c.rms_eps;
    a.logits = logits;
    a.vocab = c.vocab;
    a.part_val = sx.lm_val;
    a.part_idx = sx.lm_idx;
    if (hvd_status st = gemm(EPI_LM, a, c.vocab, D, PF_LM); st != HVD_OK) return st;
    AcceptArgs ac{};
    ac.part_val = sx.lm_val;
    ac.part_idx = sx.lm_idx;
    ac.n_part = lm_parts;
    ac.M = M;
    ac.g = sx.g;
    ac.seqs = d_seqs;
    ac.rows = d_rows;
    ac.B = B;
    ac.out = sx.out;
    ac.counter = sx.counter;
    ac.tree_parent = d_parent;
    ac.path = sx.out + 2 * B;
    if (attn_o) {  // bounded waits inside the attention + O launches
      ac.err_word = sx.flow_cnt;
      ac.err_index = (tree ? 2 + kMaxTreeNodes : 2) * B;
    }
    if (acap) {
      ac.astate = acap->state;
      ac.hist = acap->hist;
      ac.hist_cap = acap->hist_cap;
    }
    {
      ProfScope ps(k, PF_OTHER, 0.0);
      HIP_TRY(launch_accept(ac, s));
    }
    if (tree) {
      CompactArgs cp{};
      cp.pool = k->pool;
      cp.page_stride = k->page_stride;
      cp.layer_stride = k->layer_stride;
      cp.n_layers = c.n_layers;
      cp.Hkv = c.n_kv_heads;
      cp.dh = dh;
      cp.pt = k->pt;
      cp.pt_stride = k->pt_stride;
      cp.seqs = d_seqs;
      cp.out = sx.out;
      cp.path = sx.out + 2 * B;
      ProfScope ps(k, PF_OTHER, 0.0);
      HIP_TRY(launch_compact(cp, B, s));
    }
  }
  return HVD_OK;
  };  // launch_all

  if (acap) {
    // captured once; the loop replays it (no profiling events inside)
    const bool prof = k->prof;
    k->prof = false;
    hipGraph_t g = nullptr;
    HIP_TRY(hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal));
    const hvd_status st = launch_all();
    const hipError_t ec = hipStreamEndCapture(s, &g);
    k->prof = prof;
    if (st != HVD_OK) {
      if (g) (void)hipGraphDestroy(g);
      return st;
    }
    if (ec != hipSuccess) return set_err(HVD_ERR_DEVICE, std::string("graph capture: ") + hipGetErrorString(ec));
    const hipError_t ei = hipGraphInstantiate(&acap->graph, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (ei != hipSuccess) {
      acap->graph = nullptr;
      return set_err(HVD_ERR_DEVICE, std::string("graph instantiate: ") + hipGetErrorString(ei));
    }
    return HVD_OK;
  }
  if (k->prof || !k->use_graphs || eager_only) {
    if (hvd_status st = launch_all(); st != HVD_OK) return st;
  } else {
    const GraphKey key{M, B, lm_head ? 1 : 0, tree ? 1 : 0, attn_key, logits};
    auto it = k->graphs.find(key);
    if (it == k->graphs.end()) {
      if (k->graphs.size() >= kMaxGraphs) {
        for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);
        k->graphs.clear();
      }
      hipGraph_t g = nullptr;
      HIP_TRY(hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal));
      const hvd_status st = launch_all();
      const hipError_t ec = hipStreamEndCapture(s, &g);
      if (st != HVD_OK) {
        if (g) (void)hipGraphDestroy(g);
        return st;
      }
      if (ec != hipSuccess) return set_err(HVD_ERR_DEVICE, std::string("graph capture: ") + hipGetErrorString(ec));
      hipGraphExec_t ge = nullptr;
      const hipError_t ei = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
      (void)hipGraphDestroy(g);
      if (ei != hipSuccess) return set_err(HVD_ERR_DEVICE, std::string("graph instantiate: ") + hipGetErrorString(ei));
      it = k->graphs.emplace(key, ge).first;
    }
    HIP_TRY(hipGraphLaunch(it->second, s));
  }
  if (lm_head)  // results, and for trees the accepted paths behind them
    HIP_TRY(hipMemcpyAsync(k->out_host, sx.out,
                           ((tree ? 2 + kMaxTreeNodes : 2) * (size_t)B + (flow || attn_o ? 1 : 0)) * 4,
                           hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (k->prof) prof_collect(k);
  if (lm_head && (flow || attn_o) && k->out_host[(tree ? 2 + kMaxTreeNodes : 2) * B] != 0)
    return set_err(HVD_ERR_DEVICE, "a bounded in-kernel wait gave up (results invalid)");
  return HVD_OK;
}

hvd_status from_host(int code, hvd_kv_s* k) {
  if (code == HS_OK) return HVD_OK;
  return set_err((hvd_status)code, k->hs->error());
}

}  // namespace

extern "C" hvd_status hvd_prefill(hvd_model m, hvd_kv k, int32_t seq_id, const int32_t* tokens, int32_t n) {
  if (!m || !k) return set_err(HVD_ERR_ARG, "null handle");
  if (k->m != m) return set_err(HVD_ERR_ARG, "kv handle belongs to another model");
  if (hvd_status st = from_host(k->hs->begin_prefill(seq_id, tokens, n), k); st != HVD_OK) return st;
  const int body = n - 1;
  const int chunk_rows = k->prefill_rows ? k->prefill_rows : prefill_rows(m->cfg);
  for (int s0 = 0; s0 < body; s0 += chunk_rows) {
    const int cnt = std::min(chunk_rows, body - s0);
    std::vector<SeqMeta> seqs{{seq_id, s0, cnt - 1, 0}};
    std::vector<RowMeta> rows(cnt);
    for (int i = 0; i < cnt; ++i) rows[i] = {tokens[s0 + i], seq_id, s0 + i, s0 + i};
    hvd_status st = forward(k, seqs, rows, false, nullptr);
    if (st != HVD_OK) {
      k->hs->abort_prefill(seq_id);
      return st;
    }
  }
  return HVD_OK;
}

namespace {

// Carve one step's scratch out of this device's static array: the fixed
// parts (results, arrival counter, per-row argmax / inverse RMS, LM-head
// partials) first, then 8 MiB of split-K partial tiles, the rest for
// attention split-KV partials.  HVD_ERR_RANGE when the fixed parts alone do
// not fit.
hvd_status carve_static(hvd_kv_s* k, int M, int B, StepScratch& sx) {
  const hvd_config& c = k->m->cfg;
  if (!k->static_base) return set_err(HVD_ERR_DEVICE, "static scratch unavailable on this device");
  const size_t Mp = (size_t)(M + 15) / 16 * 16;
  Carver cv(k->static_base);
  sx.counter = cv.take<uint32_t>(64);
  sx.gemm_cnt = cv.take<uint32_t>(kGemmCounters);
  sx.flow_cnt = cv.take<uint32_t>(kFlowCounterWords);
  sx.out = cv.take<int32_t>((2 + kMaxTreeNodes) * (size_t)B + 1);
  sx.g = cv.take<int32_t>(Mp);
  sx.inv_rms = cv.take<float>(Mp);
  sx.lm_val = cv.take<float>(Mp * (size_t)k->n_part_lm);
  sx.lm_idx = cv.take<int32_t>(Mp * (size_t)k->n_part_lm);
  const size_t gemm_bytes = std::min<size_t>(kGemmPartBytes, 8u << 20);
  sx.gemm_part = cv.take<float>(gemm_bytes / 4);
  sx.gemm_part_bytes = gemm_bytes;
  if (cv.off >= k->static_bytes)
    return set_err(HVD_ERR_RANGE, "step too large for hvd_verify_noalloc: its fixed scratch needs " +
                                      std::to_string(cv.off) + " bytes of the " + std::to_string(k->static_bytes) +
                                      "-byte static scratch (use hvd_verify)");
  const size_t row_bytes = (size_t)c.head_dim * 4 + 2 * 4;
  const size_t rows_free = (k->static_bytes - cv.off - 2 * kAlign) / row_bytes;
  sx.part_rows = rows_free;
  sx.part_o = cv.take<float>(rows_free * c.head_dim);
  sx.part_ml = cv.take<float>(rows_free * 2);
  if (cv.off > k->static_bytes) return set_err(HVD_ERR_RANGE, "static scratch layout overflow");
  return HVD_OK;
}

hvd_status verify_chain(hvd_model m, hvd_kv k, int32_t batch, const int32_t* seq_ids, const int32_t* ctx_lens,
                        const int32_t* draft_tokens, const int32_t* draft_lens, int32_t* accepted_len,
                        int32_t* next_token, float* logits, bool use_static) {
  if (!m || !k) return set_err(HVD_ERR_ARG, "null handle");
  if (k->m != m) return set_err(HVD_ERR_ARG, "kv handle belongs to another model");
  if (!accepted_len || !next_token) return set_err(HVD_ERR_ARG, "null output");
  StepScratch stat;
  if (use_static) {
    // size check before any state change: rows = sum(k_b + 1)
    if (batch < 1 || !draft_lens) return set_err(HVD_ERR_ARG, "bad batch");
    int64_t M = 0;
    for (int b = 0; b < batch; ++b) M += (int64_t)std::max(0, draft_lens[b]) + 1;
    if (hvd_status st = carve_static(k, (int)std::min<int64_t>(M, 1 << 30), batch, stat); st != HVD_OK) return st;
  }
  if (hvd_status st = from_host(k->hs->begin_verify(batch, seq_ids, ctx_lens, draft_tokens, draft_lens), k);
      st != HVD_OK)
    return st;
  std::vector<SeqMeta> seqs(batch);
  std::vector<RowMeta> rows;
  int64_t off = 0;
  for (int b = 0; b < batch; ++b) {
    const SeqSlot& sl = k->hs->seq(seq_ids[b]);
    const int kk = draft_lens[b];
    seqs[b] = {seq_ids[b], sl.ctx, kk, (int32_t)rows.size()};
    rows.push_back({sl.pending, seq_ids[b], sl.ctx, sl.ctx});
    for (int i = 0; i < kk; ++i)
      rows.push_back({draft_tokens[off + i], seq_ids[b], sl.ctx + 1 + i, sl.ctx + 1 + i});
    off += kk;
  }
  hvd_status st = HVD_OK;
  if (use_static) {
    // the arrival counter starts at zero (an earlier failed call may have left it set)
    const bool prof = k->prof;
    k->prof = false;  // no profiling events: creating them allocates
    // counters start at zero (an earlier failed call may have left some set);
    // the accept counter and the split-K counters are adjacent
    if (hipMemsetAsync(stat.counter, 0, (size_t)((char*)(stat.gemm_cnt + kGemmCounters) - (char*)stat.counter),
                       k->stream) != hipSuccess)
      st = set_err(HVD_ERR_DEVICE, "clearing the static scratch counter failed");
    else
      st = forward(k, seqs, rows, true, logits, nullptr, nullptr, &stat);
    k->prof = prof;
  } else {
    st = forward(k, seqs, rows, true, logits);
  }
  if (st != HVD_OK) {
    k->hs->abort_verify(batch, seq_ids);
    return st;
  }
  for (int b = 0; b < batch; ++b) {
    accepted_len[b] = k->out_host[2 * b];
    next_token[b] = k->out_host[2 * b + 1];
  }
  k->hs->finish_verify(batch, seq_ids, draft_tokens, draft_lens, accepted_len, next_token);
  return HVD_OK;
}

}  // namespace

extern "C" hvd_status hvd_verify(hvd_model m, hvd_kv k, int32_t batch, const int32_t* seq_ids, const int32_t* ctx_lens,
                                 const int32_t* draft_tokens, const int32_t* draft_lens, int32_t* accepted_len,
                                 int32_t* next_token, float* logits) {
  return verify_chain(m, k, batch, seq_ids, ctx_lens, draft_tokens, draft_lens, accepted_len, next_token, logits,
                      false);
}

extern "C" hvd_status hvd_verify_noalloc(hvd_model m, hvd_kv k, int32_t batch, const int32_t* seq_ids,
                                         const int32_t* ctx_lens, const int32_t* draft_tokens,
                                         const int32_t* draft_lens, int32_t* accepted_len, int32_t* next_token,
                                         float* logits) {
  return verify_chain(m, k, batch, seq_ids, ctx_lens, draft_tokens, draft_lens, accepted_len, next_token, logits,
                      true);
}

extern "C" hvd_status hvd_verify_tree(hvd_model m, hvd_kv k, int32_t batch, const int32_t* seq_ids,
                                      const int32_t* ctx_lens, const int32_t* node_tokens, const int32_t* node_parents,
                                      const int32_t* node_counts, int32_t* accepted_len, int32_t* next_token,
                                      int32_t* accepted_nodes, float* logits) {
  if (!m || !k) return set_err(HVD_ERR_ARG, "null handle");
  if (k->m != m) return set_err(HVD_ERR_ARG, "kv handle belongs to another model");
  if (!accepted_len || !next_token) return set_err(HVD_ERR_ARG, "null output");
  if (batch < 1 || !node_counts) return set_err(HVD_ERR_ARG, "bad batch");
  // tree structure first (node counts, parents before children), then the
  // checks every verify makes (tokens, positions, pages) on the node list
  {
    int64_t off = 0;
    for (int b = 0; b < batch; ++b) {
      const int n = node_counts[b];
      if (n < 0 || n > kMaxTreeNodes) return set_err(HVD_ERR_RANGE, "tree node count outside [0, 63]");
      if (n > 0 && (!node_tokens || !node_parents)) return set_err(HVD_ERR_ARG, "null tree arrays");
      for (int j = 0; j < n; ++j)
        if (node_parents[off + j] < -1 || node_parents[off + j] >= j)
          return set_err(HVD_ERR_ARG, "a node's parent must be -1 or an earlier node");
      off += n;
    }
  }
  if (hvd_status st = from_host(k->hs->begin_verify(batch, seq_ids, ctx_lens, node_tokens, node_counts), k);
      st != HVD_OK)
    return st;
  std::vector<SeqMeta> seqs(batch);
  std::vector<RowMeta> rows;
  TreeRows tr;
  int64_t off = 0;
  for (int b = 0; b < batch; ++b) {
    const SeqSlot& sl = k->hs->seq(seq_ids[b]);
    const int n = node_counts[b];
    seqs[b] = {seq_ids[b], sl.ctx, n, (int32_t)rows.size(), 1};
    // row 0: the pending token; row j + 1: node j at rotary position
    // ctx + depth, K/V position ctx + 1 + j; ancestor bits over rows
    std::vector<int> depth(n);
    std::vector<uint64_t> anc(n + 1);
    anc[0] = 1;
    rows.push_back({sl.pending, seq_ids[b], sl.ctx, sl.ctx});
    tr.mask.push_back(anc[0]);
    tr.parent.push_back(-1);
    for (int j = 0; j < n; ++j) {
      const int p = node_parents[off + j];
      depth[j] = p < 0 ? 1 : depth[p] + 1;
      anc[j + 1] = anc[p + 1] | (1ull << (j + 1));
      rows.push_back({node_tokens[off + j], seq_ids[b], sl.ctx + depth[j], sl.ctx + 1 + j});
      tr.mask.push_back(anc[j + 1]);
      tr.parent.push_back(p);
    }
    off += n;
  }
  hvd_status st = forward(k, seqs, rows, true, logits, &tr);
  if (st != HVD_OK) {
    k->hs->abort_verify(batch, seq_ids);
    return st;
  }
  // the accepted path's tokens become the "draft" that commit keeps a prefix of
  std::vector<int32_t> path_tokens, acc(batch);
  off = 0;
  for (int b = 0; b < batch; ++b) {
    accepted_len[b] = acc[b] = k->out_host[2 * b];
    next_token[b] = k->out_host[2 * b + 1];
    const int32_t* path = k->out_host + 2 * batch + (size_t)b * kMaxTreeNodes;
    for (int d = 0; d < acc[b]; ++d) {
      path_tokens.push_back(node_tokens[off + path[d]]);
      if (accepted_nodes) accepted_nodes[(size_t)b * kMaxTreeNodes + d] = path[d];
    }
    off += node_counts[b];
  }
  k->hs->finish_verify(batch, seq_ids, path_tokens.data(), acc.data(), accepted_len, next_token);
  return HVD_OK;
}

// ------------------------------------------------------------ device-resident loop

struct hvd_async_s {
  hvd_kv_s* k = nullptr;
  std::vector<int32_t> ids;
  int32_t* state = nullptr;  // caller's: ctx[B], pending[B], steps done
  int max_steps = 0, launched = 0;
  int32_t* meta = nullptr;
  hipGraphExec_t graph = nullptr;
};

extern "C" hvd_status hvd_async_begin(hvd_model m, hvd_kv k, int32_t batch, const int32_t* seq_ids,
                                      const int32_t* ctx_lens, const int32_t* draft_lens, int32_t max_steps,
                                      int32_t* drafts, int32_t* state, int32_t* history, const int32_t* ref_tokens,
                                      int32_t ref_len, const int32_t* ref_start, hvd_async* out) {
  if (!m || !k) return set_err(HVD_ERR_ARG, "null handle");
  if (k->m != m) return set_err(HVD_ERR_ARG, "kv handle belongs to another model");
  if (!out || !state || !history) return set_err(HVD_ERR_ARG, "null state, history or out");
  if (ref_tokens && (ref_len < 1 || !ref_start)) return set_err(HVD_ERR_ARG, "copy drafter needs ref_len >= 1 and ref_start");
  if (hvd_status st = from_host(k->hs->begin_async(batch, seq_ids, ctx_lens, draft_lens, max_steps), k); st != HVD_OK)
    return st;
  std::vector<int32_t> ctx0(batch), pend0(batch);
  int64_t sum_k = 0;
  for (int b = 0; b < batch; ++b) {
    ctx0[b] = k->hs->seq(seq_ids[b]).ctx;
    pend0[b] = k->hs->seq(seq_ids[b]).pending;
    sum_k += draft_lens[b];
  }
  auto undo = [&](hvd_status st) {
    k->hs->end_async(batch, seq_ids, ctx0.data(), pend0.data());
    return st;
  };
  if (sum_k > 0 && !drafts) return undo(set_err(HVD_ERR_ARG, "null drafts buffer"));
  // the step is planned at the longest context the loop reaches (every
  // draft accepted until the last step); rows are rebuilt on the device
  AsyncCap cap;
  cap.drafts = drafts;
  cap.state = state;
  cap.hist = history;
  cap.hist_cap = max_steps;
  cap.ref = ref_tokens;
  cap.ref_len = ref_tokens ? ref_len : 0;
  std::vector<SeqMeta> seqs(batch);
  std::vector<RowMeta> rows;
  cap.page_off.push_back(0);
  for (int b = 0; b < batch; ++b) {
    const SeqSlot& sl = k->hs->seq(seq_ids[b]);
    const int kk = draft_lens[b];
    const int ctx_max = sl.ctx + (max_steps - 1) * (kk + 1);
    seqs[b] = {seq_ids[b], ctx_max, kk, (int32_t)rows.size()};
    for (int i = 0; i <= kk; ++i) rows.push_back({0, seq_ids[b], ctx_max + i, ctx_max + i});
    cap.pages.insert(cap.pages.end(), sl.pages.begin(), sl.pages.end());
    cap.page_off.push_back((int32_t)cap.pages.size());
    cap.ref_start.push_back(ref_tokens ? ref_start[b] : 0);
  }
  std::vector<int32_t> st0(2 * (size_t)batch + 1, 0);
  for (int b = 0; b < batch; ++b) {
    st0[b] = ctx0[b];
    st0[batch + b] = pend0[b];
  }
  if (hipMemcpyAsync(state, st0.data(), st0.size() * 4, hipMemcpyHostToDevice, k->stream) != hipSuccess ||
      hipStreamSynchronize(k->stream) != hipSuccess)
    return undo(set_err(HVD_ERR_DEVICE, "loop state upload failed"));
  if (hvd_status st = forward(k, seqs, rows, true, nullptr, nullptr, &cap); st != HVD_OK) {
    if (cap.graph) (void)hipGraphExecDestroy(cap.graph);
    if (cap.meta) (void)hipFree(cap.meta);
    return undo(st);
  }
  auto* a = new hvd_async_s();
  a->k = k;
  a->ids.assign(seq_ids, seq_ids + batch);
  a->state = state;
  a->max_steps = max_steps;
  a->meta = cap.meta;
  a->graph = cap.graph;
  *out = a;
  return HVD_OK;
}

extern "C" hvd_status hvd_async_step(hvd_async a, int32_t n_steps) {
  if (!a) return set_err(HVD_ERR_ARG, "null handle");
  if (n_steps < 0) return set_err(HVD_ERR_ARG, "n_steps must be >= 0");
  if ((int64_t)a->launched + n_steps > a->max_steps) return set_err(HVD_ERR_RANGE, "more steps than the loop reserved");
  for (int i = 0; i < n_steps; ++i) {
    HIP_TRY(hipGraphLaunch(a->graph, a->k->stream));
    ++a->launched;
  }
  return HVD_OK;
}

extern "C" hvd_status hvd_async_end(hvd_async a, int32_t* steps_done) {
  if (!a) return set_err(HVD_ERR_ARG, "null handle");
  hvd_kv_s* k = a->k;
  const int B = (int)a->ids.size();
  std::vector<int32_t> st(2 * (size_t)B + 1);
  hvd_status ret = HVD_OK;
  if (hipMemcpyAsync(st.data(), a->state, st.size() * 4, hipMemcpyDeviceToHost, k->stream) != hipSuccess ||
      hipStreamSynchronize(k->stream) != hipSuccess) {
    ret = set_err(HVD_ERR_DEVICE, "loop state readback failed");
  } else if (st[2 * B] != a->launched) {
    ret = set_err(HVD_ERR_STATE, "the device step count disagrees with the steps launched");
  }
  if (ret == HVD_OK) {
    k->hs->end_async(B, a->ids.data(), st.data(), st.data() + B);
  } else {  // unknown device state: the sequences leave the loop at their start
    std::vector<int32_t> c0(B), p0(B);
    for (int b = 0; b < B; ++b) {
      c0[b] = k->hs->seq(a->ids[b]).ctx;
      p0[b] = k->hs->seq(a->ids[b]).pending;
    }
    k->hs->end_async(B, a->ids.data(), c0.data(), p0.data());
  }
  if (steps_done) *steps_done = a->launched;
  (void)hipGraphExecDestroy(a->graph);
  (void)hipFree(a->meta);
  delete a;
  return ret;
}

extern "C" hvd_status hvd_commit(hvd_model m, hvd_kv k, int32_t batch, const int32_t* seq_ids, const int32_t* keep) {
  if (!m || !k) return set_err(HVD_ERR_ARG, "null handle");
  if (k->m != m) return set_err(HVD_ERR_ARG, "kv handle belongs to another model");
  return from_host(k->hs->commit(batch, seq_ids, keep), k);
}

extern "C" hvd_status hvd_truncate(hvd_kv k, int32_t seq_id, int32_t new_ctx_len, int32_t pending_token) {
  if (!k) return set_err(HVD_ERR_ARG, "null handle");
  return from_host(k->hs->truncate(seq_id, new_ctx_len, pending_token), k);
}

extern "C" hvd_status hvd_seq_free(hvd_kv k, int32_t seq_id) {
  if (!k) return set_err(HVD_ERR_ARG, "null handle");
  return from_host(k->hs->free_seq(seq_id), k);
}

extern "C" hvd_status hvd_seq_info(hvd_kv k, int32_t seq_id, int32_t* ctx_len, int32_t* pending, int32_t* vp) {
  if (!k) return set_err(HVD_ERR_ARG, "null handle");
  if (seq_id < 0 || seq_id >= k->hs->max_seqs() || !k->hs->seq(seq_id).live)
    return set_err(HVD_ERR_ARG, "unknown seq_id");
  const SeqSlot& s = k->hs->seq(seq_id);
  if (ctx_len) *ctx_len = s.ctx;
  if (pending) *pending = s.pending;
  if (vp) *vp = s.verify_pending ? 1 : 0;
  return HVD_OK;
}

extern "C" int32_t hvd_kv_free_pages(hvd_kv k) { return k ? k->hs->free_pages() : -1; }

extern "C" hvd_status hvd_profile_enable(hvd_kv k, int32_t enable) {
  if (!k) return set_err(HVD_ERR_ARG, "null handle");
  k->prof = enable != 0;
  for (int i = 0; i < kProfFamilies; ++i) {
    k->prof_ms[i] = 0;
    k->prof_bytes[i] = 0;
    k->prof_n[i] = 0;
  }
  return HVD_OK;
}

extern "C" hvd_status hvd_profile_read(hvd_kv k, int32_t family, double* ms, int64_t* launches, double* bytes) {
  if (!k || family < 0 || family >= kProfFamilies) return set_err(HVD_ERR_ARG, "bad handle or family");
  if (ms) *ms = k->prof_ms[family];
  if (launches) *launches = k->prof_n[family];
  if (bytes) *bytes = k->prof_bytes[family];
  return HVD_OK;
}

extern "C" hvd_status hvd_kv_set_option(hvd_kv k, int32_t option, int32_t value) {
  if (!k) return set_err(HVD_ERR_ARG, "null handle");
  switch (option) {
    case HVD_OPT_GRAPHS:
      k->use_graphs = value != 0;
      if (!k->use_graphs) {
        for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);
        k->graphs.clear();
      }
      return HVD_OK;
    case HVD_OPT_FLOW:
      k->use_flow = value != 0;
      for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);
      k->graphs.clear();
      return HVD_OK;
    case HVD_OPT_ATTN_O:
      k->use_attn_o = value != 0;
      for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);
      k->graphs.clear();
      return HVD_OK;
    case HVD_OPT_FLOW_ITEMS:
      if (value < 1) return set_err(HVD_ERR_ARG, "HVD_OPT_FLOW_ITEMS must be >= 1");
      k->flow_min_items = value;
      for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);
      k->graphs.clear();
      return HVD_OK;
    case HVD_OPT_GEMM_MIN_BLOCKS:
    case HVD_OPT_ATTN_MIN_ITEMS:
    case HVD_OPT_ATTN_MAX_NP:
    case HVD_OPT_SKINNY_MAX_MT:
    case HVD_OPT_NS8_MT3:
    case HVD_OPT_PREFILL_ROWS: {
      const hvd_config& c = k->m->cfg;
      if (option == HVD_OPT_GEMM_MIN_BLOCKS) {
        if (value < 1) return set_err(HVD_ERR_ARG, "HVD_OPT_GEMM_MIN_BLOCKS must be >= 1");
        k->gemm_min_blocks = value;
      } else if (option == HVD_OPT_ATTN_MIN_ITEMS) {
        if (value < 1) return set_err(HVD_ERR_ARG, "HVD_OPT_ATTN_MIN_ITEMS must be >= 1");
        k->attn_min_items = value;
      } else if (option == HVD_OPT_ATTN_MAX_NP) {
        if (value < 2 || value > kItemPages || (value & (value - 1)))
          return set_err(HVD_ERR_ARG, "HVD_OPT_ATTN_MAX_NP must be a power of two in [2, 16]");
        k->attn_max_np = value;
      } else if (option == HVD_OPT_SKINNY_MAX_MT) {
        if (value < 1 || value > 64) return set_err(HVD_ERR_ARG, "HVD_OPT_SKINNY_MAX_MT must be in [1, 64]");
        k->skinny_max_mt = value;
      } else if (option == HVD_OPT_NS8_MT3) {
        k->ns8_mt3 = value != 0;
      } else {
        if (value != 0 && (value < 16 || value % 16 || value > k->max_rows))
          return set_err(HVD_ERR_ARG, "HVD_OPT_PREFILL_ROWS must be 0 or a multiple of 16 within the row workspace");
        k->prefill_rows = value;
      }
      (void)c;
      for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);
      k->graphs.clear();
      return HVD_OK;
    }
    case HVD_OPT_MLP_SINGLE:
    case HVD_OPT_LM_SINGLE:
      if (value < 0 || value > (option == HVD_OPT_MLP_SINGLE ? 3 : 1))
        return set_err(HVD_ERR_ARG, option == HVD_OPT_MLP_SINGLE
                                        ? "HVD_OPT_MLP_SINGLE value: 0 (pair), 1 (both single), 2 (gate/up), 3 (down)"
                                        : "HVD_OPT_LM_SINGLE value: 0 or 1");
      if (option == HVD_OPT_MLP_SINGLE) {
        k->mlp_single_gu = value == 1 || value == 2;
        k->mlp_single_down = value == 1 || value == 3;
      } else {
        k->lm_single = value != 0;
      }
      for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);  // captured with the old choice
      k->graphs.clear();
      return HVD_OK;
  }
  if (option >= HVD_OPT_GEMM_SHAPE && option <= HVD_OPT_GEMM_SHAPE + PF_LM) {
    const int f = option - HVD_OPT_GEMM_SHAPE, ns = value / 100, sp = value % 100;
    if (value != 0 && !((ns == 1 || ns == 2 || ns == 4 || ns == 8) && sp >= 1 && sp <= 16))
      return set_err(HVD_ERR_ARG, "HVD_OPT_GEMM_SHAPE value: 0, or strips (1, 2, 4, 8) * 100 + K splits (1..16)");
    k->gemm_force[f][0] = value ? ns : 0;
    k->gemm_force[f][1] = value ? sp : 0;
    for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);
    k->graphs.clear();
    return HVD_OK;
  }
  if (option >= HVD_OPT_TILED_SHAPE && option <= HVD_OPT_TILED_SHAPE + PF_LM) {
    const int f = option - HVD_OPT_TILED_SHAPE, t = value / 100 - 1, sp = value % 100;
    if (value != 0 && !(t >= 0 && t <= 4 && sp >= 1 && sp <= 8))
      return set_err(HVD_ERR_ARG, "HVD_OPT_TILED_SHAPE value: 0, or (tile + 1) * 100 + K splits (1..8)");
    k->tiled_force[f][0] = value ? t + 1 : 0;
    k->tiled_force[f][1] = value ? sp : 0;
    for (auto& g : k->graphs) (void)hipGraphExecDestroy(g.second);
    k->graphs.clear();
    return HVD_OK;
  }
  return set_err(HVD_ERR_ARG, "unknown option");
}

extern "C" hvd_status hvd_flow_trace(hvd_kv k, uint64_t* dev_buf, int64_t n_words) {
  if (!k) return set_err(HVD_ERR_ARG, "null handle");
  if (dev_buf && n_words < 4) return set_err(HVD_ERR_ARG, "trace buffer too small");
  k->flow_trace = dev_buf;
  k->flow_trace_words = dev_buf ? n_words : 0;
  return HVD_OK;
}

extern "C" const char* hvd_last_error(void) { return g_err.c_str(); }
