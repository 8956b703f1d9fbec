// One-launch verify step (gfx950): the whole forward of a verify batch of at
// most two row tiles -- for every layer the QKV GEMM (+ rotary, KV write),
// the attention chunks, their split-KV merge, the O GEMM (+ residual), the
// gate/up GEMM (+ SiLU) and the down GEMM (+ residual), then the LM head --
// as one grid of 512-thread workgroups.
//
// Why: at batch 1 every one of these launches is short (5-40 us), and each
// stand-alone kernel pays its ramp (first weight bytes ~2 us after the start)
// and its tail (the last workgroups' reduction and epilogue, the drain) with
// HBM idle.  Here the workgroups of the next phase are dispatched as soon as
// slots free up, request their weights (or cached K/V) at once, and wait
// only for the data they depend on, so the weight stream does not stop at
// phase boundaries.
//
// Ordering and forward progress: workgroup w's role follows from w (layer,
// phase, unit), and roles of later phases have larger w.  A workgroup only
// waits for work of smaller w: under in-order dispatch those workgroups are
// already resident and never wait for it, so every wait ends.  Each wait is
// bounded nonetheless (kSpinLimit polls); a wait that gives up sets bit 0 of
// *err and the host reports the step as failed.
//
// Coherence: the L2 caches of the 8 XCDs are not coherent with each other.
// Data handed between workgroups (activations, K/V of the new rows, partials)
// is written with device-scope (sc1, write-through) stores and read with
// device-scope loads after the producer's completion count is seen; weights,
// cached K/V and the step's metadata are read normally.  A producer waits for
// its stores (vmcnt(0)) before counting itself done.
#include <algorithm>

#include "attn.h"
#include "skinny.h"

namespace hvd {

constexpr uint32_t kSpinLimit = 1u << 20;

// Wait until the n (<= 8) counters at ctr sum to at least target.
__device__ __forceinline__ void flow_wait(const uint32_t* ctr, int n, uint32_t target, uint32_t* err) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    for (uint32_t it = 0;; ++it) {
      uint32_t v = lane < n ? ld_u32_dev(ctr + lane) : 0u;
      v += __shfl_xor(v, 1);
      v += __shfl_xor(v, 2);
      v += __shfl_xor(v, 4);
      v = __builtin_amdgcn_readfirstlane(v);  // lane 0: the sum of lanes 0..7
      if (v >= target) break;
      if (it >= kSpinLimit) {
        if (lane == 0) atomicOr(err, 1u);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  __syncthreads();
}

// Count this workgroup's output block as finished (after all its stores).
__device__ __forceinline__ void flow_signal(uint32_t* ctr) {
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this thread's stores are done
  __syncthreads();
  if (threadIdx.x == 0) atomicAdd(ctr, 1u);
}

struct FlowHooks {
  static constexpr bool kDevOut = true;
  static constexpr int kPending = 0;
  const uint32_t* wctr;  // null: nothing to wait for
  int wn;
  uint32_t wtarget;
  uint32_t* dctr;        // null: nothing to count
  uint32_t* err;
  uint64_t* trace;       // null, or this workgroup's 4 trace words
  __device__ __forceinline__ void wait() {
    if (wctr) flow_wait(wctr, wn, wtarget, err);
    if (trace && threadIdx.x == 0) trace[1] = __builtin_amdgcn_s_memrealtime();
  }
  __device__ __forceinline__ void after_issue() {}
  __device__ __forceinline__ void done() {
    if (dctr) flow_signal(dctr);
  }
  // the workgroup's end (every role, including a K split's early exit)
  __device__ __forceinline__ void finish() {
    if (trace && threadIdx.x == 0) trace[2] = __builtin_amdgcn_s_memrealtime();
  }
};

template <int MT, int EPI>
__device__ __forceinline__ void flow_gemm(const GemmArgs& a, int ns, int nsplit, int n_cb, int u,
                                          unsigned char* smem, FlowHooks& hk) {
  const SkinnyCoord co{u % n_cb, u / n_cb, 0};
  switch (ns) {
    case 1:
      if constexpr (EPI != EPI_SILU)
        skinny_tile<MT, 1, EPI, true, true>(a, co, nsplit, n_cb, *(SkinnySmem<MT, 1, EPI>*)smem, hk);
      break;
    case 2:
      skinny_tile<MT, 2, EPI, true, true>(a, co, nsplit, n_cb, *(SkinnySmem<MT, 2, EPI>*)smem, hk);
      break;
    case 4:
      skinny_tile<MT, 4, EPI, true, true>(a, co, nsplit, n_cb, *(SkinnySmem<MT, 4, EPI>*)smem, hk);
      break;
  }
}

template <int MT, int DH>
__global__ __launch_bounds__(512, 4) void flow_step(FlowArgs f) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int id = blockIdx.x;
  const int nlay = f.L * f.per_layer;
  FlowHooks hk{nullptr, 8, 0u, nullptr, f.err, f.trace ? f.trace + 4 * (size_t)id : nullptr};
  if (hk.trace && threadIdx.x == 0) {
    uint32_t hw;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
    uint32_t xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    hk.trace[0] = __builtin_amdgcn_s_memrealtime();
    hk.trace[3] = ((uint64_t)xcc << 32) | hw;
  }
  if (id >= nlay) {  // LM head: waits for the last layer's down GEMM
    const FlowLayer& last = f.layers[f.L - 1];
    GemmArgs a = f.g[FG_LM];
    a.Ahi = (const uint4*)last.n_out_hi;
    a.Alo = (const uint4*)last.n_out_lo;
    a.ss = last.ss_out;
    hk.wctr = f.cnt + (size_t)(f.L - 1) * f.cstride + f.c_down;
    hk.wtarget = (uint32_t)f.n_cb[FG_DOWN];
    flow_gemm<MT, EPI_LM>(a, f.ns[FG_LM], f.splits[FG_LM], f.n_cb[FG_LM], id - nlay, smem, hk);
    hk.finish();
    return;
  }
  const int l = id / f.per_layer, r = id - l * f.per_layer;
  uint32_t* cl = f.cnt + (size_t)l * f.cstride;
  const FlowLayer ly = f.layers[l];
  if (r < f.ph[FL_ATTN]) {  // QKV: waits for the previous layer's down GEMM
    const int u = r;
    GemmArgs a = f.g[FG_QKV];
    a.W = ly.qkv;
    a.kv = ly.kv;
    a.Ahi = (const uint4*)ly.n_in_hi;
    a.Alo = (const uint4*)ly.n_in_lo;
    a.ss = ly.ss_in;
    a.Q = ly.q;
    if (l > 0) {
      hk.wctr = cl - f.cstride + f.c_down;
      hk.wtarget = (uint32_t)f.n_cb[FG_DOWN];
    }
    // the kv-head group the block's columns belong to (q, k or v of group g)
    const int col0 = (u % f.n_cb[FG_QKV]) * f.ns[FG_QKV] * 16;
    const int g = col0 < a.q_cols ? col0 / (f.G * f.dh)
                                  : (col0 < a.q_cols + a.kv_cols ? col0 - a.q_cols : col0 - a.q_cols - a.kv_cols) / f.dh;
    hk.dctr = cl + g;
    flow_gemm<MT, EPI_QKV>(a, f.ns[FG_QKV], f.splits[FG_QKV], f.n_cb[FG_QKV], u, smem, hk);
  } else if (r < f.ph[FL_MERGE]) {  // attention chunk: waits for its group's QKV blocks
    const int u = r - f.ph[FL_ATTN];
    ConstItem* ip = (ConstItem*)f.items + u;
    AttnArgs a = f.attn;
    a.kv = ly.kv;
    a.Q = ly.q;
    a.Ohi = ly.o_hi;
    a.Olo = ly.o_lo;
    hk.wctr = cl + ip->g;
    hk.wn = 1;
    hk.wtarget = f.qkv_group_target;
    hk.dctr = ip->nch == 1 ? cl + f.c_oin + (u & 7) : cl + f.c_unit + ip->pad4;
    attn_item<DH, 2, 8, 1, true>(a, ip, smem, hk);
  } else if (r < f.ph[FL_O]) {  // merge slice: waits for every chunk of its unit
    const int u = r - f.ph[FL_MERGE];
    const AttnItem hd = f.heads[u / f.merge_spb];
    flow_wait(cl + f.c_unit + hd.pad4, 1, (uint32_t)hd.nch, f.err);
    if (hk.trace && threadIdx.x == 0) hk.trace[1] = __builtin_amdgcn_s_memrealtime();
    CombineArgs cb = f.comb;
    cb.Ohi = ly.o_hi;
    cb.Olo = ly.o_lo;
    combine_slice<DH, 4, 512, true>(cb, hd, u % f.merge_spb);
    flow_signal(cl + f.c_oin + (u & 7));
  } else if (r < f.ph[FL_GU]) {  // O: waits for every attention output of the layer
    const int u = r - f.ph[FL_O];
    GemmArgs a = f.g[FG_O];
    a.W = ly.o;
    a.gain_next = ly.g_mlp;
    a.Ahi = (const uint4*)ly.o_hi;
    a.Alo = (const uint4*)ly.o_lo;
    a.X = const_cast<float*>(ly.x_in);
    a.X_out = ly.x_mid;
    a.Nhi = ly.n_mid_hi;
    a.Nlo = ly.n_mid_lo;
    a.ss_out = ly.ss_mid;
    hk.wctr = cl + f.c_oin;
    hk.wtarget = f.oin_target;
    hk.dctr = cl + f.c_o + (u & 7);
    flow_gemm<MT, EPI_RESID>(a, f.ns[FG_O], f.splits[FG_O], f.n_cb[FG_O], u, smem, hk);
  } else if (r < f.ph[FL_DOWN]) {  // gate/up: waits for the O GEMM
    const int u = r - f.ph[FL_GU];
    GemmArgs a = f.g[FG_GU];
    a.W = ly.gu;
    a.Ahi = (const uint4*)ly.n_mid_hi;
    a.Alo = (const uint4*)ly.n_mid_lo;
    a.ss = ly.ss_mid;
    a.act_hi = ly.a_hi;
    a.act_lo = ly.a_lo;
    hk.wctr = cl + f.c_o;
    hk.wtarget = (uint32_t)f.n_cb[FG_O];
    hk.dctr = cl + f.c_gu + (u & 7);
    flow_gemm<MT, EPI_SILU>(a, f.ns[FG_GU], f.splits[FG_GU], f.n_cb[FG_GU], u, smem, hk);
  } else {  // down: waits for the gate/up GEMM
    const int u = r - f.ph[FL_DOWN];
    GemmArgs a = f.g[FG_DOWN];
    a.W = ly.down;
    a.gain_next = l + 1 < f.L ? f.layers[l + 1].g_attn : f.g_final;
    a.Ahi = (const uint4*)ly.a_hi;
    a.Alo = (const uint4*)ly.a_lo;
    a.X = ly.x_mid;
    a.X_out = ly.x_out;
    a.Nhi = ly.n_out_hi;
    a.Nlo = ly.n_out_lo;
    a.ss_out = ly.ss_out;
    hk.wctr = cl + f.c_gu;
    hk.wtarget = (uint32_t)f.n_cb[FG_GU];
    hk.dctr = cl + f.c_down + (u & 7);
    flow_gemm<MT, EPI_RESID>(a, f.ns[FG_DOWN], f.splits[FG_DOWN], f.n_cb[FG_DOWN], u, smem, hk);
  }
  hk.finish();
}

template <int MT>
static size_t flow_lds_mt(int dh) {
  size_t b = 0;
  b = std::max(b, sizeof(SkinnySmem<MT, 4, EPI_QKV>));
  b = std::max(b, sizeof(SkinnySmem<MT, 4, EPI_RESID>));
  b = std::max(b, sizeof(SkinnySmem<MT, 4, EPI_SILU>));
  b = std::max(b, sizeof(SkinnySmem<MT, 4, EPI_LM>));
  b = std::max(b, attn_lds_bytes(dh, 2));
  return b;
}

// Head dim 128 only: the 8-wave attention workgroup stages a page of a head
// dim 64 head with fewer 16-byte units than it has threads.
bool flow_supported(int MT, int dh, int np, const int* ns) {
  if (MT < 1 || MT > 2 || dh != 128 || np != 2) return false;
  for (int f = 0; f < FG_N; ++f)
    if (ns[f] != 1 && ns[f] != 2 && ns[f] != 4) return false;
  return ns[FG_GU] != 1;
}

template <int MT, int DH>
static void launch_flow_t(const FlowArgs& f, hipStream_t s) {
  const size_t lds = flow_lds_mt<MT>(DH);
  hvd_launch((flow_step<MT, DH>), dim3(f.L * f.per_layer + f.n_lm), dim3(512), (uint32_t)lds, s, f);
}

hipError_t launch_flow(const FlowArgs& f, int MT, hipStream_t s) {
  int ns[FG_N];
  for (int i = 0; i < FG_N; ++i) ns[i] = f.ns[i];
  if (!flow_supported(MT, f.dh, f.np, ns)) return hipErrorInvalidValue;
  // every pointer the kernel dereferences without a per-layer override
  // every pointer the kernel takes from here rather than from the layer table
  if (!f.layers || !f.cnt || !f.err || !f.g_final || !f.items || !f.g[FG_LM].W || !f.g[FG_LM].part_val ||
      !f.g[FG_LM].part_idx || !f.attn.pt || !f.attn.part_o || !f.attn.part_ml ||
      (f.ph[FL_O] > f.ph[FL_MERGE] && !f.heads))
    return hipErrorInvalidValue;
  for (int i = 0; i < FG_N; ++i)
    if (!f.g[i].part || !f.g[i].cnt) return hipErrorInvalidValue;
  if (!f.g[FG_QKV].pt || !f.g[FG_QKV].rows || !f.g[FG_QKV].rope) return hipErrorInvalidValue;
  if (MT == 1) launch_flow_t<1, 128>(f, s);
  else launch_flow_t<2, 128>(f, s);
  return hipGetLastError();
}

template <int MT, int DH>
static hipError_t flow_set_lds_t() {
  return hipFuncSetAttribute((const void*)flow_step<MT, DH>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)flow_lds_mt<MT>(DH));
}

hipError_t flow_set_lds_limit() {
  hipError_t e = flow_set_lds_t<1, 128>();
  if (e == hipSuccess) e = flow_set_lds_t<2, 128>();
  return e;
}

}  // namespace hvd
