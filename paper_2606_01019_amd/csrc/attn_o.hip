// Attention, split-KV merge and O GEMM of one layer as one launch (gfx950).
//
// At small verify batches the attention and its merge are short, latency-
// bound passes during which HBM idles, and the O GEMM right after them
// streams the Hq*dh x D output projection (32 MB for the 8B shape); a read
// of that size costs ~4 us of launch, first-byte latency and drain on top
// of its transfer time.  Here one grid of 256-thread workgroups in two
// roles, all resident at once (two workgroups per CU), runs the three:
//  * attention workgroups (the first n_attn): their attention items, each
//    writing chunk partials (or a one-chunk item's normalised output) with
//    device-scope (write-through) stores; once every attention workgroup
//    has counted its items done, the merge of the chunk partials (the same
//    per-row rescaled sums as the stand-alone merge), spread over them;
//  * O workgroups (one per 16-column strip): from the start, the strip's
//    weights into registers (each of the 4 waves holds every 4th K step)
//    and the residual epilogue's inputs; once every merge is counted, the
//    product with the attention output (fp16 hi + lo activation pair, as
//    the stand-alone GEMM), the waves' K ranges reduced in LDS in a fixed
//    order, and the residual epilogue (residual add, next RMSNorm's
//    operand, sums of squares).
// So the O weights stream while the attention runs, and the merge needs no
// launch of its own.  The roles sit in different workgroups because a
// wave's memory counter completes in issue order: a wave with the weight
// strip in flight could not wait for any later load of its own sooner.
//
// Counting: 32 counters, 128 bytes apart, per phase; attention workgroup r
// adds to counter r % 32 and one wave polls all of them.  They are zeroed
// once per step and layer l waits for (l + 1) * n_attn arrivals.  Every
// wait is bounded (kAoSpinLimit polls); a wait that gives up sets bit 0 of
// *err, which the host reports as a failed step.
//
// Coherence: the L2 caches of the 8 XCDs are not coherent with each other.
// Partials and the attention output are written with device-scope stores
// and read with ordinary loads: each is a buffer no workgroup of the launch
// reads before the count that covers it is complete (a reader's L2 holds
// no copy from earlier in the launch).  A producer waits for its stores
// (vmcnt(0)) before it counts itself done.  Everything else (weights, K/V,
// query rows, residual) was written by earlier launches.
//
// Forward progress needs every workgroup resident: n_attn + strips is at
// most two per CU (the register and LDS budget allow two), and the host
// launches it only when the GPU has enough CUs.
#include "attn.h"
#include "skinny.h"

namespace hvd {

constexpr uint32_t kAoSpinLimit = 1u << 20;
constexpr int kAoQS = 8;     // merge lanes per (row, 8 dims)
constexpr int kAoWaves = 4;  // waves per workgroup

__device__ __forceinline__ void ao_signal(uint32_t* cnt, int r) {
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this thread's stores are done
  __syncthreads();
  if (threadIdx.x == 0) atomicAdd(cnt + (r % kAoSlots) * kAoSlotWords, 1u);
}

__device__ __forceinline__ void ao_wait(const uint32_t* cnt, uint32_t target, uint32_t* err) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    for (uint32_t it = 0;; ++it) {
      uint32_t v = lane < kAoSlots ? ld_u32_dev(cnt + lane * kAoSlotWords) : 0u;
#pragma unroll
      for (int o = 1; o < kAoSlots; o <<= 1) v += __shfl_xor(v, o);
      v = __builtin_amdgcn_readfirstlane(v);
      if (v >= target) break;
      if (it >= kAoSpinLimit) {
        if (lane == 0) atomicOr(err, 1u);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
}

// Attention items of this launch write their outputs with device-scope stores.
struct AoAttnHooks {
  static constexpr bool kDevOut = true;
  static constexpr int kPending = 0;
  __device__ __forceinline__ void wait() {}
  __device__ __forceinline__ void after_issue() {}
  __device__ __forceinline__ void done() {}
};

constexpr size_t ao_attn_lds(int np) { return (size_t)np * kPage * 128 * 2 * 2 * (np <= 4 ? 2 : 1); }

template <int MT>
struct AoSmem {
  float red[kAoWaves][MT][256];
  float tile[MT * 16][16 + 1];
  EpiPre<MT, 1, EPI_RESID> pre;
};

template <int MT>
constexpr size_t ao_lds(int np) {
  return ao_attn_lds(np) > sizeof(AoSmem<MT>) ? ao_attn_lds(np) : sizeof(AoSmem<MT>);
}

template <int NP, int TPW>
__device__ __forceinline__ void ao_attention(const AttnOArgs& a, int r, unsigned char* smem) {
  constexpr int DH = 128, NT = 64 * kAoWaves;
  uint64_t* tr = a.trace ? a.trace + (size_t)blockIdx.x * kAoTraceWords : nullptr;
  auto stamp = [&](int i) __attribute__((always_inline)) {
    if (tr && threadIdx.x == 0) tr[i] = __builtin_amdgcn_s_memrealtime();
  };
  stamp(0);
  AoAttnHooks hk;
  for (int it = r; it < a.n_items; it += a.n_attn) {
    attn_item<DH, NP, kAoWaves, TPW, false>(a.at, (ConstItem*)a.at.items + it, smem, hk);
    __syncthreads();  // the next item restages the LDS buffers
  }
  stamp(1);
  ao_signal(a.cnt, r);
  stamp(2);
  ao_wait(a.cnt, a.target, a.err);
  stamp(3);
  const int n_units = a.n_heads * a.merge_spb;
  for (int u = r; u < n_units; u += a.n_attn) {
    const AttnItem& hd = a.cb.heads[u / a.merge_spb];
    if (hd.k >= 0) combine_slice<DH, kAoQS, NT, true, false>(a.cb, hd, u % a.merge_spb);
  }
  stamp(4);
  ao_signal(a.cnt + kAoSlots * kAoSlotWords, r);
  stamp(5);
}

template <int MT, int WK>
__device__ __forceinline__ void ao_oproj(const AttnOArgs& a, int w, unsigned char* smem) {
  constexpr int NT = 64 * kAoWaves;
  AoSmem<MT>& sm = *(AoSmem<MT>*)smem;
  const GemmArgs& go = a.go;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  uint64_t* tr = a.trace ? a.trace + (size_t)blockIdx.x * kAoTraceWords : nullptr;
  auto stamp = [&](int i) __attribute__((always_inline)) {
    if (tr && tid == 0) tr[i] = __builtin_amdgcn_s_memrealtime();
  };
  stamp(0);
  // epilogue inputs (residual tile, next norm's gain), then the strip
  EpiRegs<MT, 1, EPI_RESID> er;
  epi_issue<MT, 1, EPI_RESID>(go, er, w, 0, MT);
  const u32x4* wp =
      (const u32x4*)go.W + (size_t)(w >> 2) * go.wg + (size_t)(w & 3) * 64 + (size_t)wave * go.wk + lane;
  // Every workgroup reads all of the attention output later; the workgroups
  // of one XCD take the K steps in orders rotated by w / 8 so they do not all
  // ask its L2 for the same lines at once.  wr[j] holds rotated step j.
  const int rot = (w >> 3) % WK;
  u32x4 wr[WK];
#pragma unroll
  for (int j = 0; j < WK; ++j) {
    const int jj = j + rot < WK ? j + rot : j + rot - WK;
    wr[j] = __builtin_nontemporal_load(wp + (size_t)jj * kAoWaves * go.wk);
  }
  epi_settle<MT, 1, EPI_RESID>(er);
  epi_commit<MT, 1, EPI_RESID>(go, er, sm.pre, w, 0, MT);
  stamp(1);
  ao_wait(a.cnt + kAoSlots * kAoSlotWords, a.target, a.err);
  stamp(6);
  // the attention output times the resident strip: wave v holds K steps v,
  // v + 4, ... (in the rotated order)
  const size_t astride = (size_t)go.MTtot * 64;
  const u32x4* hp = (const u32x4*)go.Ahi;
  const u32x4* lp = (const u32x4*)go.Alo;
  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < WK; ++j) {
    const int jj = j + rot < WK ? j + rot : j + rot - WK;
    const size_t kt = (size_t)(wave + kAoWaves * jj);
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const u32x4 ah = hp[kt * astride + m * 64 + lane];
      const u32x4 al = lp[kt * astride + m * 64 + lane];
      acc[m] = mfma_f16(ah, wr[j], acc[m]);
      acc[m] = mfma_f16(al, wr[j], acc[m]);
    }
  }
  stamp(2);
  // reduce the waves' K ranges through LDS in a fixed order
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int i = 0; i < 4; ++i) sm.red[wave][m][lane * 4 + i] = acc[m][i];
  __syncthreads();
  for (int e = tid; e < MT * 256; e += NT) {
    const int m = e / 256, li = e % 256;
    const int ln = li >> 2, i = li & 3;
    const float v = (sm.red[0][m][li] + sm.red[1][m][li]) + (sm.red[2][m][li] + sm.red[3][m][li]);
    sm.tile[m * 16 + (ln >> 4) * 4 + i][ln & 15] = v;
  }
  __syncthreads();
  gemm_epilogue<MT, 1, EPI_RESID, false>(go, sm.tile, sm.pre, w, 0, MT);
  stamp(7);
}

// MT: row tiles of the O GEMM; NP: pages per attention sub-chunk; TPW: row
// tiles per wave of an attention item (64 or 128 query rows per item); WK:
// K steps per wave of the O GEMM (K = kAoWaves * WK * 32).
template <int MT, int NP, int TPW, int WK>
__global__ __launch_bounds__(64 * kAoWaves, 2) void attn_o(AttnOArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int b = blockIdx.x;
  if (b < a.n_attn) ao_attention<NP, TPW>(a, b, smem);
  else ao_oproj<MT, WK>(a, b - a.n_attn, smem);
}

bool attn_o_supported(int dh, int np, int MT, int KT, int NT, int n_cus) {
  return dh == 128 && (np == 2 || np == 4) && (MT == 1 || MT == 2) && (KT == 32 || KT == 64 || KT == 128) &&
         NT >= 1 && NT <= n_cus;
}

template <int MT, int NP, int TPW, int WK>
static void launch_attn_o_t(const AttnOArgs& a, hipStream_t s) {
  hvd_launch((attn_o<MT, NP, TPW, WK>), dim3(a.n_attn + a.go.NT), dim3(64 * kAoWaves), (uint32_t)ao_lds<MT>(NP), s,
             a);
}

template <int MT, int NP, int TPW>
static hipError_t launch_attn_o_k(const AttnOArgs& a, hipStream_t s) {
  switch (a.go.KT) {
    case 32: launch_attn_o_t<MT, NP, TPW, 8>(a, s); break;
    case 64: launch_attn_o_t<MT, NP, TPW, 16>(a, s); break;
    case 128: launch_attn_o_t<MT, NP, TPW, 32>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int MT, int NP>
static hipError_t launch_attn_o_np(const AttnOArgs& a, int rows_per_item, hipStream_t s) {
  if (rows_per_item == 64) return launch_attn_o_k<MT, NP, 1>(a, s);
  if (rows_per_item == 128) return launch_attn_o_k<MT, NP, 2>(a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_attn_o(const AttnOArgs& a, int np, int rows_per_item, int MT, hipStream_t s) {
  if (a.at.dh != 128 || a.go.MTtot != MT || !a.cnt || !a.err || !a.go.W || !a.go.X || !a.go.Ahi || !a.go.Alo ||
      !a.go.gain_next || !a.go.Nhi || !a.go.Nlo || !a.go.ss_out || !a.at.items || !a.at.Q || !a.at.kv ||
      !a.at.pt || !a.at.part_o || !a.at.part_ml || (a.n_heads > 0 && (!a.cb.heads || a.merge_spb < 1)) ||
      a.cb.rpi != rows_per_item || a.n_attn < 1)
    return hipErrorInvalidValue;
  if (MT == 1 && np == 2) return launch_attn_o_np<1, 2>(a, rows_per_item, s);
  if (MT == 1 && np == 4) return launch_attn_o_np<1, 4>(a, rows_per_item, s);
  if (MT == 2 && np == 2) return launch_attn_o_np<2, 2>(a, rows_per_item, s);
  if (MT == 2 && np == 4) return launch_attn_o_np<2, 4>(a, rows_per_item, s);
  return hipErrorInvalidValue;
}

template <int MT, int NP, int TPW>
static hipError_t ao_set_lds_t() {
  hipError_t e = hipSuccess;
  for (const void* f : {(const void*)attn_o<MT, NP, TPW, 8>, (const void*)attn_o<MT, NP, TPW, 16>,
                        (const void*)attn_o<MT, NP, TPW, 32>})
    if (e == hipSuccess) e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)ao_lds<MT>(NP));
  return e;
}

hipError_t attn_o_set_lds_limit() {
  hipError_t e = ao_set_lds_t<1, 2, 1>();
  if (e == hipSuccess) e = ao_set_lds_t<1, 4, 1>();
  if (e == hipSuccess) e = ao_set_lds_t<2, 2, 1>();
  if (e == hipSuccess) e = ao_set_lds_t<2, 4, 1>();
  if (e == hipSuccess) e = ao_set_lds_t<1, 2, 2>();
  if (e == hipSuccess) e = ao_set_lds_t<1, 4, 2>();
  if (e == hipSuccess) e = ao_set_lds_t<2, 2, 2>();
  if (e == hipSuccess) e = ao_set_lds_t<2, 4, 2>();
  return e;
}

}  // namespace hvd
