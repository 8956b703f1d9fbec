// Verify attention over the paged fp16 KV cache (gfx950, MFMA 16x16x32 f16).
//
// For one sequence, the (k+1) query rows of the verify step times the
// Hq/Hkv q-heads of one kv head g form R = (k+1)*group query vectors; row
// r = i*group + hh is draft row i (K/V at position ctx+i) of q-head
// g*group+hh and may attend to key positions 0..ctx+i.  For a token tree,
// row i is the pending token (i = 0) or node i-1, and it attends to
// positions 0..ctx-1 and to the positions of its ancestors and itself.  A
// workgroup (4 or 8 waves) handles one KV chunk of one (sequence, kv head,
// row group of 64, 128 or 256 rows), in sub-chunks of up to kAttnChunk
// positions: it copies a sub-chunk's K and V pages into LDS with every load
// in flight at once (decode-size chunks are latency-bound, not
// bandwidth-bound), then each wave runs its 1 or 2 row tiles over it,
// carrying the online-softmax state to the next sub-chunk.
//
// Scores are computed transposed, S^T = K Q^T, so the fp32 C fragment of a
// lane holds 4 key positions of one query row; the same registers, converted
// to fp16, are the B operand of O^T = V^T P^T with the contraction index
// permuted consistently on both operands (positions {4g..4g+3, 16+4g..16+4g+3}
// for lane group g).  V is stored transposed inside each 16-token page
// ([dh][16]) and kept transposed in LDS, where each row's positions are
// regrouped so that a lane group's eight contraction positions of a 32-key
// block sit in one 16-byte granule (one LDS read per V fragment).  LDS rows
// are XOR-swizzled so the 16 lanes of a fragment read hit distinct banks.
// Online softmax in fp32 base 2 (the hardware exp2, whose results below
// 2^-126 flush to zero); rows see only their causal prefix (for a token
// tree: the context and the positions of their own path, from a per-row
// ancestor mask); keys at
// positions >= ctx+k+1 are never used (their contents may be stale).
// A single-chunk item writes the normalized output straight into the O GEMM's
// hi/lo operand; multi-chunk items write (m, l, unnormalized O) partials that
// attn_combine merges.
#include "attn.h"

namespace hvd {

template <int DH, int NP, int NW, int TPW>
__global__ __launch_bounds__(64 * NW, attn_occupancy(DH, NP, NW)) void verify_attn(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  NoHooks hk;
  attn_item<DH, NP, NW, TPW, false>(a, (ConstItem*)a.items + blockIdx.x, smem, hk);
}

template <int DH, int QS>
__global__ __launch_bounds__(256) void attn_combine(CombineArgs a) {
  constexpr int RPB = 256 / (DH / 8 * QS);
  const int spb = (a.max_rows + RPB - 1) / RPB;
  const AttnItem hd = a.heads[blockIdx.x / spb];
  if (hd.k < 0) return;  // grid padding
  combine_slice<DH, QS, 256, false>(a, hd, blockIdx.x % spb);
}

int attn_pages_per_sub(int chunk) {
  int np = 2;
  while (np < kItemPages && np * kPage < chunk) np *= 2;
  return np;
}

// K and V of one sub-chunk, twice for the double-buffered sub-chunks (<= 4 pages)
size_t attn_lds_bytes(int dh, int np) { return (size_t)np * kPage * dh * 2 * 2 * (np <= 4 ? 2 : 1); }

template <int DH, int NW, int TPW>
static hipError_t launch_attn_dh(const AttnArgs& a, int n_items, int np, hipStream_t s) {
  const size_t lds = attn_lds_bytes(DH, np);
  const dim3 block(64 * NW);
  switch (np) {
    case 2: hvd_launch((verify_attn<DH, 2, NW, TPW>), dim3(n_items), block, lds, s, a); break;
    case 4: hvd_launch((verify_attn<DH, 4, NW, TPW>), dim3(n_items), block, lds, s, a); break;
    case 8: hvd_launch((verify_attn<DH, 8, NW, TPW>), dim3(n_items), block, lds, s, a); break;
    case 16:
      if constexpr (TPW == 1 || DH == 64) {
        hvd_launch((verify_attn<DH, 16, NW, TPW>), dim3(n_items), block, lds, s, a);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// rows_per_item: 64 (4 waves of one row tile), 128 (8 waves of one tile;
// 4 waves of two for head dim 64, whose page has too few 16-byte units for
// 8 waves) or 256 (8 waves of two tiles; head dim 128, sub-chunks of at most
// 8 pages so the staging registers fit two waves per SIMD)
hipError_t launch_attn(const AttnArgs& a, int n_items, int chunk, int rows_per_item, int max_np, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  // Sub-chunks of 2 pages for 64-row items, 4 otherwise (measured at
  // context 16384: smaller sub-chunks need fewer staging registers, so more
  // workgroups share a CU and hide each other's load latency; the next
  // sub-chunk's loads overlap the current one's MFMAs anyway)
  int np = attn_pages_per_sub(chunk);
  const int pref = rows_per_item == 64 ? 2 : 4;
  const int cap = max_np < pref ? max_np : pref;
  while (np > 2 && np > cap) np /= 2;
  switch (rows_per_item) {
    case 64:
      if (a.dh == 128) return launch_attn_dh<128, 4, 1>(a, n_items, np, s);
      if (a.dh == 64) return launch_attn_dh<64, 4, 1>(a, n_items, np, s);
      return hipErrorInvalidValue;
    case 128:
      if (a.dh == 128) return launch_attn_dh<128, 8, 1>(a, n_items, np, s);
      if (a.dh == 64) return launch_attn_dh<64, 4, 2>(a, n_items, np, s);
      return hipErrorInvalidValue;
    case 256:
      if (a.dh == 128) return launch_attn_dh<128, 8, 2>(a, n_items, np < 8 ? np : 8, s);
      return hipErrorInvalidValue;
    case 384:  // three row tiles per wave: 2-page sub-chunks only (register budget)
      if (a.dh != 128) return hipErrorInvalidValue;
      hvd_launch((verify_attn<128, 2, 8, 3>), dim3(n_items), dim3(512), attn_lds_bytes(128, 2), s, a);
      return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

template <int DH, int QS>
static void launch_combine_q(const CombineArgs& a, int n_heads, hipStream_t s) {
  constexpr int RPB = 256 / (DH / 8 * QS);
  hvd_launch((attn_combine<DH, QS>), dim3(n_heads * ((a.max_rows + RPB - 1) / RPB)), dim3(256), 0, s, a);
}

template <int DH>
static void launch_combine_dh(const CombineArgs& a, int n_heads, hipStream_t s) {
  if (a.rpi <= 64) launch_combine_q<DH, 8>(a, n_heads, s);
  else if (a.rpi <= 128) launch_combine_q<DH, 4>(a, n_heads, s);
  else launch_combine_q<DH, 2>(a, n_heads, s);
}

hipError_t launch_combine(const CombineArgs& a, int n_heads, hipStream_t s) {
  if (n_heads <= 0) return hipSuccess;
  if (a.max_rows <= 0 || a.max_rows > a.rpi) return hipErrorInvalidValue;
  if (a.dh == 128)
    launch_combine_dh<128>(a, n_heads, s);
  else if (a.dh == 64)
    launch_combine_dh<64>(a, n_heads, s);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <int DH, int NP, int NW, int TPW>
static hipError_t set_lds(void) {
  return hipFuncSetAttribute((const void*)verify_attn<DH, NP, NW, TPW>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)attn_lds_bytes(DH, NP));
}

template <int DH, int NW>
static hipError_t set_lds_tpw1(void) {
  hipError_t e = set_lds<DH, 2, NW, 1>();
  if (e == hipSuccess) e = set_lds<DH, 4, NW, 1>();
  if (e == hipSuccess) e = set_lds<DH, 8, NW, 1>();
  if (e == hipSuccess) e = set_lds<DH, 16, NW, 1>();
  return e;
}

hipError_t attn_set_lds_limit() {
  hipError_t e = set_lds_tpw1<128, 4>();
  if (e == hipSuccess) e = set_lds_tpw1<128, 8>();
  if (e == hipSuccess) e = set_lds_tpw1<64, 4>();
  if (e == hipSuccess) e = set_lds<64, 2, 4, 2>();
  if (e == hipSuccess) e = set_lds<64, 4, 4, 2>();
  if (e == hipSuccess) e = set_lds<64, 8, 4, 2>();
  if (e == hipSuccess) e = set_lds<64, 16, 4, 2>();
  if (e == hipSuccess) e = set_lds<128, 2, 8, 2>();
  if (e == hipSuccess) e = set_lds<128, 4, 8, 2>();
  if (e == hipSuccess) e = set_lds<128, 8, 8, 2>();
  if (e == hipSuccess) e = set_lds<128, 2, 8, 3>();
  return e;
}

}  // namespace hvd
