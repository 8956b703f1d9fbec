// Weight-streaming GEMMs of the verify forward (gfx950, MFMA 16x16x32 f16).
//
// Y[m, n] = sum_k A[m, k] * W[n, k] with W the weight in torch Linear layout
// (bf16 values, stored as fp16: the conversion is exact but for magnitudes
// below 2^-17), pre-packed so that one 16x32 B-operand fragment is 1 KB
// contiguous (one 16-byte load per lane), and A the activation carried as a
// hi + lo pair of fp16 fragments (two MFMAs per tile: hi*W + lo*W keeps ~22
// significant bits of the fp32 activation; the MFMA pipe is idle in this
// HBM-bound regime).
//
// Work split: a workgroup of 8 waves owns NS strips of 16 output columns
// (NS = 1, 2, 4 or 8, chosen per GEMM so the launch has enough workgroups)
// and up to 64 rows; its waves take the K steps round-robin.  Each wave
// streams the NS strips' weight fragments of a K step (the 4 strips of a
// 64-column group are contiguous after packing) and reuses each activation
// fragment for all NS strips, with a prefetch queue of depth U (weights and
// activations issued together so the in-order vmcnt waits never stall on a
// younger load).  The epilogue's own inputs (row sums of squares, residual
// tile, rotary factors, KV page ids) are fetched into LDS right after the
// first weight loads, so no dependent memory round trip is left for the end.
// Partial sums are reduced through LDS in a fixed order.  When the column
// blocks alone are too few to keep enough weight bytes in flight, K is also
// split across workgroups (gridDim.y): each publishes its partial tile with
// write-through stores and counts its arrival; the last split to arrive sums
// all splits in split order (deterministic) and runs the epilogue, so a K
// split costs no second kernel.  Fused epilogues:
//   EPI_QKV   inverse-RMS row scale, rotary embedding on q and k (pairs are
//             adjacent columns after the load-time permutation), q -> Q
//             buffer, k/v -> paged fp16 KV cache;
//   EPI_RESID residual add into the fp32 stream X, then the next RMSNorm's
//             gain and hi/lo split into the next GEMM's A operand, and
//             per-strip sums of squares for the next inverse RMS;
//   EPI_SILU  inverse-RMS scale, silu(gate) * up into the down GEMM's A;
//   EPI_LM    inverse-RMS scale, optional fp32 logits, per-row max / lowest
//             argmax over the workgroup's columns.
#include "skinny.h"

namespace hvd {

// Stand-alone launch: workgroup (blockIdx) -> output block.
template <int MT, int NS, int EPI, bool HL>
__global__ __launch_bounds__(512, gemm_occupancy(MT)) void gemm_skinny(GemmArgs a) {
  __shared__ SkinnySmem<MT, NS, EPI> sm;
  NoHooks hk;
  skinny_tile<MT, NS, EPI, HL, false>(a, skinny_coord(), (int)gridDim.y, (int)gridDim.x, sm, hk);
}

template <int MT, int NS, int EPI, bool HL>
static void launch_one(const GemmArgs& a, int splits, int mblocks, hipStream_t s) {
  const dim3 grid(a.NT / NS, splits, mblocks);
  hvd_launch((gemm_skinny<MT, NS, EPI, HL>), grid, dim3(512), 0, s, a);
}

template <int NS, int EPI>
static hipError_t launch_ns(const GemmArgs& a, int splits, int mblocks, int mt, bool hi_lo, hipStream_t s) {
  // single-pass activations only for the MLP and LM-head GEMMs at 3-4 row tiles
  constexpr bool kSingle = EPI == EPI_SILU || EPI == EPI_RESID || EPI == EPI_LM;
  switch (mt) {
    case 1:
      if constexpr (kSingle) {
        if (!hi_lo) {
          launch_one<1, NS, EPI, false>(a, splits, mblocks, s);
          break;
        }
      }
      launch_one<1, NS, EPI, true>(a, splits, mblocks, s);
      break;
    case 2:
      if constexpr (kSingle) {
        if (!hi_lo) {
          launch_one<2, NS, EPI, false>(a, splits, mblocks, s);
          break;
        }
      }
      launch_one<2, NS, EPI, true>(a, splits, mblocks, s);
      break;
    case 5:  // one block of five row tiles (65-80 rows): the weights are read once.  Single
             // pass (8 strips for gate/up and the LM head only: the residual epilogue's LDS
             // would not fit), or the hi + lo pair for the residual GEMMs at up to 4 strips
      if constexpr (kSingle && (NS <= 4 || EPI == EPI_SILU || EPI == EPI_LM)) {
        if (!hi_lo) {
          launch_one<5, NS, EPI, false>(a, splits, mblocks, s);
          break;
        }
      }
      if constexpr (EPI == EPI_RESID && NS <= 4) {
        if (hi_lo) {
          launch_one<5, NS, EPI, true>(a, splits, mblocks, s);
          break;
        }
      }
      return hipErrorInvalidValue;
    case 3:
    case 4:
      if constexpr (NS == 8) {  // 8-strip blocks at 3-4 row tiles: single pass only (LDS)
        if constexpr (kSingle) {
          if (!hi_lo) {
            if (mt == 3) launch_one<3, 8, EPI, false>(a, splits, mblocks, s);
            else launch_one<4, 8, EPI, false>(a, splits, mblocks, s);
            break;
          }
        }
        return hipErrorInvalidValue;
      } else if constexpr (NS <= 4) {
        if (kSingle && !hi_lo) {
          if constexpr (kSingle) {
            if (mt == 3) launch_one<3, NS, EPI, false>(a, splits, mblocks, s);
            else launch_one<4, NS, EPI, false>(a, splits, mblocks, s);
          }
        } else if (mt == 3) {
          launch_one<3, NS, EPI, true>(a, splits, mblocks, s);
        } else {
          launch_one<4, NS, EPI, true>(a, splits, mblocks, s);
        }
        break;
      }
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& a, int ns, int splits, int mblocks, int mt, bool hi_lo, hipStream_t s) {
  switch (ns) {
    case 1:
      if constexpr (EPI != EPI_SILU) return launch_ns<1, EPI>(a, splits, mblocks, mt, hi_lo, s);
      return hipErrorInvalidValue;
    case 2: return launch_ns<2, EPI>(a, splits, mblocks, mt, hi_lo, s);
    case 4: return launch_ns<4, EPI>(a, splits, mblocks, mt, hi_lo, s);
    case 8: return launch_ns<8, EPI>(a, splits, mblocks, mt, hi_lo, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(int epi, const GemmArgs& a, int ns, int splits, int mblocks, int mt_block, bool hi_lo,
                       hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_epi<EPI_QKV>(a, ns, splits, mblocks, mt_block, hi_lo, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, ns, splits, mblocks, mt_block, hi_lo, s);
    case EPI_SILU: return launch_epi<EPI_SILU>(a, ns, splits, mblocks, mt_block, hi_lo, s);
    case EPI_LM: return launch_epi<EPI_LM>(a, ns, splits, mblocks, mt_block, hi_lo, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace hvd
