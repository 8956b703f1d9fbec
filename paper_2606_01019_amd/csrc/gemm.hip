// Weight-streaming GEMMs of the verify forward (gfx950, MFMA 16x16x32 bf16).
//
// Y[m, n] = sum_k A[m, k] * W[n, k] with W the bf16 weight in torch Linear
// layout, pre-packed so that one 16x32 B-operand fragment is 1 KB contiguous
// (one 16-byte load per lane), and A the activation carried as a hi + lo pair
// of bf16 fragments (two MFMAs per tile: hi*W + lo*W keeps ~16 significant
// bits of the fp32 activation; the MFMA pipe is idle in this HBM-bound regime).
//
// Work split: a workgroup of 8 waves owns NS strips of 16 output columns
// (NS = 1, 2 or 4, chosen per GEMM so the launch has enough workgroups) and
// up to 64 rows; its waves split K into 8 contiguous pieces.  Each wave
// streams the NS strips' weight fragments of a K step (the 4 strips of a
// 64-column group are contiguous after packing) and reuses each activation
// fragment for all NS strips, with a prefetch queue of depth U (weights and
// activations issued together so the in-order vmcnt waits never stall on a
// younger load).  Partial sums are reduced through LDS in a fixed order.
// When the column blocks alone are too few to keep enough weight bytes in
// flight, K is also split across workgroups (gridDim.y): each publishes its
// partial tile and a second kernel sums the splits in order (deterministic;
// a kernel boundary is cheaper here than device-scope release fences).  The
// fused epilogue:
//   EPI_QKV   inverse-RMS row scale, rotary embedding on q and k (pairs are
//             adjacent columns after the load-time permutation), q -> Q
//             buffer, k/v -> paged fp16 KV cache;
//   EPI_RESID residual add into the fp32 stream X, then the next RMSNorm's
//             gain and hi/lo split into the next GEMM's A operand, and
//             per-strip sums of squares for the next inverse RMS;
//   EPI_SILU  inverse-RMS scale, silu(gate) * up into the down GEMM's A;
//   EPI_LM    inverse-RMS scale, optional fp32 logits, per-row max / lowest
//             argmax over the workgroup's columns.
#include "common.h"
#include "kernels.h"

namespace hvd {

// Prefetch depth: K steps in flight per wave.  A stage holds NS weight and
// 2*MT activation fragments (4 VGPRs each); up to 2 row tiles the kernel is
// sized for 4 waves per SIMD (two 8-wave workgroups per CU), beyond that 2.
constexpr int gemm_occupancy(int MT) { return MT <= 2 ? 4 : 2; }
constexpr int gemm_depth(int MT, int NS) {
  const int budget = gemm_occupancy(MT) == 4 ? 80 : 160;
  const int d = budget / (4 * (NS + 2 * MT));
  return d < 1 ? 1 : (d > 8 ? 8 : d);
}

constexpr int kKG = 8;      // waves per workgroup, each a contiguous K range

// Fused epilogue on the reduced [rows][cols] tile of one workgroup.
template <int MT, int kNS, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& a, float (*tile)[kNS * 16 + 1], const float* inv_rms,
                                              int cb, int mt0, int mcount) {
  constexpr int COLS = kNS * 16;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int rows_here = mcount * 16;
  const int row0 = mt0 * 16;
  const int col0 = cb * COLS;
  if constexpr (EPI == EPI_QKV) {
    const int half = a.dh >> 1;
    for (int e = tid; e < rows_here * (COLS / 2); e += 512) {
      int r = e / (COLS / 2), cp = (e % (COLS / 2)) * 2;
      int R = row0 + r;
      if (R >= a.M) continue;
      float v0 = tile[r][cp] * inv_rms[r];
      float v1 = tile[r][cp + 1] * inv_rms[r];
      int C = col0 + cp;
      RowMeta rm = a.rows[R];
      if (C < a.q_cols + a.kv_cols) {
        int base = C < a.q_cols ? 0 : a.q_cols;
        int dp = (C - base) % a.dh;  // even: pair (dp, dp+1) = (j, j + dh/2) in the original order
        int j = dp >> 1;
        float2 cs = a.rope[(size_t)rm.pos * half + j];
        float o0 = v0 * cs.x - v1 * cs.y;
        float o1 = v1 * cs.x + v0 * cs.y;
        if (C < a.q_cols) {
          a.Q[(size_t)R * a.q_cols + C] = (_Float16)o0;
          a.Q[(size_t)R * a.q_cols + C + 1] = (_Float16)o1;
        } else {
          int g = (C - base) / a.dh;
          int page = a.pt[(size_t)rm.slot * a.pt_stride + (rm.pos >> 4)];
          _Float16* kp = a.kv + (size_t)page * a.page_stride + ((size_t)g * kPage + (rm.pos & 15)) * a.dh + dp;
          kp[0] = (_Float16)o0;
          kp[1] = (_Float16)o1;
        }
      } else {
        int cv = C - a.q_cols - a.kv_cols;
        int g = cv / a.dh, d = cv % a.dh;
        int page = a.pt[(size_t)rm.slot * a.pt_stride + (rm.pos >> 4)];
        _Float16* vp = a.kv + (size_t)page * a.page_stride + (size_t)a.Hkv * kPage * a.dh +
                       ((size_t)g * a.dh + d) * kPage + (rm.pos & 15);
        vp[0] = (_Float16)v0;
        vp[kPage] = (_Float16)v1;
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    // octets of 8 consecutive columns of one row: 16-byte fragment stores
    constexpr int OCT = COLS / 8;
    for (int base = 0; base < rows_here * OCT; base += 512) {
      int e = base + tid;
      bool ok = e < rows_here * OCT;
      int r = ok ? e / OCT : 0, o = ok ? e % OCT : 0;
      int R = row0 + r, C = col0 + o * 8;
      float sq = 0.f;
      if (ok) {
        float* xp = a.X + (size_t)R * a.D + C;
        float4 x0 = *(float4*)xp, x1 = *(float4*)(xp + 4);
        float xv[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
        uint16_t hi[8], lo[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          xv[i] += tile[r][o * 8 + i];
          sq += xv[i] * xv[i];
          split_bf16(xv[i] * a.gain_next[C + i], hi[i], lo[i]);
        }
        *(float4*)xp = float4{xv[0], xv[1], xv[2], xv[3]};
        *(float4*)(xp + 4) = float4{xv[4], xv[5], xv[6], xv[7]};
        size_t off = afrag_off(R, C, a.MTtot);
        uint4 h, l;
        h.x = hi[0] | ((uint32_t)hi[1] << 16); h.y = hi[2] | ((uint32_t)hi[3] << 16);
        h.z = hi[4] | ((uint32_t)hi[5] << 16); h.w = hi[6] | ((uint32_t)hi[7] << 16);
        l.x = lo[0] | ((uint32_t)lo[1] << 16); l.y = lo[2] | ((uint32_t)lo[3] << 16);
        l.z = lo[4] | ((uint32_t)lo[5] << 16); l.w = lo[6] | ((uint32_t)lo[7] << 16);
        *(uint4*)(a.Nhi + off) = h;
        *(uint4*)(a.Nlo + off) = l;
      }
      float other = __shfl_xor(sq, 1);
      if (ok && (o & 1) == 0) a.ss_out[(size_t)R * (a.D >> 4) + (C >> 4)] = sq + other;
    }
  } else if constexpr (EPI == EPI_SILU) {
    // strip pairs (2s = gate, 2s+1 = up) -> act columns (cb*2 + s)*16 + c
    constexpr int OCT = COLS / 16;  // act octets per row
    for (int e = tid; e < rows_here * OCT; e += 512) {
      int r = e / OCT, o = e % OCT;
      int s_ = o >> 1, c8 = (o & 1) * 8;
      int R = row0 + r;
      int F = (cb * (kNS / 2) + s_) * 16 + c8;
      uint16_t hi[8], lo[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float g = tile[r][s_ * 32 + c8 + i] * inv_rms[r];
        float u = tile[r][s_ * 32 + 16 + c8 + i] * inv_rms[r];
        float act = g / (1.f + __expf(-g)) * u;
        split_bf16(act, hi[i], lo[i]);
      }
      size_t off = afrag_off(R, F, a.MTtot);
      uint4 h, l;
      h.x = hi[0] | ((uint32_t)hi[1] << 16); h.y = hi[2] | ((uint32_t)hi[3] << 16);
      h.z = hi[4] | ((uint32_t)hi[5] << 16); h.w = hi[6] | ((uint32_t)hi[7] << 16);
      l.x = lo[0] | ((uint32_t)lo[1] << 16); l.y = lo[2] | ((uint32_t)lo[3] << 16);
      l.z = lo[4] | ((uint32_t)lo[5] << 16); l.w = lo[6] | ((uint32_t)lo[7] << 16);
      *(uint4*)(a.act_hi + off) = h;
      *(uint4*)(a.act_lo + off) = l;
    }
  } else {  // EPI_LM
    // one wave per row (loop): logits, then max / lowest argmax over COLS columns
    for (int r = wave; r < rows_here; r += 8) {
      int R = row0 + r;
      if (R >= a.M) break;
      float best = -INFINITY;
      int bidx = 0x7fffffff;
      for (int c = lane; c < COLS; c += 64) {
        float v = tile[r][c] * inv_rms[r];
        if (a.logits) a.logits[(size_t)R * a.vocab + col0 + c] = v;
        if (v > best) { best = v; bidx = col0 + c; }
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        float ov = __shfl_xor(best, o);
        int oi = __shfl_xor(bidx, o);
        if (ov > best || (ov == best && oi < bidx)) { best = ov; bidx = oi; }
      }
      if (lane == 0) {
        a.part_val[(size_t)R * a.n_part + blockIdx.x] = best;
        a.part_idx[(size_t)R * a.n_part + blockIdx.x] = bidx;
      }
    }
  }
}

// Inverse RMS of the workgroup's rows from per-16-column sums of squares,
// summed in a fixed order (rows past the last tile get 1/sqrt(eps)).
template <int MT>
__device__ __forceinline__ void gemm_inv_rms(const GemmArgs& a, float* inv_rms, int mt0, int mcount) {
  constexpr int ROWS = MT * 16;
  const int tid = threadIdx.x;
  if (a.ss != nullptr) {
    constexpr int TPR = (512 / ROWS) >= 32 ? 32 : (512 / ROWS) >= 16 ? 16 : (512 / ROWS) >= 8 ? 8 : 4;
    const int r = tid / TPR, j = tid % TPR;
    if (r < ROWS) {
      float sacc = 0.f;
      if (r < mcount * 16) {
        const float* srow = a.ss + (size_t)(mt0 * 16 + r) * a.ss_n;
        for (int i = j; i < a.ss_n; i += TPR) sacc += srow[i];
      }
#pragma unroll
      for (int o = TPR / 2; o > 0; o >>= 1) sacc += __shfl_xor(sacc, o);
      if (j == 0) inv_rms[r] = rsqrtf(sacc * a.inv_dim + a.eps);
    }
  } else if (tid < ROWS) {
    inv_rms[tid] = 1.f;
  }
}

template <int MT, int kNS, int EPI>
__global__ __launch_bounds__(512, gemm_occupancy(MT)) void gemm_skinny(GemmArgs a) {
  constexpr int U = gemm_depth(MT, kNS);
  constexpr int ROWS = MT * 16;
  constexpr int COLS = kNS * 16;

  __shared__ float red[4][kNS][MT][256];
  __shared__ float tile[ROWS][COLS + 1];
  __shared__ float inv_rms[ROWS];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int cb = blockIdx.x;
  const int mt0 = blockIdx.z * MT;
  const int mcount = min(MT, a.MTtot - mt0);

  // K range of this wave: the workgroup's share of K (split gridDim.y ways)
  // divided kKG ways
  const int kts = (a.KT + gridDim.y - 1) / gridDim.y;
  const int wk0 = blockIdx.y * kts, wk1 = min(a.KT, wk0 + kts);
  const int per = (wk1 - wk0 + kKG - 1) / kKG;
  const int k0 = wk0 + wave * per;
  const int k1 = min(wk1, k0 + per);

  f32x4 acc[MT][kNS];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int n = 0; n < kNS; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};

  // strip s, K step kt at ((s/4*KT + kt)*4 + s%4)*64: strip n of this
  // block at wp[n] + kt*256
  const u32x4* wp[kNS];
#pragma unroll
  for (int n = 0; n < kNS; ++n) {
    const int st = cb * kNS + n;
    wp[n] = (const u32x4*)a.W + ((size_t)(st >> 2) * a.KT * 4 + (st & 3)) * 64 + lane;
  }
  const size_t astride = (size_t)a.MTtot * 64;
  const u32x4* hp = (const u32x4*)a.Ahi + (size_t)mt0 * 64 + lane;
  const u32x4* lp = (const u32x4*)a.Alo + (size_t)mt0 * 64 + lane;

  u32x4 qb[U][kNS], qh[U][MT], ql[U][MT];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int kt = k0 + u;
    if (kt < k1) {
#pragma unroll
      for (int n = 0; n < kNS; ++n) qb[u][n] = __builtin_nontemporal_load(wp[n] + (size_t)kt * 256);
#pragma unroll
      for (int m = 0; m < MT; ++m)
        if (m < mcount) {
          qh[u][m] = hp[kt * astride + m * 64];
          ql[u][m] = lp[kt * astride + m * 64];
        }
    }
  }
  for (int kb = k0; kb < k1; kb += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kt = kb + u;
      if (kt < k1) {
#pragma unroll
        for (int m = 0; m < MT; ++m)
          if (m < mcount) {
#pragma unroll
            for (int n = 0; n < kNS; ++n) {
              acc[m][n] = mfma_bf16(qh[u][m], qb[u][n], acc[m][n]);
              acc[m][n] = mfma_bf16(ql[u][m], qb[u][n], acc[m][n]);
            }
          }
        const int nk = kt + U;
        if (nk < k1) {
#pragma unroll
          for (int n = 0; n < kNS; ++n) qb[u][n] = __builtin_nontemporal_load(wp[n] + (size_t)nk * 256);
#pragma unroll
          for (int m = 0; m < MT; ++m)
            if (m < mcount) {
              qh[u][m] = hp[nk * astride + m * 64];
              ql[u][m] = lp[nk * astride + m * 64];
            }
        }
      }
    }
  }

  // ---- reduce the 8 K ranges through LDS in two rounds (fixed order)
  if (wave >= 4) {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int n = 0; n < kNS; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[wave - 4][n][m][lane * 4 + i] = acc[m][n][i];
  }
  __syncthreads();
  if (wave < 4) {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int n = 0; n < kNS; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[wave][n][m][lane * 4 + i] += acc[m][n][i];
  }
  __syncthreads();
  for (int e = tid; e < kNS * MT * 256; e += 512) {
    const int n = e / (MT * 256), rem = e % (MT * 256);
    const int m = rem / 256, li = rem % 256;
    const int ln = li >> 2, i = li & 3;
    const float v = (red[0][n][m][li] + red[1][n][m][li]) + (red[2][n][m][li] + red[3][n][m][li]);
    tile[m * 16 + (ln >> 4) * 4 + i][n * 16 + (ln & 15)] = v;
  }
  if (gridDim.y > 1) {
    // K split across workgroups: publish the partial tile; gemm_finish sums
    // the splits in order and runs the epilogue.
    float* dst = a.part + ((size_t)(blockIdx.z * gridDim.x + cb) * gridDim.y + blockIdx.y) * ROWS * COLS;
    for (int e = tid; e < mcount * 16 * COLS; e += 512) dst[e] = tile[e / COLS][e % COLS];
    return;
  }
  gemm_inv_rms<MT>(a, inv_rms, mt0, mcount);
  __syncthreads();
  gemm_epilogue<MT, kNS, EPI>(a, tile, inv_rms, cb, mt0, mcount);
}

// Second pass of a K-split GEMM: one workgroup per (column block, row block)
// sums the splits' partial tiles in split order, then runs the epilogue.
template <int MT, int kNS, int EPI>
__global__ __launch_bounds__(512) void gemm_finish(GemmArgs a, int splits) {
  constexpr int ROWS = MT * 16;
  constexpr int COLS = kNS * 16;
  __shared__ float tile[ROWS][COLS + 1];
  __shared__ float inv_rms[ROWS];
  const int cb = blockIdx.x;
  const int mt0 = blockIdx.z * MT;
  const int mcount = min(MT, a.MTtot - mt0);
  const float* src = a.part + (size_t)(blockIdx.z * gridDim.x + cb) * splits * ROWS * COLS;
  for (int e = threadIdx.x; e < mcount * 16 * COLS; e += 512) {
    float v = 0.f;
    for (int q = 0; q < splits; ++q) v += src[(size_t)q * ROWS * COLS + e];
    tile[e / COLS][e % COLS] = v;
  }
  gemm_inv_rms<MT>(a, inv_rms, mt0, mcount);
  __syncthreads();
  gemm_epilogue<MT, kNS, EPI>(a, tile, inv_rms, cb, mt0, mcount);
}

template <int NS, int EPI>
static hipError_t launch_ns(const GemmArgs& a, int splits, int mblocks, int mt, hipStream_t s) {
  dim3 grid(a.NT / NS, splits, mblocks);
  dim3 fgrid(a.NT / NS, 1, mblocks);
  switch (mt) {
#define HVD_CASE(X)                                                                                   \
  case X:                                                                                             \
    hipLaunchKernelGGL((gemm_skinny<X, NS, EPI>), grid, dim3(512), 0, s, a);                          \
    if (splits > 1) hipLaunchKernelGGL((gemm_finish<X, NS, EPI>), fgrid, dim3(512), 0, s, a, splits); \
    break;
    HVD_CASE(1) HVD_CASE(2) HVD_CASE(3) HVD_CASE(4)
#undef HVD_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& a, int ns, int splits, int mblocks, int mt, hipStream_t s) {
  switch (ns) {
    case 1:
      if constexpr (EPI != EPI_SILU) return launch_ns<1, EPI>(a, splits, mblocks, mt, s);
      return hipErrorInvalidValue;
    case 2: return launch_ns<2, EPI>(a, splits, mblocks, mt, s);
    case 4: return launch_ns<4, EPI>(a, splits, mblocks, mt, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(int epi, const GemmArgs& a, int ns, int splits, int mblocks, int mt_block, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_epi<EPI_QKV>(a, ns, splits, mblocks, mt_block, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, ns, splits, mblocks, mt_block, s);
    case EPI_SILU: return launch_epi<EPI_SILU>(a, ns, splits, mblocks, mt_block, s);
    case EPI_LM: return launch_epi<EPI_LM>(a, ns, splits, mblocks, mt_block, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace hvd
