// Weight-streaming GEMMs of the verify forward (gfx950, MFMA 16x16x32 bf16).
//
// Y[m, n] = sum_k A[m, k] * W[n, k] with W the bf16 weight in torch Linear
// layout, pre-packed so that one 16x32 B-operand fragment is 1 KB contiguous
// (one 16-byte load per lane), and A the activation carried as a hi + lo pair
// of bf16 fragments (two MFMAs per tile: hi*W + lo*W keeps ~16 significant
// bits of the fp32 activation; the MFMA pipe is idle in this HBM-bound regime).
//
// Work split: a workgroup of 8 waves owns SW 16-column strips and all M rows;
// its waves split K into 8/SW contiguous ranges.  Each wave streams its weight
// fragments with a prefetch queue of depth U (weights and activations issued
// together so the in-order vmcnt waits never stall on a younger load), then
// the partial sums are reduced through LDS and the fused epilogue runs:
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

template <int MT>
struct Depth {
  static constexpr int U = MT == 1 ? 8 : (MT == 2 ? 6 : (MT <= 4 ? 3 : 2));
};

template <int EPI>
struct StripsPerBlock {
  static constexpr int SW = (EPI == EPI_SILU || EPI == EPI_LM) ? 2 : 1;
};

template <int MT, int EPI>
__global__ __launch_bounds__(512) void gemm_skinny(GemmArgs a) {
  constexpr int SW = StripsPerBlock<EPI>::SW;
  constexpr int KG = 8 / SW;
  constexpr int U = Depth<MT>::U;
  constexpr int ROWS = MT * 16;
  constexpr int COLS = SW * 16;

  __shared__ float red[8][MT][256];
  __shared__ float tile[ROWS][COLS + 1];
  __shared__ float inv_rms[ROWS];

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int sw = wave % SW, kg = wave / SW;
  const int strip = blockIdx.x * SW + sw;
  const int mt0 = blockIdx.z * MT;
  const int mcount = min(MT, a.MTtot - mt0);

  const int kper = (a.KT + KG - 1) / KG;
  const int k0 = kg * kper;
  const int k1 = min(a.KT, k0 + kper);

  f32x4 acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  const u32x4* wp = (const u32x4*)a.W + (size_t)strip * a.KT * 64 + lane;
  const size_t astride = (size_t)a.MTtot * 64;
  const u32x4* hp = (const u32x4*)a.Ahi + (size_t)mt0 * 64 + lane;
  const u32x4* lp = (const u32x4*)a.Alo + (size_t)mt0 * 64 + lane;

  u32x4 qb[U], qh[U][MT], ql[U][MT];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    int kt = k0 + u;
    if (kt < k1) {
      qb[u] = __builtin_nontemporal_load(wp + (size_t)kt * 64);
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
      int kt = kb + u;
      if (kt < k1) {
#pragma unroll
        for (int m = 0; m < MT; ++m)
          if (m < mcount) {
            acc[m] = mfma_bf16(qh[u][m], qb[u], acc[m]);
            acc[m] = mfma_bf16(ql[u][m], qb[u], acc[m]);
          }
        int nk = kt + U;
        if (nk < k1) {
          qb[u] = __builtin_nontemporal_load(wp + (size_t)nk * 64);
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

  // ---- reduce the K groups through LDS
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    red[wave][m][lane * 4 + 0] = acc[m][0];
    red[wave][m][lane * 4 + 1] = acc[m][1];
    red[wave][m][lane * 4 + 2] = acc[m][2];
    red[wave][m][lane * 4 + 3] = acc[m][3];
  }
  // inverse RMS of this block's rows, summed in a fixed order
  if (a.ss != nullptr) {
    // threads per row: largest power of two with ROWS * TPR <= 512
    constexpr int TPR = (512 / ROWS) >= 32 ? 32 : (512 / ROWS) >= 16 ? 16 : (512 / ROWS) >= 8 ? 8 : 4;
    int r = tid / TPR, j = tid % TPR;
    if (r < ROWS) {
      float s = 0.f;
      if (r < mcount * 16) {
        const float* srow = a.ss + (size_t)(mt0 * 16 + r) * a.ss_n;
        for (int i = j; i < a.ss_n; i += TPR) s += srow[i];
      }
#pragma unroll
      for (int o = TPR / 2; o > 0; o >>= 1) s += __shfl_xor(s, o);
      if (j == 0) inv_rms[r] = rsqrtf(s * a.inv_dim + a.eps);
    }
  }
  __syncthreads();
  for (int e = tid; e < SW * MT * 256; e += 512) {
    int s_ = e / (MT * 256), rem = e % (MT * 256);
    int m = rem / 256, li = rem % 256;
    int ln = li >> 2, i = li & 3;
    float v = 0.f;
#pragma unroll
    for (int g = 0; g < KG; ++g) v += red[g * SW + s_][m][li];
    int row = m * 16 + (ln >> 4) * 4 + i;
    int col = s_ * 16 + (ln & 15);
    tile[row][col] = v;
  }
  if (a.ss == nullptr && tid < ROWS) inv_rms[tid] = 1.f;
  __syncthreads();

  const int row0 = mt0 * 16;
  const int col0 = blockIdx.x * COLS;
  const int rows_here = mcount * 16;

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
    // strip pairs (2s = gate, 2s+1 = up) -> act columns (blockIdx.x*SW/2 + s)*16 + c
    constexpr int OCT = COLS / 16;  // act octets per row
    for (int e = tid; e < rows_here * OCT; e += 512) {
      int r = e / OCT, o = e % OCT;
      int s_ = o >> 1, c8 = (o & 1) * 8;
      int R = row0 + r;
      int F = (blockIdx.x * (SW / 2) + s_) * 16 + c8;
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

int gemm_strips_per_block(int epi) {
  switch (epi) {
    case EPI_QKV: return StripsPerBlock<EPI_QKV>::SW;
    case EPI_RESID: return StripsPerBlock<EPI_RESID>::SW;
    case EPI_SILU: return StripsPerBlock<EPI_SILU>::SW;
    default: return StripsPerBlock<EPI_LM>::SW;
  }
}

template <int EPI>
static hipError_t launch_epi(const GemmArgs& a, int mblocks, int mt, hipStream_t s) {
  dim3 grid(a.NT / StripsPerBlock<EPI>::SW, 1, mblocks);
  switch (mt) {
#define HVD_CASE(X) \
  case X: hipLaunchKernelGGL((gemm_skinny<X, EPI>), grid, dim3(512), 0, s, a); break;
    HVD_CASE(1) HVD_CASE(2) HVD_CASE(3) HVD_CASE(4) HVD_CASE(5) HVD_CASE(6) HVD_CASE(7) HVD_CASE(8)
#undef HVD_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(int epi, const GemmArgs& a, int mblocks, int mt_block, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_epi<EPI_QKV>(a, mblocks, mt_block, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, mblocks, mt_block, s);
    case EPI_SILU: return launch_epi<EPI_SILU>(a, mblocks, mt_block, s);
    case EPI_LM: return launch_epi<EPI_LM>(a, mblocks, mt_block, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace hvd
