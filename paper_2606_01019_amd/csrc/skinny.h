// Device code of the weight-streaming GEMM (gfx950, MFMA 16x16x32 f16),
// shared by the stand-alone kernel (gemm.hip) and the one-launch verify step
// (flow.hip): epilogue inputs and fused epilogues, and one output block of
// the skinny GEMM as a device function.  See gemm.hip for the design.
#pragma once

#include "common.h"
#include "kernels.h"

namespace hvd {

// Prefetch depth: K steps in flight per wave.  A stage holds NS weight and
// 2*MT activation fragments (4 VGPRs each); up to 2 row tiles the kernel is
// sized for 4 waves per SIMD (two 8-wave workgroups per CU), beyond that 2.
// (A one-workgroup-per-CU variant with a 16-stage queue measured no faster:
// these launches are not limited by weight bytes in flight.)
constexpr int gemm_occupancy(int MT) { return MT <= 2 ? 4 : 2; }
constexpr int gemm_depth(int MT, int NS, bool HL) {
  // 8 strips x 5 row tiles (gate/up, LM head at 65-80 rows): the accumulators leave
  // room for one stage; measured faster than 4 strips with three stages
  // (twice the workgroups, which then run in two rounds at one per CU)
  if (MT == 5 && NS == 8) return 1;
  const int budget = gemm_occupancy(MT) == 4 ? 80 : (HL ? 160 : 128);
  const int d = budget / (4 * (NS + (HL ? 2 : 1) * MT));
  return d < 1 ? 1 : (d > 8 ? 8 : d);
}

constexpr int kKG = 8;  // waves per workgroup, each a contiguous K range

// Epilogue inputs staged in LDS for the epilogue.
template <int MT, int NS, int EPI>
struct EpiPre {
  static constexpr int ROWS = MT * 16, COLS = NS * 16;
  float inv_rms[ROWS];
  float x[EPI == EPI_RESID ? ROWS : 1][EPI == EPI_RESID ? COLS : 1];
  float gain[EPI == EPI_RESID ? COLS : 1];
  float2 rope[EPI == EPI_QKV ? ROWS : 1][EPI == EPI_QKV ? COLS / 2 : 1];
  int page[EPI == EPI_QKV ? ROWS : 1];
  int pos[EPI == EPI_QKV ? ROWS : 1];  // the K/V position's offset in its page
};

// The same inputs on their way in, held in registers.  epi_issue() requests
// them before the first weight stage (memory returns in order, so a wait for
// them never waits for a weight stage), epi_commit() writes them to LDS
// while the first stages are still in flight.  Rotary factors depend on the
// row positions: epi_issue_rope() requests them after the first stages and
// epi_commit_rope() stores them after the main loop.  Every load reads a
// valid address (indices past the block are clamped and their values
// dropped), so no load sits under a branch.
template <int MT, int NS, int EPI>
struct EpiRegs {
  static constexpr int ROWS = MT * 16, COLS = NS * 16;
  static constexpr bool NORM = EPI != EPI_RESID;  // GEMM input is RMS-normalised
  static constexpr int TPR = ROWS <= 16 ? 32 : ROWS <= 32 ? 16 : ROWS <= 64 ? 8 : 4;  // threads per row of sums of squares
  static constexpr int SSQ = 4;  // float4 of sums of squares per thread held here (more: read late)
  static constexpr int XQ = EPI == EPI_RESID ? (ROWS * COLS / 4 + 511) / 512 : 1;
  static constexpr int RQ = EPI == EPI_QKV ? (ROWS * COLS / 2 + 511) / 512 : 1;
  // rotary factors ride along the main loop only for small row blocks
  // (larger ones are short of registers: they request them after it)
  static constexpr bool EARLY_ROPE = MT <= 2;
  float4 ss[NORM ? SSQ : 1];
  float4 x[XQ];
  float gain;
  RowMeta rm;
  int rpos[RQ];
  float2 rope[RQ];
};

template <int MT, int NS, int EPI>
__device__ __forceinline__ void epi_issue(const GemmArgs& a, EpiRegs<MT, NS, EPI>& e, int cb, int mt0, int mcount) {
  using E = EpiRegs<MT, NS, EPI>;
  constexpr int COLS = E::COLS;
  const int tid = threadIdx.x;
  const int row0 = mt0 * 16, col0 = cb * COLS, rows_here = mcount * 16;
  if constexpr (E::NORM) {
    const int r = tid / E::TPR, j = tid % E::TPR;
    const float4* srow = (const float4*)(a.ss + (size_t)(row0 + (r < rows_here ? r : 0)) * a.ss_n);
    const int nq = a.ss_n >> 2;
#pragma unroll
    for (int i = 0; i < E::SSQ; ++i) {
      const int q = j + i * E::TPR;
      e.ss[i] = srow[q < nq ? q : 0];
    }
  }
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int i = 0; i < E::XQ; ++i) {
      int el = tid + i * 512;
      if (el >= rows_here * (COLS / 4)) el = 0;
      const int r = el / (COLS / 4), c4 = (el % (COLS / 4)) * 4;
      e.x[i] = *(const float4*)(a.X + (size_t)(row0 + r) * a.D + col0 + c4);
    }
    e.gain = a.gain_next[col0 + (tid < COLS ? tid : 0)];
  }
  if constexpr (EPI == EPI_QKV) {
    const int last = a.M - 1;
    e.rm = a.rows[min(row0 + min(tid, rows_here - 1), last)];
#pragma unroll
    for (int i = 0; i < E::RQ; ++i) {
      int el = tid + i * 512;
      if (el >= rows_here * (COLS / 2)) el = 0;
      e.rpos[i] = a.rows[min(row0 + el / (COLS / 2), last)].pos;
    }
  }
}

// Marks the point from which the epilogue inputs may be used: the compiler
// sees new values here, so it can neither fold them into work placed
// before the weight stream nor wait for them earlier.
template <int MT, int NS, int EPI>
__device__ __forceinline__ void epi_settle(EpiRegs<MT, NS, EPI>& e) {
  using E = EpiRegs<MT, NS, EPI>;
  if constexpr (E::NORM) {
#pragma unroll
    for (int i = 0; i < E::SSQ; ++i) asm volatile("" : "+v"(e.ss[i].x), "+v"(e.ss[i].y), "+v"(e.ss[i].z), "+v"(e.ss[i].w));
  }
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int i = 0; i < E::XQ; ++i) asm volatile("" : "+v"(e.x[i].x), "+v"(e.x[i].y), "+v"(e.x[i].z), "+v"(e.x[i].w));
    asm volatile("" : "+v"(e.gain));
  }
  if constexpr (EPI == EPI_QKV) {
    asm volatile("" : "+v"(e.rm.pos), "+v"(e.rm.kvs));
#pragma unroll
    for (int i = 0; i < E::RQ; ++i) asm volatile("" : "+v"(e.rpos[i]));
  }
}

template <int MT, int NS, int EPI>
__device__ __forceinline__ void epi_issue_rope(const GemmArgs& a, EpiRegs<MT, NS, EPI>& e, int cb) {
  if constexpr (EPI == EPI_QKV) {
    using E = EpiRegs<MT, NS, EPI>;
    constexpr int COLS = E::COLS;
    const int col0 = cb * COLS;
    const bool rotated = col0 < a.q_cols + a.kv_cols;  // block holds q or k columns
    const int half = a.dh >> 1;
#pragma unroll
    for (int i = 0; i < E::RQ; ++i) {
      const int cp = (threadIdx.x + i * 512) % (COLS / 2);
      const int C = col0 + 2 * cp;
      const int base = C < a.q_cols ? 0 : a.q_cols;
      const int j = rotated ? ((C - base) % a.dh) >> 1 : 0;
      e.rope[i] = a.rope[(size_t)e.rpos[i] * half + j];
    }
  }
}

template <int MT, int NS, int EPI>
__device__ __forceinline__ void epi_commit(const GemmArgs& a, const EpiRegs<MT, NS, EPI>& e,
                                           EpiPre<MT, NS, EPI>& p, int cb, int mt0, int mcount) {
  using E = EpiRegs<MT, NS, EPI>;
  constexpr int ROWS = E::ROWS, COLS = E::COLS;
  const int tid = threadIdx.x;
  const int row0 = mt0 * 16, rows_here = mcount * 16;
  if constexpr (E::NORM) {
    // inverse RMS from per-16-column sums of squares, summed in a fixed order
    const int r = tid / E::TPR, j = tid % E::TPR;
    const int nq = a.ss_n >> 2;
    float sacc = 0.f;
#pragma unroll
    for (int i = 0; i < E::SSQ; ++i) {
      const float4 v = e.ss[i];
      if (j + i * E::TPR < nq) sacc += (v.x + v.y) + (v.z + v.w);
    }
    if (nq > E::SSQ * E::TPR) {  // wide rows: the rest is read here
      const float4* srow = (const float4*)(a.ss + (size_t)(row0 + (r < rows_here ? r : 0)) * a.ss_n);
      for (int q = j + E::SSQ * E::TPR; q < nq; q += E::TPR) {
        const float4 v = srow[q];
        sacc += (v.x + v.y) + (v.z + v.w);
      }
    }
#pragma unroll
    for (int o = E::TPR / 2; o > 0; o >>= 1) sacc += __shfl_xor(sacc, o);
    if (j == 0 && r < ROWS) p.inv_rms[r] = r < rows_here ? rsqrtf(sacc * a.inv_dim + a.eps) : 1.f;
  } else if (tid < ROWS) {
    p.inv_rms[tid] = 1.f;
  }
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int i = 0; i < E::XQ; ++i) {
      const int el = tid + i * 512;
      if (el < rows_here * (COLS / 4)) {
        const int r = el / (COLS / 4), c4 = (el % (COLS / 4)) * 4;
        p.x[r][c4] = e.x[i].x;
        p.x[r][c4 + 1] = e.x[i].y;
        p.x[r][c4 + 2] = e.x[i].z;
        p.x[r][c4 + 3] = e.x[i].w;
      }
    }
    if (tid < COLS) p.gain[tid] = e.gain;
  }
  if constexpr (EPI == EPI_QKV) {
    if (tid < rows_here) {
      const bool ok = row0 + tid < a.M;
      p.pos[tid] = ok ? (e.rm.kvs & (kPage - 1)) : 0;
      p.page[tid] = ok ? e.rm.kvs / kPage : 0;
    }
  }
}

template <int MT, int NS, int EPI>
__device__ __forceinline__ void epi_commit_rope(const GemmArgs& a, const EpiRegs<MT, NS, EPI>& e,
                                                EpiPre<MT, NS, EPI>& p, int mt0, int mcount) {
  if constexpr (EPI == EPI_QKV) {
    using E = EpiRegs<MT, NS, EPI>;
    constexpr int COLS = E::COLS;
    const int rows_here = mcount * 16;
#pragma unroll
    for (int i = 0; i < E::RQ; ++i) {
      const int el = threadIdx.x + i * 512;
      if (el < rows_here * (COLS / 2)) {
        const int r = el / (COLS / 2), cp = el % (COLS / 2);
        p.rope[r][cp] = mt0 * 16 + r < a.M ? e.rope[i] : float2{1.f, 0.f};
      }
    }
  }
}

__device__ __forceinline__ uint4 pack8(const uint16_t* v) {
  return uint4{v[0] | ((uint32_t)v[1] << 16), v[2] | ((uint32_t)v[3] << 16), v[4] | ((uint32_t)v[5] << 16),
               v[6] | ((uint32_t)v[7] << 16)};
}

// Fused epilogue on the reduced [rows][cols] tile of one workgroup.
template <int MT, int NS, int EPI, bool COH = false>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& a, float (*tile)[NS * 16 + 1],
                                              const EpiPre<MT, NS, EPI>& p, int cb, int mt0, int mcount) {
  constexpr int COLS = NS * 16;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int rows_here = mcount * 16;
  const int row0 = mt0 * 16;
  const int col0 = cb * COLS;

  if constexpr (EPI == EPI_QKV) {
    for (int e = tid; e < rows_here * (COLS / 2); e += 512) {
      const int r = e / (COLS / 2), cp = e % (COLS / 2);
      const int R = row0 + r;
      if (R >= a.M) continue;
      const float v0 = tile[r][2 * cp] * p.inv_rms[r];
      const float v1 = tile[r][2 * cp + 1] * p.inv_rms[r];
      const int C = col0 + 2 * cp;
      if (C < a.q_cols + a.kv_cols) {
        const int base = C < a.q_cols ? 0 : a.q_cols;
        const int dp = (C - base) % a.dh;  // even: pair (dp, dp+1) = (j, j + dh/2) in the original order
        const float2 cs = p.rope[r][cp];
        const float o0 = v0 * cs.x - v1 * cs.y;
        const float o1 = v1 * cs.x + v0 * cs.y;
        if (C < a.q_cols) {
          if constexpr (COH) {
            st_u32_dev((uint32_t*)(a.Q + (size_t)R * a.q_cols + C), pack_h2(o0, o1));
          } else {
            a.Q[(size_t)R * a.q_cols + C] = (_Float16)o0;
            a.Q[(size_t)R * a.q_cols + C + 1] = (_Float16)o1;
          }
        } else {
          const int g = (C - base) / a.dh;
          _Float16* kp =
              a.kv + (size_t)p.page[r] * a.page_stride + ((size_t)g * kPage + (p.pos[r] & 15)) * a.dh + dp;
          if constexpr (COH) {
            st_u32_dev((uint32_t*)kp, pack_h2(o0, o1));
          } else {
            kp[0] = (_Float16)o0;
            kp[1] = (_Float16)o1;
          }
        }
      } else {
        const int cv = C - a.q_cols - a.kv_cols;
        const int g = cv / a.dh, d = cv % a.dh;
        _Float16* vp = a.kv + (size_t)p.page[r] * a.page_stride + (size_t)a.Hkv * kPage * a.dh +
                       ((size_t)g * a.dh + d) * kPage + (p.pos[r] & 15);
        if constexpr (COH) {
          st_u16_dev((uint16_t*)vp, f2h(v0));
          st_u16_dev((uint16_t*)(vp + kPage), f2h(v1));
        } else {
          vp[0] = (_Float16)v0;
          vp[kPage] = (_Float16)v1;
        }
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    // octets of 8 consecutive columns of one row: 16-byte fragment stores
    constexpr int OCT = COLS / 8;
    for (int base = 0; base < rows_here * OCT; base += 512) {
      const int e = base + tid;
      const bool ok = e < rows_here * OCT;
      const int r = ok ? e / OCT : 0, o = ok ? e % OCT : 0;
      const int R = row0 + r, C = col0 + o * 8;
      float sq = 0.f;
      if (ok) {
        float xv[8];
        uint16_t hi[8], lo[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          xv[i] = p.x[r][o * 8 + i] + tile[r][o * 8 + i];
          sq += xv[i] * xv[i];
          split_f16(xv[i] * p.gain[o * 8 + i], hi[i], lo[i]);
        }
        float* const xdst = a.X_out ? a.X_out : a.X;
        float* xp = xdst + (size_t)R * a.D + C;
        const size_t off = afrag_off(R, C, a.MTtot);
        if constexpr (COH) {
          st_f4_dev(xdst, (R * a.D + C) * 4, float4{xv[0], xv[1], xv[2], xv[3]});
          st_f4_dev(xdst, (R * a.D + C + 4) * 4, float4{xv[4], xv[5], xv[6], xv[7]});
          st_16_dev(a.Nhi, (uint32_t)(off * 2), pack8(hi));
          st_16_dev(a.Nlo, (uint32_t)(off * 2), pack8(lo));
        } else {
          *(float4*)xp = float4{xv[0], xv[1], xv[2], xv[3]};
          *(float4*)(xp + 4) = float4{xv[4], xv[5], xv[6], xv[7]};
          *(uint4*)(a.Nhi + off) = pack8(hi);
          *(uint4*)(a.Nlo + off) = pack8(lo);
        }
      }
      const float other = __shfl_xor(sq, 1);
      if (ok && (o & 1) == 0) {
        float* sp = a.ss_out + (size_t)R * (a.D >> 4) + (C >> 4);
        if constexpr (COH) store_dev(sp, sq + other);
        else *sp = sq + other;
      }
    }
  } else if constexpr (EPI == EPI_SILU) {
    // strip pairs (2s = gate, 2s+1 = up) -> act columns (cb*NS/2 + s)*16 + c
    constexpr int OCT = COLS / 16;  // act octets per row
    for (int e = tid; e < rows_here * OCT; e += 512) {
      const int r = e / OCT, o = e % OCT;
      const int s_ = o >> 1, c8 = (o & 1) * 8;
      const int R = row0 + r;
      const int F = (cb * (NS / 2) + s_) * 16 + c8;
      uint16_t hi[8], lo[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float g = tile[r][s_ * 32 + c8 + i] * p.inv_rms[r];
        const float u = tile[r][s_ * 32 + 16 + c8 + i] * p.inv_rms[r];
        const float act = g / (1.f + __expf(-g)) * u;
        split_f16(act, hi[i], lo[i]);
      }
      const size_t off = afrag_off(R, F, a.MTtot);
      if constexpr (COH) {
        st_16_dev(a.act_hi, (uint32_t)(off * 2), pack8(hi));
        st_16_dev(a.act_lo, (uint32_t)(off * 2), pack8(lo));
      } else {
        *(uint4*)(a.act_hi + off) = pack8(hi);
        *(uint4*)(a.act_lo + off) = pack8(lo);
      }
    }
  } else {  // EPI_LM
    // one wave per row (loop): logits, then max / lowest argmax over COLS columns
    for (int r = wave; r < rows_here; r += 8) {
      const int R = row0 + r;
      if (R >= a.M) break;
      float best = -INFINITY;
      int bidx = 0x7fffffff;
      for (int c = lane; c < COLS; c += 64) {
        const float v = tile[r][c] * p.inv_rms[r];
        if (a.logits) a.logits[(size_t)R * a.vocab + col0 + c] = v;
        if (v > best) {
          best = v;
          bidx = col0 + c;
        }
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(best, o);
        const int oi = __shfl_xor(bidx, o);
        if (ov > best || (ov == best && oi < bidx)) {
          best = ov;
          bidx = oi;
        }
      }
      if (lane == 0) {
        a.part_val[(size_t)R * a.n_part + cb] = best;
        a.part_idx[(size_t)R * a.n_part + cb] = bidx;
      }
    }
  }
}

// Workgroup -> (column block, K split, row block).  With several row
// blocks, those of one (column block, split) get workgroup ids 8 apart: the
// same XCD under round-robin dispatch, started at nearly the same time, so
// the weights are read from HBM once and from that XCD's L2 after.
struct SkinnyCoord {
  int cb, split, mb;
};
__device__ __forceinline__ SkinnyCoord skinny_coord() {
  const int gx = gridDim.x, gy = gridDim.y, mbs = gridDim.z;
  if (mbs == 1) return {(int)blockIdx.x, (int)blockIdx.y, 0};
  const int lin = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const int units = gx * gy, u8 = units - units % 8;
  int unit, mb;
  if (lin < u8 * mbs) {
    const int r = lin / 8;
    mb = r % mbs;
    unit = (r / mbs) * 8 + lin % 8;
  } else {  // the last units % 8 units: row blocks adjacent
    const int rem = lin - u8 * mbs;
    unit = u8 + rem / mbs;
    mb = rem % mbs;
  }
  return {unit % gx, unit / gx, mb};
}

// HL: activation as the fp16 hi + lo pair (two MFMAs per tile), or the hi
// part alone (one MFMA; used for the MLP GEMMs of verify batches over 32 rows)
// LDS of one skinny tile: the cross-wave reduction buffer (taking NH passes
// over the strips: two for 8 strips x 4 row tiles, whose full buffer would
// not fit), the reduced tile and the epilogue inputs.
template <int MT, int NS, int EPI>
struct SkinnySmem {
  static constexpr int NH = (NS == 8 && MT >= 4) ? 2 : 1;
  float red[4][NS / NH][MT][256];
  float tile[MT * 16][NS * 16 + 1];
  EpiPre<MT, NS, EPI> pre;
  int last_split;
};

// One output block (column block co.cb, K split co.split of nsplit, row block
// co.mb) of the weight-streaming GEMM, computed by one 512-thread workgroup.
// COH: the work runs inside a larger kernel whose other workgroups consume
// its outputs: they are written with device-scope (write-through) stores,
// and the first weight stages are requested before hk.wait().  Inputs are
// read with ordinary (L2-cached) loads, so every input buffer must be one
// that this launch writes once and reads only after it is complete.
// HL: activation as the fp16 hi + lo pair (two MFMAs per tile), or the hi
// part alone (one MFMA; used for the MLP GEMMs of verify batches over 32 rows)
template <int MT, int NS, int EPI, bool HL, bool COH, class Hooks>
__device__ __forceinline__ void skinny_tile(const GemmArgs& a, const SkinnyCoord co, const int nsplit, const int n_cb,
                                            SkinnySmem<MT, NS, EPI>& sm, Hooks& hk) {
  constexpr int U = gemm_depth(MT, NS, HL);
  constexpr int ROWS = MT * 16;
  constexpr int COLS = NS * 16;
  constexpr int NH = SkinnySmem<MT, NS, EPI>::NH;
  constexpr int NSH = NS / NH;
  auto& red = sm.red;
  auto& tile = sm.tile;
  auto& pre = sm.pre;

  const int tid = threadIdx.x;
  // wave index made wave-uniform so K ranges and fragment bases stay in
  // scalar registers (one VGPR per lane of addressing, no register reuse
  // that would force the prefetch queue to drain)
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int cb = co.cb;
  const int mt0 = co.mb * MT;
  const int mcount = min(MT, a.MTtot - mt0);
  const bool split = nsplit > 1;

  // K steps of this wave: the workgroup's share of K (split nsplit ways),
  // dealt round-robin to its kKG waves, so at any moment the workgroup reads
  // one contiguous window of weights (kKG adjacent K steps) rather than kKG
  // distant streams
  const int kts = (a.KT + nsplit - 1) / nsplit;
  const int wk0 = co.split * kts, wk1 = min(a.KT, wk0 + kts);
  const int kb = wk0 + wave;
  const int nsteps = kb < wk1 ? (wk1 - kb + kKG - 1) / kKG : 0;  // wave-uniform

  f32x4 acc[MT][NS];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int n = 0; n < NS; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};

  // strip n of this block, K step kt, at wp[n] + kt*wk
  const u32x4* wp[NS];
#pragma unroll
  for (int n = 0; n < NS; ++n) {
    const int st = cb * NS + n;
    wp[n] = (const u32x4*)a.W + (size_t)(st >> 2) * a.wg + (size_t)(st & 3) * 64;
  }
  const size_t astride = (size_t)a.MTtot * 64;
  const u32x4* hp = (const u32x4*)a.Ahi + (size_t)mt0 * 64;
  const u32x4* lp = (const u32x4*)a.Alo + (size_t)mt0 * 64;

  // Stage u of the prefetch queue holds the fragments of one K step.  Row
  // tiles past this block's last are computed, then dropped (no per-tile
  // branches in the loop); their lanes count as rows past a.M below.
  u32x4 qb[U][NS], qh[U][MT], ql[U][HL ? MT : 1];
  auto load_w = [&](int u, int j) __attribute__((always_inline)) {
    const int kt = kb + j * kKG;
#pragma unroll
    for (int n = 0; n < NS; ++n) qb[u][n] = __builtin_nontemporal_load(wp[n] + (size_t)kt * a.wk + lane);
  };
  // A lane holds one row's 8 halves (row = lane % 16 of its tile); the
  // outputs of rows at or past a.M are dropped, so those lanes need no data.
  // Blocks of one or two row tiles: those lanes skip the load and keep what
  // their register held (zero at first), which also saves the data return.
  // Larger blocks (where the branches measured slower): those lanes read
  // their 16-lane group's last live row, the cache lines the live lanes
  // fetch anyway.  Either way a tile with at most 8 live rows reads one of
  // its group's two 128-byte lines.
  constexpr bool MASKED = MT <= 2;
  bool lok[MT];
  int alane[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int live = min(16, max(1, a.M - (mt0 + m) * 16));
    lok[m] = (mt0 + m) * 16 + (lane & 15) < a.M;
    alane[m] = m * 64 + (MASKED ? lane : min(lane & 15, live - 1) + (lane & 48));
  }
  if constexpr (MASKED) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        qh[u][m] = u32x4{0u, 0u, 0u, 0u};
        if constexpr (HL) ql[u][m] = u32x4{0u, 0u, 0u, 0u};
      }
  }
  auto load_a = [&](int u, int j) __attribute__((always_inline)) {
    const int kt = kb + j * kKG;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      if (!MASKED || lok[m]) {
        qh[u][m] = hp[kt * astride + alane[m]];
        if constexpr (HL) ql[u][m] = lp[kt * astride + alane[m]];
      }
    }
  };
  auto load = [&](int u, int j) __attribute__((always_inline)) {
    load_w(u, j);
    load_a(u, j);
  };
  auto consume = [&](int u) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int n = 0; n < NS; ++n) {
        acc[m][n] = mfma_f16(qh[u][m], qb[u][n], acc[m][n]);
        if constexpr (HL) acc[m][n] = mfma_f16(ql[u][m], qb[u][n], acc[m][n]);
      }
  };

  EpiRegs<MT, NS, EPI> er;
  if (nsteps >= U) {
    // prologue: inside a larger kernel, the weights of the first U steps go
    // out before the wait for the inputs; otherwise the epilogue inputs go
    // first, then weights and activations step by step
    if constexpr (COH) {
#pragma unroll
      for (int u = 0; u < U; ++u) load_w(u, u);
      hk.wait();
      epi_issue<MT, NS, EPI>(a, er, cb, mt0, mcount);
#pragma unroll
      for (int u = 0; u < U; ++u) load_a(u, u);
    } else {
      epi_issue<MT, NS, EPI>(a, er, cb, mt0, mcount);  // (a split block's copy goes unused)
#pragma unroll
      for (int u = 0; u < U; ++u) load(u, u);
    }
    epi_settle<MT, NS, EPI>(er);
    if constexpr (EpiRegs<MT, NS, EPI>::EARLY_ROPE) epi_issue_rope<MT, NS, EPI>(a, er, cb);
    epi_commit<MT, NS, EPI>(a, er, pre, cb, mt0, mcount);
    int j = 0;
    // steady state: every stage is consumed and refilled, no branches
    for (; j + 2 * U <= nsteps; j += U) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        consume(u);
        load(u, j + u + U);
      }
    }
    // tail: the U stages in flight hold steps j..j+U-1; fewer than U remain after them
    const int rem = nsteps - (j + U);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      consume(u);
      if (u < rem) load(u, j + U + u);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (u < rem) consume(u);
  } else {
    // fewer steps than stages: all of them in flight at once
    if constexpr (COH) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (u < nsteps) load_w(u, u);
      hk.wait();
      epi_issue<MT, NS, EPI>(a, er, cb, mt0, mcount);
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (u < nsteps) load_a(u, u);
    } else {
      epi_issue<MT, NS, EPI>(a, er, cb, mt0, mcount);
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (u < nsteps) load(u, u);
    }
    epi_settle<MT, NS, EPI>(er);
    if constexpr (EpiRegs<MT, NS, EPI>::EARLY_ROPE) epi_issue_rope<MT, NS, EPI>(a, er, cb);
    epi_commit<MT, NS, EPI>(a, er, pre, cb, mt0, mcount);
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (u < nsteps) consume(u);
  }
  if constexpr (!EpiRegs<MT, NS, EPI>::EARLY_ROPE) epi_issue_rope<MT, NS, EPI>(a, er, cb);
  epi_commit_rope<MT, NS, EPI>(a, er, pre, mt0, mcount);

  // ---- reduce the 8 K ranges through LDS in two rounds (fixed order), in
  // NH passes over the strips
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    if (h) __syncthreads();  // the previous pass has read red
    if (wave >= 4) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int n = 0; n < NSH; ++n)
#pragma unroll
          for (int i = 0; i < 4; ++i) red[wave - 4][n][m][lane * 4 + i] = acc[m][h * NSH + n][i];
    }
    __syncthreads();
    if (wave < 4) {
#pragma unroll
      for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int n = 0; n < NSH; ++n)
#pragma unroll
          for (int i = 0; i < 4; ++i) red[wave][n][m][lane * 4 + i] += acc[m][h * NSH + n][i];
    }
    __syncthreads();
    for (int e = tid; e < NSH * MT * 256; e += 512) {
      const int n = e / (MT * 256), rem = e % (MT * 256);
      const int m = rem / 256, li = rem % 256;
      const int ln = li >> 2, i = li & 3;
      const float v = (red[0][n][m][li] + red[1][n][m][li]) + (red[2][n][m][li] + red[3][n][m][li]);
      tile[m * 16 + (ln >> 4) * 4 + i][(h * NSH + n) * 16 + (ln & 15)] = v;
    }
  }
  __syncthreads();

  if (split) {
    // K split across workgroups: publish this split's partial tile with
    // device-scope (write-through) stores, then count arrivals; the last
    // split of the (row block, column block) to arrive sums every split in
    // split order (the same order whichever arrives last, so results are
    // deterministic) and runs the epilogue.  No second kernel.
    constexpr int EPT = (ROWS * COLS + 511) / 512;  // tile entries per thread
    constexpr int SB = 8;                           // splits per batch of loads
    int& last_split = sm.last_split;
    const int unit = co.mb * n_cb + cb;
    const int n_el = mcount * 16 * COLS;
    float* part = a.part + (size_t)unit * nsplit * ROWS * COLS;
    float* dst = part + (size_t)co.split * ROWS * COLS;
    for (int e = tid; e < n_el; e += 512) store_dev(dst + e, tile[e / COLS][e % COLS]);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this thread's stores are done
    __syncthreads();
    if (tid == 0) last_split = atomicAdd(a.cnt + unit, 1u) == (uint32_t)nsplit - 1u;
    __syncthreads();
    if (!last_split) return;
    float v[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) v[i] = 0.f;
    for (int q0 = 0; q0 < nsplit; q0 += SB) {
      float t[EPT][SB];
#pragma unroll
      for (int i = 0; i < EPT; ++i)
#pragma unroll
        for (int q = 0; q < SB; ++q) {
          const int el = tid + i * 512;
          const int qq = q0 + q < nsplit ? q0 + q : 0;
          t[i][q] = load_dev(part + (size_t)qq * ROWS * COLS + (el < n_el ? el : 0));
        }
#pragma unroll
      for (int i = 0; i < EPT; ++i)
#pragma unroll
        for (int q = 0; q < SB; ++q)
          if (q0 + q < nsplit) v[i] += t[i][q];
    }
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      const int el = tid + i * 512;
      if (el < n_el) tile[el / COLS][el % COLS] = v[i];
    }
    if (tid == 0) store_dev_u32(a.cnt + unit, 0u);  // ready for the next launch
    __syncthreads();
  }
  gemm_epilogue<MT, NS, EPI, COH>(a, tile, pre, cb, mt0, mcount);
  hk.done();
}


}  // namespace hvd
