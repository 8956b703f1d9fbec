// Large-batch GEMMs of the verify forward (gfx950, MFMA 32x32x16 f16): many
// verify rows at once (batched sequences, long drafts) and prefill chunks,
// where the weight-streaming kernel would re-read the weights per 64 rows.
//
// Y[m, n] = sum_k A[m, k] W[n, k] over the same packed operands as the
// streaming kernel: 1 KB fragments of 16 rows (or weight columns) x 32 K.
// A workgroup of WY x WX waves owns a BM x BN tile (BM = 32 WM WY, BN =
// 32 WN WX) and walks its K range in 32-wide steps: every step's A and W
// fragments are copied from global memory straight into a ring of ST LDS
// slots (global_load_lds: no registers, ST - 1 steps in flight ahead of the
// MFMAs), and each wave multiplies its 32WM x 32WN sub-tile with WM x WN
// MFMA tiles of 32 x 32.
// The 256 x 256 tile (8 waves) needs about 32 bytes of operand per clock and
// CU at full MFMA rate; 128-row tiles (4 waves) serve smaller batches.
// HI_LO chooses the activation precision: the fp16 hi + lo pair (two MFMAs
// per tile, ~22 bits) or the hi part alone (one MFMA, 11 bits).
//
// Workgroups are numbered so that each XCD receives a contiguous run of
// tiles with the row blocks of a column block adjacent: the weight tile is
// fetched from HBM once into that XCD's L2 and re-read from there by the
// other row blocks.  A K split (gridDim covers S splits) writes fp32 partial
// tiles; the last split of a tile to arrive sums them in split order and runs
// the epilogue.
//
// The epilogue works on the accumulator registers: MFMA 32x32 output element
// (row 8*(r/4) + 4*(lane/32) + r%4, column lane%32) of register r.  Partner
// columns (rotary pairs, gate/up strips) are exchanged with lane shuffles.
#include "common.h"
#include "kernels.h"

#include <type_traits>

namespace hvd {

typedef float f32x16 __attribute__((ext_vector_type(16)));

typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt on the vector-memory counter only (gfx9 encoding: vmcnt in bits
// 3:0 and 15:14, expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// Workgroup barrier without the memory fence of __syncthreads (whose release
// would wait for every LDS copy in flight); the empty asm statements keep the
// compiler from moving LDS accesses across it.
__device__ __forceinline__ void block_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ f32x16 mfma32_f16(const u32x4& a, const u32x4& b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                0, 0);
}

// Workgroup -> (split, column block, row block): XCD x (= id % 8 under the
// round-robin dispatch) gets logical tiles [start_x, start_x + n_x), row
// blocks fastest.
struct TileCoord {
  int split, cb, rb;
};
__device__ __forceinline__ TileCoord tile_coord(int id, int total, int RB, int CB) {
  const int x = id & 7, local = id >> 3;
  const int q = total >> 3, rem = total & 7;
  const int logical = x * q + min(x, rem) + local;
  TileCoord t;
  t.rb = logical % RB;
  t.cb = (logical / RB) % CB;
  t.split = logical / (RB * CB);
  return t;
}

template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// Epilogue on the accumulators of one wave.  rows/cols are global indices of
// the wave's sub-tile origin.  inv_rms: per-row inverse RMS (NORM GEMMs).
template <int WY, int WX, int WM, int WN, int EPI>
__device__ __forceinline__ void tiled_epilogue(const GemmArgs& a, const f32x16 (&acc)[WM][WN], int row_w, int col_w,
                                               const float* inv_rms, float2* lm_best, int* lm_idx, int cb) {
  constexpr int BM = 32 * WM * WY;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wy = wave / WX, wx = wave % WX;
  const int lhi = lane >> 5, lc = lane & 31;
  // Residual inputs are read one group of 4 rows ahead of the stores, and the
  // gains once: a load issued after a store waits for that store before its
  // value can be used.
  constexpr bool XR = EPI == EPI_RESID;
  float xq[2][XR ? 4 : 1][XR ? WN : 1];
  auto load_x = [&](int g, float (&dst)[XR ? 4 : 1][XR ? WN : 1]) {
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int R = row_w + 32 * (g >> 2) + 8 * (g & 3) + 4 * lhi + rr;
#pragma unroll
      for (int j = 0; j < WN; ++j) dst[rr][j] = R < a.M ? a.X[(size_t)R * a.D + col_w + 32 * j + lc] : 0.f;
    }
  };
  float gn[XR ? WN : 1];  // next layer's norm gain at this lane's columns
  if constexpr (XR) {
#pragma unroll
    for (int j = 0; j < WN; ++j) gn[j] = a.gain_next[col_w + 32 * j + lc];
    load_x(0, xq[0]);
  }
  // Per-row inputs (inverse RMS; position and KV slot for QKV): lane lc reads
  // row lc of each 32-row tile once, and the rows are handed out by shuffles.
  constexpr bool RQ = EPI == EPI_QKV;
  float irl[WM];
  int posl[RQ ? WM : 1], kvsl[RQ ? WM : 1];
#pragma unroll
  for (int i = 0; i < WM; ++i) {
    const int R = row_w + 32 * i + lc;
    const bool ok = R < a.M;
    irl[i] = (EPI != EPI_RESID && ok) ? inv_rms[R] : 1.f;
    if constexpr (RQ) {
      posl[i] = ok ? a.rows[R].pos : 0;
      kvsl[i] = ok ? a.rows[R].kvs : 0;
    }
  }
  // QKV: rotary (cos, sin) pairs one group of 4 rows ahead of the stores.
  // Wave tiles of 128 columns read them at the store instead: two groups of
  // pairs would take 64 more registers beside 128 or 256 accumulators.
  constexpr bool PCS = RQ && WN <= 2;
  float2 csq[2][PCS ? 4 : 1][PCS ? WN : 1];
  auto load_cs = [&](int g, float2 (&dst)[PCS ? 4 : 1][PCS ? WN : 1]) {
    const int half = a.dh >> 1;
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      const int t = 8 * (g & 3) + 4 * lhi + rr;
      const int pos = __shfl(posl[g >> 2], t);
      const bool rok = row_w + 32 * (g >> 2) + t < a.M;
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        const int C = col_w + 32 * j + lc;
        dst[rr][j] = float2{1.f, 0.f};
        if (rok && C < a.q_cols + a.kv_cols) {
          const int base = C < a.q_cols ? 0 : a.q_cols;
          dst[rr][j] = a.rope[(size_t)pos * half + (((C - base) % a.dh) >> 1)];
        }
      }
    }
  };
  if constexpr (PCS) load_cs(0, csq[0]);
  // the row-tile index is a compile-time constant, so the accumulators are
  // never indexed at run time (a rolled loop would move them to scratch)
  static_for<0, WM>([&](auto ic) {
    constexpr int i = decltype(ic)::value;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int R = row_w + 32 * i + 8 * (r >> 2) + 4 * lhi + (r & 3);
      const bool rok = R < a.M;
      const int t = 8 * (r >> 2) + 4 * lhi + (r & 3);  // row within the 32-row tile
      const int g = 4 * i + (r >> 2);
      if constexpr (XR) {
        if ((r & 3) == 0 && g + 1 < 4 * WM) load_x(g + 1, xq[(g + 1) & 1]);
      }
      if constexpr (PCS) {
        if ((r & 3) == 0 && g + 1 < 4 * WM) load_cs(g + 1, csq[(g + 1) & 1]);
      }
      const float ir = __shfl(irl[i], t);
      if constexpr (EPI == EPI_QKV) {
        // shuffles run on every lane: a shuffle under the branches below would
        // read lanes that are switched off
        const int kvs = __shfl(kvsl[i], t);
        const int pos = PCS ? 0 : __shfl(posl[i], t);
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          const int C = col_w + 32 * j + lc;
          const float v = acc[i][j][r] * ir;
          const float pv = __shfl_xor(v, 1);  // rotary partner (adjacent column)
          if (!rok) continue;
          if (C < a.q_cols + a.kv_cols) {
            if ((C & 1) == 0) {
              const int base = C < a.q_cols ? 0 : a.q_cols;
              const int dp = (C - base) % a.dh;
              float2 cs;
              if constexpr (PCS) {
                cs = csq[(r >> 2) & 1][r & 3][j];
              } else {
                cs = a.rope[(size_t)pos * (a.dh >> 1) + (dp >> 1)];
              }
              const float o0 = v * cs.x - pv * cs.y;
              const float o1 = pv * cs.x + v * cs.y;
              const uint32_t packed = (uint32_t)f2h(o0) | ((uint32_t)f2h(o1) << 16);
              if (C < a.q_cols) {
                *(uint32_t*)(a.Q + (size_t)R * a.q_cols + C) = packed;
              } else {
                const int hg = (C - base) / a.dh;
                *(uint32_t*)(a.kv + (size_t)(kvs / kPage) * a.page_stride +
                             ((size_t)hg * kPage + (kvs & (kPage - 1))) * a.dh + dp) = packed;
              }
            }
          } else {
            const int cv = C - a.q_cols - a.kv_cols;
            const int hg = cv / a.dh, d = cv % a.dh;
            a.kv[(size_t)(kvs / kPage) * a.page_stride + (size_t)a.Hkv * kPage * a.dh +
                 ((size_t)hg * a.dh + d) * kPage + (kvs & (kPage - 1))] = (_Float16)v;
          }
        }
      } else if constexpr (EPI == EPI_RESID) {
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          const int C = col_w + 32 * j + lc;
          float x = 0.f;
          if (rok) {
            x = xq[(r >> 2) & 1][r & 3][j] + acc[i][j][r];
            a.X[(size_t)R * a.D + C] = x;
            uint16_t hi, lo;
            split_f16(x * gn[j], hi, lo);
            const size_t off = afrag_off(R, C, a.MTtot);
            a.Nhi[off] = hi;
            a.Nlo[off] = lo;
          }
          // sum of squares over the 16 columns of this lane's strip
          float sq = x * x;
          sq += __shfl_xor(sq, 1);
          sq += __shfl_xor(sq, 2);
          sq += __shfl_xor(sq, 4);
          sq += __shfl_xor(sq, 8);
          if (rok && (lc & 15) == 0) a.ss_out[(size_t)R * (a.D >> 4) + (C >> 4)] = sq;
        }
      } else if constexpr (EPI == EPI_SILU) {
        // a 32-column tile is one (gate strip, up strip) pair
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          const int C = col_w + 32 * j + lc;
          const float v = acc[i][j][r] * ir;
          const float pv = __shfl_xor(v, 16);
          if (rok && lc < 16) {
            const float act = v / (1.f + __expf(-v)) * pv;
            const int F = (C >> 5) * 16 + lc;
            uint16_t hi, lo;
            split_f16(act, hi, lo);
            const size_t off = afrag_off(R, F, a.MTtot);
            a.act_hi[off] = hi;
            a.act_lo[off] = lo;
          }
        }
      } else {  // EPI_LM: per-row max / lowest argmax over this wave's columns
        float best = -INFINITY;
        int bidx = 0x7fffffff;
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          const int C = col_w + 32 * j + lc;
          const float v = acc[i][j][r] * ir;
          if (rok && a.logits) a.logits[(size_t)R * a.vocab + C] = v;
          if (v > best) {  // columns ascend with j: ties keep the lower one
            best = v;
            bidx = C;
          }
        }
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) {
          const float ov = __shfl_xor(best, o);
          const int oi = __shfl_xor(bidx, o);
          if (ov > best || (ov == best && oi < bidx)) {
            best = ov;
            bidx = oi;
          }
        }
        if (lc == 0) {
          const int lr = R - (row_w - wy * 32 * WM);  // row within the workgroup tile
          lm_best[wx * BM + lr] = float2{best, 0.f};
          lm_idx[wx * BM + lr] = bidx;
        }
      }
    }
  });
  if constexpr (EPI == EPI_LM) {
    __syncthreads();
    // merge the column parts (lower columns first) and publish
    for (int lr = threadIdx.x; lr < BM; lr += 64 * WY * WX) {
      const int R = (row_w - wy * 32 * WM) + lr;  // the tile origin
      float b = lm_best[lr].x;
      int bi = lm_idx[lr];
#pragma unroll
      for (int x = 1; x < WX; ++x) {
        const float b2 = lm_best[x * BM + lr].x;
        const int bi2 = lm_idx[x * BM + lr];
        if (b2 > b || (b2 == b && bi2 < bi)) {
          b = b2;
          bi = bi2;
        }
      }
      if (R < a.M) {
        a.part_val[(size_t)R * a.n_part + cb] = b;
        a.part_idx[(size_t)R * a.n_part + cb] = bi;
      }
    }
  }
}

// 128 x 128 wave tiles (256 accumulators) run one wave per SIMD
constexpr int tiled_occupancy(int WM, int WN) { return WM * WN >= 16 ? 1 : 2; }

template <int WY, int WX, int WM, int WN, int EPI, bool HI_LO>
__global__ __launch_bounds__(64 * WY * WX, tiled_occupancy(WM, WN)) void gemm_tiled(
    GemmArgs a, const float* __restrict__ inv_rms, int RB, int CB, int S) {
  constexpr int NW = WY * WX;
  constexpr int BM = 32 * WM * WY, BN = 32 * WN * WX;
  constexpr int AF = BM / 16;              // A fragments per K step
  constexpr int NA = HI_LO ? 2 * AF : AF;  // with the lo part
  constexpr int WF = BN / 16;              // weight fragments per K step
  constexpr int NF = NA + WF;
  constexpr int LPT = NF / NW;  // 16-byte loads per thread per K step (NF*64 / (64*NW))
  static_assert(NF % NW == 0, "fragments per step");
  // ring depth: two workgroups per CU for the small tiles, else one
  constexpr int LDS_BUDGET = (NW == 4 && WM * WN < 16) ? 76 * 1024 : 150 * 1024;
  constexpr int ST0 = LDS_BUDGET / (NF * 1024);
  constexpr int ST = ST0 < 3 ? 3 : (ST0 > 6 ? 6 : ST0);
  __shared__ u32x4 sbuf[ST][NF][64];
  __shared__ float2 lm_best[EPI == EPI_LM ? WX * BM : 1];
  __shared__ int lm_idx[EPI == EPI_LM ? WX * BM : 1];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wy = wave / WX, wx = wave % WX;
  const TileCoord tc = tile_coord(blockIdx.x, gridDim.x, RB, CB);
  const int mt0 = tc.rb * AF;
  const int kts = (a.KT + S - 1) / S;
  const int kb = tc.split * kts, ke = min(a.KT, kb + kts);

  // this thread's share of a K step: unit u = q*64*NW + tid is fragment
  // q*NW + wave (wave-uniform), lane u%64
  const u32x4* src[LPT];
  size_t kstride[LPT];
#pragma unroll
  for (int q = 0; q < LPT; ++q) {
    const int f = q * NW + wave;
    if (f < NA) {
      const int mt = min(mt0 + (f % AF), a.MTtot - 1);  // rows past the operand: any valid tile
      src[q] = (const u32x4*)(f < AF ? a.Ahi : a.Alo) + (size_t)mt * 64 + lane;
      kstride[q] = (size_t)a.MTtot * 64;
    } else {
      const int st = tc.cb * WF + (f - NA);
      src[q] = (const u32x4*)a.W + (size_t)(st >> 2) * a.wg + (size_t)(st & 3) * 64 + lane;
      kstride[q] = a.wk;
    }
  }
  // copy K step kt into ring slot `slot`: lane l's 16 bytes land at
  // sbuf[slot][f][l].  Steps past the range re-copy the last one, so every
  // iteration issues the same number of copies (constant vmcnt targets).
  auto issue = [&](int slot, int kt) __attribute__((always_inline)) {
    kt = min(kt, ke - 1);
#pragma unroll
    for (int q = 0; q < LPT; ++q)
      __builtin_amdgcn_global_load_lds((const void*)(src[q] + (size_t)kt * kstride[q]),
                                       (lds_void*)&sbuf[slot][q * NW + wave][0], 16, 0, 0);
  };

  f32x16 acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // operand fragment of 32 rows (or columns) starting at fragment f0, K
  // sub-step s (16 of the 32): lane l takes row l%32, K 16s + 8(l/32)..+8
  const int fl = (lane & 15) + 16 * (lane >> 5);  // lane within the fragment, s = 0
  const int fo = (lane >> 4) & 1;                 // second fragment for lanes 16-31 / 48-63
  // the operands of one K step, held in registers: read from LDS one step
  // ahead so the reads of step i+1 overlap the MFMAs of step i
  struct Ops {
    u32x4 ah[2][WM], al[2][HI_LO ? WM : 1], bw[2][WN];
  };
  auto read_ops = [&](int buf, Ops& o) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int i = 0; i < WM; ++i) {
        o.ah[s][i] = sbuf[buf][wy * 2 * WM + 2 * i + fo][fl + 32 * s];
        if constexpr (HI_LO) o.al[s][i] = sbuf[buf][AF + wy * 2 * WM + 2 * i + fo][fl + 32 * s];
      }
#pragma unroll
      for (int j = 0; j < WN; ++j) o.bw[s][j] = sbuf[buf][NA + wx * 2 * WN + 2 * j + fo][fl + 32 * s];
    }
  };
  // the MFMAs of one step; the first one goes out before `between` (the
  // next step's LDS reads), so the register wait it needs covers only the
  // previous step's reads, and the reads then overlap the remaining MFMAs
  auto mfma_ops = [&](const Ops& o, auto&& between) __attribute__((always_inline)) {
    acc[0][0] = mfma32_f16(o.ah[0][0], o.bw[0][0], acc[0][0]);
    __builtin_amdgcn_sched_barrier(0);
    between();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          if (s != 0 || i != 0 || j != 0) acc[i][j] = mfma32_f16(o.ah[s][i], o.bw[s][j], acc[i][j]);
          if constexpr (HI_LO) acc[i][j] = mfma32_f16(o.al[s][i], o.bw[s][j], acc[i][j]);
        }
  };

  // Ring schedule: step j lives in slot j % ST.  Iteration i waits until
  // step i+1 has landed (own copies: vmcnt; everyone's: barrier), refills
  // the slot of step i-1 with step i+ST-1, reads step i+1's operands and
  // multiplies step i's (read in the previous iteration).
  const int nk = ke - kb;
  if (nk > 0) {
    Ops o0, o1;
#pragma unroll
    for (int st = 0; st < ST - 1; ++st) issue(st, kb + st);
    vm_wait<LPT * (ST - 2)>();
    block_barrier();
    read_ops(0, o0);
    for (int i = 0; i < nk; i += 2) {
      vm_wait<LPT * (ST - 3)>();
      block_barrier();
      issue((i + ST - 1) % ST, kb + i + ST - 1);
      mfma_ops(o0, [&]() { read_ops((i + 1) % ST, o1); });
      __builtin_amdgcn_sched_barrier(0);
      if (i + 1 < nk) {
        vm_wait<LPT * (ST - 3)>();
        block_barrier();
        issue((i + ST) % ST, kb + i + ST);
        mfma_ops(o1, [&]() { read_ops((i + 2) % ST, o0); });
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  vm_wait<0>();  // no copy may land after the workgroup's LDS is released

  const int row_w = tc.rb * BM + wy * 32 * WM;
  const int col_w = tc.cb * BN + wx * 32 * WN;
  if (S > 1) {
    // K split: publish this split's partial tile with device-scope
    // (write-through) stores, in lane-native order (float4 group g of
    // accumulator (i, j) of lane l at ((i*WN + j)*4 + g)*64 + l of the
    // wave's slice), then count arrivals.  The last split of the tile to
    // arrive reads every split's partial back, its own included, and sums
    // them in split order (the same order whichever arrives last, so results
    // are deterministic), then runs the epilogue: no second kernel.
    const int unit = tc.rb * CB + tc.cb;
    auto slice = [&](int sp) {
      return a.part + ((((size_t)sp * RB + tc.rb) * CB + tc.cb) * NW + wave) * (size_t)(16 * WM * WN * 64);
    };
    float* mine = slice(tc.split);
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          st_f4_dev(mine, (uint32_t)((((i * WN + j) * 4 + g) * 64 + lane) * 16),
                    float4{acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]});
    __builtin_amdgcn_s_waitcnt(vmcnt_enc(0));  // this thread's stores are done
    __syncthreads();
    // whether this split arrived last goes through the (now idle) operand ring
    uint32_t* last_flag = (uint32_t*)&sbuf[0][0][0];
    if (tid == 0) *last_flag = atomicAdd(a.cnt + unit, 1u) == (uint32_t)S - 1u;
    __syncthreads();
    if (!*last_flag) return;
    if (tid == 0) store_dev_u32(a.cnt + unit, 0u);  // every split has arrived: ready for the next launch
    for (int sp = 0; sp < S; ++sp) {
      const float* src = slice(sp);
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const float4 x = ld_f4_dev(src, (uint32_t)((((i * WN + j) * 4 + g) * 64 + lane) * 16));
            if (sp == 0) {
              acc[i][j][4 * g] = x.x;
              acc[i][j][4 * g + 1] = x.y;
              acc[i][j][4 * g + 2] = x.z;
              acc[i][j][4 * g + 3] = x.w;
            } else {
              acc[i][j][4 * g] += x.x;
              acc[i][j][4 * g + 1] += x.y;
              acc[i][j][4 * g + 2] += x.z;
              acc[i][j][4 * g + 3] += x.w;
            }
          }
    }
  }
  tiled_epilogue<WY, WX, WM, WN, EPI>(a, acc, row_w, col_w, inv_rms, lm_best, lm_idx, tc.cb);
}

// Inverse RMS of each row from its per-16-column sums of squares (one wave
// per row, fixed summation order).
__global__ __launch_bounds__(256) void row_inv_rms(const float* __restrict__ ss, int ss_n, int M, float inv_dim,
                                                   float eps, float* __restrict__ out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= M) return;
  float s = 0.f;
  for (int q = lane; q < ss_n; q += 64) s += ss[(size_t)row * ss_n + q];
  s = wave_sum(s);
  if (lane == 0) out[row] = rsqrtf(s * inv_dim + eps);
}

template <int WY, int WX, int WM, int WN, int EPI, bool HI_LO>
static hipError_t launch_t(const GemmArgs& a, const float* inv_rms, int splits, hipStream_t s) {
  const int BM = 32 * WM * WY, BN = 32 * WN * WX, NT = 64 * WY * WX;
  const int CB = a.NT * 16 / BN, RB = (a.MTtot * 16 + BM - 1) / BM;
  const int total = CB * RB * splits;
  hvd_launch((gemm_tiled<WY, WX, WM, WN, EPI, HI_LO>), dim3(total), dim3(NT), 0, s, a, inv_rms, RB, CB,
                     splits);
  return hipGetLastError();
}

template <int EPI, bool HI_LO>
static hipError_t launch_th(const GemmArgs& a, const float* inv_rms, int tile, int splits, hipStream_t s) {
  switch (tile) {
    case 0: return launch_t<2, 2, 2, 2, EPI, HI_LO>(a, inv_rms, splits, s);  // 128 x 128, 4 waves
    case 1: return launch_t<2, 2, 2, 4, EPI, HI_LO>(a, inv_rms, splits, s);  // 128 x 256, 4 waves
    case 2: return launch_t<4, 2, 2, 4, EPI, HI_LO>(a, inv_rms, splits, s);  // 256 x 256, 8 waves
    case 3: return launch_t<2, 2, 4, 4, EPI, HI_LO>(a, inv_rms, splits, s);  // 256 x 256, 4 waves
    case 4: return launch_t<2, 4, 2, 2, EPI, HI_LO>(a, inv_rms, splits, s);  // 128 x 256, 8 waves
  }
  return hipErrorInvalidValue;
}

template <int EPI>
static hipError_t launch_te(const GemmArgs& a, const float* inv_rms, int tile, bool hi_lo, int splits, hipStream_t s) {
  return hi_lo ? launch_th<EPI, true>(a, inv_rms, tile, splits, s) : launch_th<EPI, false>(a, inv_rms, tile, splits, s);
}

hipError_t launch_gemm_tiled(int epi, const GemmArgs& a, int tile, bool hi_lo, int splits, float* inv_rms,
                             hipStream_t s) {
  if (epi != EPI_RESID) {
    const int rows = a.MTtot * 16;
    hvd_launch(row_inv_rms, dim3((rows + 3) / 4), dim3(256), 0, s, a.ss, a.ss_n, rows, a.inv_dim, a.eps,
                       inv_rms);
  }
  switch (epi) {
    case EPI_QKV: return launch_te<EPI_QKV>(a, inv_rms, tile, hi_lo, splits, s);
    case EPI_RESID: return launch_te<EPI_RESID>(a, inv_rms, tile, hi_lo, splits, s);
    case EPI_SILU: return launch_te<EPI_SILU>(a, inv_rms, tile, hi_lo, splits, s);
    case EPI_LM: return launch_te<EPI_LM>(a, inv_rms, tile, hi_lo, splits, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace hvd
