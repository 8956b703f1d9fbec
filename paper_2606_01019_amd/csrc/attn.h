// Device code of the verify attention and its split-KV merge, shared by the
// stand-alone kernels (attn.hip) and the one-launch verify step (flow.hip).
// See attn.hip for the design.
#pragma once

#include "common.h"
#include "kernels.h"

#include <type_traits>

namespace hvd {

// Item reads go through the constant address space: items are read-only
// while attention runs, and uniform addresses there become scalar loads
// whose results (the first sub-chunk's page ids included) sit in SGPRs.
typedef const __attribute__((address_space(4))) AttnItem ConstItem;

// Slack of the online softmax's reference max (base-2 units): the largest
// weight 2^(s - m) is 2^kAttnLazy.
constexpr float kAttnLazy = 8.f;

// NP = pages staged per sub-chunk (the launch picks it from the chunk
// length), so short decode chunks issue only the loads they need.  NW waves
// hold TPW row tiles each: an item covers up to 16*NW*TPW query rows (64 for
// short drafts, up to 256 so one item covers all rows of a long draft and
// its keys are read once).
// Workgroups per CU the register budget is sized for: two 4-wave
// workgroups share a CU while their staged sub-chunks fit LDS together.
constexpr int attn_occupancy(int DH, int NP, int NW) { return NW == 4 && NP * kPage * DH <= 64 * 128 ? 2 : 1; }

// One attention work item by one workgroup of 64 * NW threads (smem: the
// sub-chunk staging buffers).  COH: the item runs inside a larger kernel:
// the K/V of positions >= ctx (written by the same launch into pages that
// are reused from launch to launch) is read with device-scope loads, the
// outputs are written with device-scope stores, and the query rows (a
// buffer written once per launch) with ordinary loads; hk.wait() runs once
// the first sub-chunk's cached K/V is requested, hk.done() after the outputs.
// Hooks::kDevOut alone asks for device-scope outputs (inputs from earlier
// launches).  hk.after_issue() runs once the first sub-chunk's K/V and the
// query rows are requested and may request Hooks::kPending more loads per
// thread, which the item does not wait for.
template <int DH, int NP, int NW, int TPW, bool COH, class Hooks>
__device__ __forceinline__ void attn_item(const AttnArgs& a, ConstItem* ip, unsigned char* smem, Hooks& hk) {
  constexpr int NT = 64 * NW;           // threads
  constexpr int RPI = 16 * NW * TPW;    // query rows per item
  constexpr int CH = NP * kPage;        // positions per sub-chunk
  constexpr int KSEG = DH / 8;          // 16-byte segments per K row
  // V^T in LDS: row d holds the sub-chunk's CH positions in 16-byte
  // granules, granule 4b + j of 32-position block b holding positions
  // 32b + 4j .. 32b + 4j + 3 and 32b + 16 + 4j .. + 3 -- exactly the eight
  // K values one lane group needs as the B operand of a 16x16x32 MFMA over
  // that block (one 16-byte read, no register shuffling).  Granules are
  // XOR-swizzled by row so that the 16 rows one read instruction touches at
  // a time land in distinct banks (64 banks of 4 bytes).
  constexpr int VGR = CH / 8;                        // granules per row
  constexpr int VGM = VGR < 16 ? VGR : 16;           // swizzle span (granules)
  constexpr unsigned VRB = CH >= 128 ? 1 : 128 / CH; // rows per 256 bytes
  auto vgran = [](int gr, int d) __attribute__((always_inline)) {
    return (gr & ~(VGM - 1)) | ((gr & (VGM - 1)) ^ (int)(((unsigned)d / VRB) & (VGM - 1)));
  };
  // half-word offset within a row of 8-byte unit u (positions 4u .. 4u+3)
  auto vslot = [&](int u, int d) __attribute__((always_inline)) {
    return vgran(((u >> 3) << 2) | (u & 3), d) * 8 + ((u >> 2) & 1) * 4;
  };
  constexpr int LPP = 4 * DH / NT;      // 16-byte loads per thread per page (K and V: 4*DH units)
  static_assert(NP >= 2 && NP <= kItemPages && (NP & (NP - 1)) == 0, "pages per sub-chunk");
  static_assert(LPP >= 1 && LPP * NT == 4 * DH, "page units per thread");
  // Sub-chunks of up to 4 pages are double-buffered in LDS: a sub-chunk is
  // staged into the buffer its predecessor's predecessor used, which every
  // wave has finished reading once it passed the previous staging barrier,
  // so one barrier per sub-chunk suffices.
  constexpr bool DB = NP <= 4;
  constexpr bool DEV_OUT = COH || Hooks::kDevOut;
  static_assert(Hooks::kPending >= 0 && Hooks::kPending < 64, "loads left in flight");
  constexpr int BUF_BYTES = CH * DH * 2 * 2;       // K and V of one sub-chunk
  _Float16* sK = (_Float16*)smem;                  // [CH][DH], segment-swizzled
  _Float16* sV = (_Float16*)(smem + CH * DH * 2);  // [DH][CH], granule-regrouped and swizzled

  const int kdr = ip->k;
  if (kdr < 0) return;  // grid padding
  const int slot = ip->slot, ctx = ip->ctx, cu = ip->cu, g = ip->g;
  const int nch = ip->nch, rg = ip->rg, part = ip->part;
  const bool tree = ip->tree != 0;  // token tree: rows see the context and their own path
  const int p_begin = ip->p_begin, p_end = ip->p_end;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int G = a.group;
  const int R = (kdr + 1) * G;
  const int lg = lane >> 4;
  const size_t vhalf = (size_t)a.Hkv * kPage * DH;
  const _Float16* kvg = a.kv + (size_t)g * kPage * DH;  // this kv head's K block in a page

  // per-wave state of its (up to) TPW 16-row tiles, kept across sub-chunks
  int tile_row[TPW];
  bool tile_on[TPW];
  f16x8 qf[TPW][DH / 32];
  float m[TPW], lsum[TPW];
  f32x4 o[TPW][DH / 16];
#pragma unroll
  for (int q = 0; q < TPW; ++q) {
    m[q] = -INFINITY;
    lsum[q] = 0.f;
    const int row_base = rg * RPI + (wave + NW * q) * 16;
    tile_on[q] = row_base < R;
    tile_row[q] = row_base + (lane & 15);
#pragma unroll
    for (int d = 0; d < DH / 16; ++d) o[q][d] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // ---- K/V loads of one sub-chunk, all in flight at once (page-major: per
  // page, units [0, 2DH) are K rows, [2DH, 4DH) V rows of the head).  Pages
  // past the sub-chunk's end repeat its first page (in-bounds, cached; their
  // V is zeroed when staged).  The next sub-chunk's loads are issued before
  // the current one is computed, so its latency hides behind the MFMAs.
  // tree rows: ancestor sets (rows past R take the last row's)
  uint64_t anc[TPW];
#pragma unroll
  for (int q = 0; q < TPW; ++q) {
    const int r = tile_row[q];
    anc[q] = tree ? a.tree_mask[cu + (r < R ? r / G : kdr)] : 0;
  }
  // query fragments (rows past R read a valid row; their results are dropped)
  auto load_q = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < TPW; ++q) {
      const int r = tile_row[q];
      const int i = r < R ? r / G : kdr;
      const int h = g * G + (r < R ? r % G : 0);
#pragma unroll
      for (int kd = 0; kd < DH / 32; ++kd) {
        const size_t e = ((size_t)(cu + i) * a.Hq + h) * DH + kd * 32 + lg * 8;
        qf[q][kd] = *(const f16x8*)(a.Q + e);
      }
    }
  };
  u32x4 buf[NP][LPP];
  // coh: the sub-chunk holds positions >= ctx, written by this kernel
  auto issue = [&](const int (&pgid)[NP], bool coh) __attribute__((always_inline)) {
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int j = 0; j < LPP; ++j) {
        const int u = j * NT + tid;
        const size_t off = u < 2 * DH ? (size_t)u * 8 : vhalf + (size_t)(u - 2 * DH) * 8;
        const _Float16* page = kvg + (size_t)pgid[p] * a.page_stride;
        if (COH && coh)
          buf[p][j] = ld_16_dev(page, (uint32_t)(off * 2));
        else
          buf[p][j] = *(const u32x4*)(page + off);
      }
  };
  {
    int pgid[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) pgid[p] = ip->pages[p];
    if constexpr (COH) {
      // cached positions only: requested before the wait
      const bool fresh = p_begin + CH > ctx;
      if (!fresh) issue(pgid, false);
      hk.wait();
      if (fresh) issue(pgid, true);
    } else {
      issue(pgid, false);
    }
    load_q();
  }
  // pool pages of the next sub-chunk to issue, one per lane (lane p < NP:
  // page p; past the sub-chunk's end, its first page), loaded a sub-chunk
  // ahead so issuing never waits on a page-table read
  auto next_pages = [&](int nsub) __attribute__((always_inline)) {
    const int np_sub = (min(CH, p_end - nsub) + kPage - 1) / kPage;
    return a.pt[(size_t)slot * a.pt_stride + (nsub >> 4) + (lane < np_sub ? lane : 0)];
  };
  int pg_next = p_begin + CH < p_end ? next_pages(p_begin + CH) : 0;
  hk.after_issue();
  // Wait here for everything issued so far (the first sub-chunk is staged
  // right after anyway): the waitcnt pass then knows the query fragments are
  // in, and places no wait for them inside the loop, where it would also
  // wait for the next sub-chunk's loads.  Loads the hook added stay in flight.
  __builtin_amdgcn_s_waitcnt(vmcnt_enc(Hooks::kPending));

  int nbuf = 0;
  for (int sub = p_begin; sub < p_end; sub += CH) {
    const int n_pos = min(CH, p_end - sub);
    if constexpr (DB) {
      sK = (_Float16*)(smem + nbuf * BUF_BYTES);
      sV = (_Float16*)(smem + nbuf * BUF_BYTES + CH * DH * 2);
      nbuf ^= 1;
    } else {
      if (sub != p_begin) __syncthreads();  // previous sub-chunk fully consumed
    }
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int j = 0; j < LPP; ++j) {
        const int u = j * NT + tid;
        u32x4 x = buf[p][j];
        if (u < 2 * DH) {
          const int t = u / KSEG, sgm = u % KSEG;
          const int pos = p * kPage + t;
          *(u32x4*)(sK + pos * DH + ((sgm ^ (pos & 15)) & (KSEG - 1)) * 8) = x;
        } else {
          const int v = u - 2 * DH;
          const int d = v >> 1, hh = v & 1;
          // 8 positions pp .. pp+7 of row d; positions past the end are
          // zeroed (their probabilities are 0, and stale values must not
          // turn that into NaN)
          const int pp = p * kPage + hh * 8;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t keep = (pp + 2 * e + 1 < n_pos) ? 0xffffffffu : (pp + 2 * e < n_pos ? 0xffffu : 0u);
            x[e] &= keep;
          }
          const int u0 = pp >> 2;  // 8-byte units (4 positions)
          _Float16* row = sV + (size_t)d * CH;
          *(uint2*)(row + vslot(u0, d)) = uint2{x[0], x[1]};
          *(uint2*)(row + vslot(u0 + 1, d)) = uint2{x[2], x[3]};
        }
      }
    __syncthreads();
    if (sub + CH < p_end) {
      int pgid[NP];
#pragma unroll
      for (int p = 0; p < NP; ++p) pgid[p] = __builtin_amdgcn_readlane(pg_next, p);
      issue(pgid, sub + 2 * CH > ctx);
      if (sub + 2 * CH < p_end) pg_next = next_pages(sub + 2 * CH);
    }

    // The wave's row tiles over the sub-chunk in groups of SG 16-position
    // blocks: all scores S^T = K Q^T of a group first (independent
    // accumulator chains; each K fragment read from LDS once and used by
    // every tile of the wave), one online-softmax update per tile, then
    // O^T += V^T P^T over the group's block pairs (each V fragment read once
    // for all tiles).  Every position is computed; those past the end are
    // masked, so no load is conditional.  Tile 0 is live whenever any is.
    constexpr int NB = CH / 16;                      // 16-position blocks
    // blocks per score group (register budget; at least one block pair)
    constexpr int SG0 = 4 / TPW < 2 ? 2 : 4 / TPW;
    constexpr int SG = NB < SG0 ? NB : SG0;
    if (tile_on[0]) {
      int lim[TPW];  // last visible position of each tile's rows, sub-chunk-relative
#pragma unroll
      for (int q = 0; q < TPW; ++q) {
        const int r = tile_row[q];
        lim[q] = ctx + (r < R ? r / G : kdr) - sub;
      }
      // smallest of them over the wave (its first row: rows ascend)
      const int lim_min = tree ? ctx - 1 - sub : ctx + (rg * RPI + wave * 16) / G - sub;
      // Waves of two row tiles: the group loop is instantiated per count NQ
      // of live tiles (a prefix of the wave's tiles), so no per-tile branch
      // sits inside it, and K and V fragments are read ahead of their
      // MFMAs.  One tile (whose 4-wave items run two to a CU) measured
      // slower with the read-ahead's registers; three fill the registers:
      // there, one instance that tests each tile, fragments read where used.
      constexpr bool KPIPE = TPW == 2;
      auto live = [&](int q) __attribute__((always_inline)) { return KPIPE || q == 0 || tile_on[q]; };
      auto run = [&](auto nq) __attribute__((always_inline)) {
        constexpr int NQ = decltype(nq)::value;
#pragma unroll 1
        for (int g0 = 0; g0 < NB; g0 += SG) {  // not unrolled: keeps each group's LDS reads in its group
          f32x4 sc[TPW][SG];
          // K fragments one head-dim step ahead of the MFMAs that use them
          // (three-tile waves: read per step, for registers)
          f16x8 kf[KPIPE ? 2 : 1][SG];
          auto read_k = [&](int kd, f16x8 (&dst)[SG]) __attribute__((always_inline)) {
            const int sg = kd * 4 + lg;
#pragma unroll
            for (int b = 0; b < SG; ++b) {
              const int p = (g0 + b) * 16 + (lane & 15);
              dst[b] = *(const f16x8*)(sK + p * DH + ((sg ^ (p & 15)) & (KSEG - 1)) * 8);
            }
          };
          if constexpr (KPIPE) read_k(0, kf[0]);
#pragma unroll
          for (int kd = 0; kd < DH / 32; ++kd) {
            if constexpr (KPIPE) {
              if (kd + 1 < DH / 32) read_k(kd + 1, kf[(kd + 1) & 1]);
            } else {
              read_k(kd, kf[0]);
            }
#pragma unroll
            for (int q = 0; q < NQ; ++q)
              if (live(q)) {
#pragma unroll
                for (int b = 0; b < SG; ++b)
                  sc[q][b] = mfma_f16(kf[KPIPE ? kd & 1 : 0][b], qf[q][kd], kd ? sc[q][b] : f32x4{0.f, 0.f, 0.f, 0.f});
              }
          }
          // V fragments of the first block pair, requested before the softmax
          // so that their LDS latency overlaps it
          auto read_v = [&](int c, f16x8 (&dst)[DH / 16]) __attribute__((always_inline)) {
            const int gr = 2 * g0 + 4 * c + lg;  // granule of block g0/2 + c for this lane group
#pragma unroll
            for (int dt = 0; dt < DH / 16; ++dt) {
              const int d = dt * 16 + (lane & 15);
              dst[dt] = *(const f16x8*)(sV + (size_t)d * CH + vgran(gr, d) * 8);
            }
          };
          f16x8 vv[DH / 16];
          if constexpr (KPIPE) read_v(0, vv);
          f16x8 pf[TPW][SG / 2 > 0 ? SG / 2 : 1];
          // whole group visible to every row of the wave (wave-uniform): no mask
          const bool full = (g0 + SG) * 16 <= min(lim_min + 1, n_pos);
#pragma unroll
          for (int q = 0; q < NQ; ++q) {
            if (!live(q)) continue;
            // running max m in log2 units; scores scaled inside the exp2's fma
            float bm = -INFINITY;
            if (full) {
#pragma unroll
              for (int b = 0; b < SG; ++b)
#pragma unroll
                for (int j = 0; j < 4; ++j) bm = fmaxf(bm, sc[q][b][j]);
            } else {
#pragma unroll
              for (int b = 0; b < SG; ++b)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                  const int pa = (g0 + b) * 16 + lg * 4 + j;
                  bool vis = pa <= lim[q];
                  if (tree) {  // the context, then the row's ancestors (bit j = position ctx + j)
                    const int rel = pa + sub - ctx;
                    vis = rel < 0 || ((anc[q] >> (rel & 63)) & 1);
                  }
                  sc[q][b][j] = (vis && pa < n_pos) ? sc[q][b][j] : -INFINITY;
                  bm = fmaxf(bm, sc[q][b][j]);
                }
            }
            bm = rows_max(bm);
            // Lazy rescaling: a row's reference m moves only when a score
            // exceeds it by more than kAttnLazy (base-2 units).  The weights
            // 2^(s - m) then stay below 2^kAttnLazy (well inside the fp16 P
            // operand's range), (m, l, O) stay consistent, and the
            // accumulators are rescaled only when some row's reference moves.
            const float cand = bm * a.scale_log2;
            if (__builtin_amdgcn_ballot_w64(cand > m[q] + kAttnLazy)) {
              const bool grow = cand > m[q] + kAttnLazy;
              const float alpha = grow ? __builtin_amdgcn_exp2f(m[q] - cand) : 1.f;  // 0 from -inf
              lsum[q] *= alpha;
#pragma unroll
              for (int dt = 0; dt < DH / 16; ++dt) o[q][dt] *= alpha;
              if (grow) m[q] = cand;
            }
            const float ms = m[q] == -INFINITY ? 0.f : m[q];  // nothing visible yet: every weight is 0
            float ps = 0.f;
#pragma unroll
            for (int b = 0; b < SG; ++b)
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                sc[q][b][j] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[q][b][j], a.scale_log2, -ms));
                ps += sc[q][b][j];
              }
            lsum[q] += ps;
            // B operand of block pair c: positions 32c' + {4lg..4lg+3} and
            // 32c' + 16 + {4lg..4lg+3}, c' = g0/2 + c
#pragma unroll
            for (int c = 0; c < SG / 2; ++c)
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                pf[q][c][j] = (_Float16)sc[q][2 * c][j];
                pf[q][c][4 + j] = (_Float16)sc[q][2 * c + 1][j];
              }
          }
#pragma unroll
          for (int c = 0; c < SG / 2; ++c) {
            if (c > 0 || !KPIPE) read_v(c, vv);
#pragma unroll
            for (int q = 0; q < NQ; ++q)
              if (live(q)) {
#pragma unroll
                for (int dt = 0; dt < DH / 16; ++dt) o[q][dt] = mfma_f16(vv[dt], pf[q][c], o[q][dt]);
              }
          }
        }
      };
      if constexpr (TPW == 1 || !KPIPE) {
        run(std::integral_constant<int, TPW>{});
      } else if (tile_on[TPW - 1]) {
        run(std::integral_constant<int, TPW>{});
      } else {
        run(std::integral_constant<int, 1>{});
      }
    }
  }

#pragma unroll
  for (int q = 0; q < TPW; ++q) {
    if (!tile_on[q]) continue;
    const float l = rows_sum(lsum[q]);
    const int r = tile_row[q];
    const bool rvalid = r < R;
    if (nch == 1) {
      if (rvalid) {
        const int i = r / G, h = g * G + r % G;
        const float inv = l > 0.f ? 1.f / l : 0.f;
        const int row = cu + i;
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) {
          const int col = h * DH + dt * 16 + lg * 4;
          uint16_t hi[4], lo[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) split_f16(o[q][dt][j] * inv, hi[j], lo[j]);
          const size_t off = afrag_off(row, col, a.MTtot);
          const uint2 vh = uint2{hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16)};
          const uint2 vl = uint2{lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16)};
          if constexpr (DEV_OUT) {
            st_u64_dev((uint64_t*)(a.Ohi + off), (uint64_t)vh.x | ((uint64_t)vh.y << 32));
            st_u64_dev((uint64_t*)(a.Olo + off), (uint64_t)vl.x | ((uint64_t)vl.y << 32));
          } else {
            *(uint2*)(a.Ohi + off) = vh;
            *(uint2*)(a.Olo + off) = vl;
          }
        }
      }
    } else {
      const int lr = (wave + NW * q) * 16 + (lane & 15);
      const size_t ps = (size_t)part * RPI + lr;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) {
        const float4 v = float4{o[q][dt][0], o[q][dt][1], o[q][dt][2], o[q][dt][3]};
        if constexpr (DEV_OUT) st_f4_dev(a.part_o, (uint32_t)((ps * DH + dt * 16 + lg * 4) * 4), v);
        else *(float4*)(a.part_o + ps * DH + dt * 16 + lg * 4) = v;
      }
      if (lg == 0) {
        if constexpr (DEV_OUT)
          st_u64_dev((uint64_t*)(a.part_ml + ps * 2), (uint64_t)__float_as_uint(m[q]) |
                                                          ((uint64_t)__float_as_uint(l) << 32));
        else
          *(float2*)(a.part_ml + ps * 2) = float2{m[q], l};
      }
    }
  }
  hk.done();
}



// Merge the chunk partials of one (sequence, kv head, row group):
// O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c.  The merge is
// latency-bound, so QS lanes share one (row, 8 dims): lane q takes chunks
// q, q + QS, ... as a running (M, L, acc) merge over batches whose loads are
// all issued before any is used, and the QS lanes then merge by shuffles.
// One block per (head entry, slice of RPB rows); a.max_rows bounds the
// slices per entry.  QS is 8 for short drafts (few rows to spread over) and
// smaller when an entry has more rows, so blocks past a short entry's rows
// stay few.
// One (head entry, row slice) of the merge by a block of NT threads.  COH:
// partials are read, and the output written, with device-scope accesses
// (COH_IN false: partials read with ordinary loads, for partial buffers no
// reader touches before they are complete and whose lines have one writer).
template <int DH, int QS, int NT, bool COH, bool COH_IN = COH>
__device__ __forceinline__ void combine_slice(const CombineArgs& a, const AttnItem& hd, int slice) {
  constexpr int OCT = DH / 8;            // 8-dim octets per row
  constexpr int RPB = NT / (OCT * QS);   // rows per block
  constexpr int NB = 8;                  // chunks per lane per batch
  const int G = a.group;
  const int R = (hd.k + 1) * G;
  const int t = threadIdx.x;
  const int qq = t % QS, o8 = (t / QS % OCT) * 8;
  const int lr = slice * RPB + t / (QS * OCT);
  const int r = hd.rg * a.rpi + lr;
  if (lr >= a.rpi || r >= R) return;  // the QS lanes of a row leave together
  const float* ml = a.part_ml + ((size_t)hd.part * a.rpi + lr) * 2;
  const float* po = a.part_o + ((size_t)hd.part * a.rpi + lr) * DH + o8;
  const size_t cstride_ml = (size_t)a.rpi * 2, cstride_o = (size_t)a.rpi * DH;
  float M = -INFINITY, L = 0.f;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int c0 = qq; c0 < hd.nch; c0 += QS * NB) {
    float2 mlc[NB];
    float4 x0[NB], x1[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int c = c0 + j * QS;
      mlc[j] = float2{-INFINITY, 0.f};
      x0[j] = x1[j] = float4{0.f, 0.f, 0.f, 0.f};
      if (c < hd.nch) {
        if constexpr (COH_IN) {
          const uint64_t mv = ld_u64_dev((const uint64_t*)(ml + c * cstride_ml));
          mlc[j] = float2{__uint_as_float((uint32_t)mv), __uint_as_float((uint32_t)(mv >> 32))};
          x0[j] = ld_f4_dev(a.part_o, (uint32_t)((po - a.part_o + c * cstride_o) * 4));
          x1[j] = ld_f4_dev(a.part_o, (uint32_t)((po - a.part_o + c * cstride_o + 4) * 4));
        } else {
          mlc[j] = *(const float2*)(ml + c * cstride_ml);
          x0[j] = *(const float4*)(po + c * cstride_o);
          x1[j] = *(const float4*)(po + c * cstride_o + 4);
        }
      }
    }
    float Mn = M;
#pragma unroll
    for (int j = 0; j < NB; ++j) Mn = fmaxf(Mn, mlc[j].x);
    const float sc = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mn);
    L *= sc;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] *= sc;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const float w = (mlc[j].x == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mlc[j].x - Mn);
      L += w * mlc[j].y;
      acc[0] += w * x0[j].x; acc[1] += w * x0[j].y; acc[2] += w * x0[j].z; acc[3] += w * x0[j].w;
      acc[4] += w * x1[j].x; acc[5] += w * x1[j].y; acc[6] += w * x1[j].z; acc[7] += w * x1[j].w;
    }
    M = Mn;
  }
  // merge the QS lanes of this (row, octet)
  float Mx = M;
#pragma unroll
  for (int o = 1; o < QS; o *= 2) Mx = fmaxf(Mx, __shfl_xor(Mx, o));
  const float sc = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mx);
  L *= sc;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] *= sc;
#pragma unroll
  for (int o = 1; o < QS; o *= 2) {
    L += __shfl_xor(L, o);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], o);
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const int i = r / G, h = hd.g * G + r % G;
  uint16_t hi[8], lo[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) split_f16(acc[j] * inv, hi[j], lo[j]);
  const size_t off = afrag_off(hd.cu + i, h * DH + o8, a.MTtot);
  const uint4 vh = uint4{hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16),
                         hi[4] | ((uint32_t)hi[5] << 16), hi[6] | ((uint32_t)hi[7] << 16)};
  const uint4 vl = uint4{lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16),
                         lo[4] | ((uint32_t)lo[5] << 16), lo[6] | ((uint32_t)lo[7] << 16)};
  if constexpr (COH) {
    if (qq == 0 || QS == 1) st_16_dev(a.Ohi, (uint32_t)(off * 2), vh);
    if (qq == 1 || QS == 1) st_16_dev(a.Olo, (uint32_t)(off * 2), vl);
  } else {
    if (qq == 0 || QS == 1) *(uint4*)(a.Ohi + off) = vh;
    if (qq == 1 || QS == 1) *(uint4*)(a.Olo + off) = vl;
  }
}




}  // namespace hvd
