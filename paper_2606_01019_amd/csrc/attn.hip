// Verify attention over the paged fp16 KV cache (gfx950, MFMA 16x16x32 f16).
//
// For one sequence, the (k+1) query rows of the verify step times the
// Hq/Hkv q-heads of one kv head g form R = (k+1)*group query vectors; row
// r = i*group + hh is draft row i (position ctx+i) of q-head g*group+hh and
// may attend to key positions 0..ctx+i.  A workgroup (4 waves) handles one KV
// chunk of one (sequence, kv head, row group of up to 128 rows), in
// sub-chunks of up to kAttnChunk positions: it copies a sub-chunk's K and V
// pages into LDS with every load in flight at once (decode-size chunks are
// latency-bound, not bandwidth-bound), then each wave runs its <= 2 row tiles
// over it, carrying the online-softmax state to the next sub-chunk.
//
// Scores are computed transposed, S^T = K Q^T, so the fp32 C fragment of a
// lane holds 4 key positions of one query row; the same registers, converted
// to fp16, are the B operand of O^T = V^T P^T with the contraction index
// permuted consistently on both operands (positions {4g..4g+3, 16+4g..16+4g+3}
// for lane group g).  V is stored transposed inside each 16-token page
// ([dh][16]) and kept transposed in LDS.  LDS rows are XOR-swizzled so the
// 16 lanes of a fragment read hit distinct banks.
// Online softmax in fp32 base 2; rows see only their causal prefix; keys at
// positions >= ctx+k+1 are never used (their contents may be stale).
// A single-chunk item writes the normalized output straight into the O GEMM's
// hi/lo operand; multi-chunk items write (m, l, unnormalized O) partials that
// attn_combine merges in chunk order.
#include "common.h"
#include "kernels.h"

namespace hvd {

template <int DH>
__global__ __launch_bounds__(256) void verify_attn(AttnArgs a) {
  constexpr int CH = kAttnChunk;
  constexpr int KSEG = DH / 8;          // 16-byte segments per K row
  extern __shared__ __align__(16) unsigned char smem[];
  _Float16* sK = (_Float16*)smem;                       // [CH][DH], segment-swizzled
  _Float16* sV = (_Float16*)(smem + CH * DH * 2);       // [DH][CH], 8-byte-unit-swizzled

  __shared__ int spg[kAttnChunk / kPage];  // page ids of the current sub-chunk
  const AttnItem it = a.items[blockIdx.x];
  if (it.k < 0) return;  // grid padding
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int G = a.group;
  const int R = (it.k + 1) * G;
  const int p_begin = it.p_begin;
  const int p_end = it.p_end;
  const int lg = lane >> 4;
  const size_t vhalf = (size_t)a.Hkv * kPage * DH;

  // per-wave state of its (up to) two 16-row tiles, kept across sub-chunks
  int tile_row[2];
  bool tile_on[2];
  f16x8 qf[2][DH / 32];
  float m[2] = {-INFINITY, -INFINITY}, lsum[2] = {0.f, 0.f};
  f32x4 o[2][DH / 16];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int row_base = it.rg * 128 + (wave + 4 * q) * 16;
    tile_on[q] = row_base < R;
    tile_row[q] = row_base + (lane & 15);
    const int r = tile_row[q];
    const bool rvalid = r < R;
    const int i = rvalid ? r / G : it.k;
    const int h = it.g * G + (rvalid ? r % G : 0);
#pragma unroll
    for (int kd = 0; kd < DH / 32; ++kd)
      qf[q][kd] = (tile_on[q] && rvalid)
                      ? *(const f16x8*)(a.Q + ((size_t)(it.cu + i) * a.Hq + h) * DH + kd * 32 + lg * 8)
                      : f16x8{0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int d = 0; d < DH / 16; ++d) o[q][d] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  for (int sub = p_begin; sub < p_end; sub += CH) {
    const int n_pos = min(CH, p_end - sub);
    const int n_pages = (n_pos + kPage - 1) / kPage;
    if (sub != p_begin) __syncthreads();  // previous sub-chunk fully consumed
    if (tid < n_pages) spg[tid] = a.pt[(size_t)it.slot * a.pt_stride + (sub >> 4) + tid];
    __syncthreads();
    // ---- stage K and V of the sub-chunk into LDS (all loads issued before any use)
    {
      constexpr int K_UNITS = CH * KSEG;              // 16-byte units of K
      constexpr int V_UNITS = CH / kPage * DH * 2;    // 16-byte units of V (2 per d row per page)
      constexpr int PER = (K_UNITS + V_UNITS) / 256;
      uint4 buf[PER];
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int u = j * 256 + tid;
        const bool isk = u < K_UNITS;
        const int v = u - K_UNITS;
        const int page_i = isk ? u / (kPage * KSEG) : v / (DH * 2);
        const int off = isk ? u % (kPage * KSEG) : v % (DH * 2);  // K: t*KSEG + s; V: d*2 + half
        buf[j] = uint4{0, 0, 0, 0};
        if (page_i < n_pages) {
          const int pg = spg[page_i];
          const _Float16* base = a.kv + (size_t)pg * a.page_stride +
                                 (isk ? (size_t)it.g * kPage * DH : vhalf + (size_t)it.g * DH * kPage);
          buf[j] = *(const uint4*)(base + (size_t)off * 8);
        }
      }
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int u = j * 256 + tid;
        if (u < K_UNITS) {
          const int page_i = u / (kPage * KSEG), off = u % (kPage * KSEG);
          const int t = off / KSEG, sgm = off % KSEG;
          const int p = page_i * kPage + t;
          *(uint4*)(sK + p * DH + ((sgm ^ (p & 15)) & (KSEG - 1)) * 8) = buf[j];
        } else {
          const int v = u - K_UNITS;
          const int page_i = v / (DH * 2), off = v % (DH * 2);
          const int d = off >> 1, hh = off & 1;
          // 8 positions page_i*16 + hh*8 .. +7 of row d; zero positions past the end
          uint4 x = buf[j];
          const int pp = page_i * kPage + hh * 8;
          if (pp + 8 > n_pos) {
            uint16_t* e = (uint16_t*)&x;
#pragma unroll
            for (int q = 0; q < 8; ++q)
              if (pp + q >= n_pos) e[q] = 0;
          }
          const int u0 = pp >> 2;  // 8-byte units (4 positions)
          uint2* row = (uint2*)(sV + (size_t)d * CH);
          row[(u0 & ~15) | ((u0 & 15) ^ (d & 15))] = uint2{x.x, x.y};
          row[((u0 + 1) & ~15) | (((u0 + 1) & 15) ^ (d & 15))] = uint2{x.z, x.w};
        }
      }
    }
    __syncthreads();

#pragma unroll
    for (int q = 0; q < 2; ++q) {
      if (!tile_on[q]) continue;
      const int r = tile_row[q];
      const int i = r < R ? r / G : it.k;
      const int lim = it.ctx + i - sub;  // last visible position, sub-chunk-relative
      for (int p0 = 0; p0 < n_pos; p0 += 32) {
        const bool has1 = p0 + 16 < n_pos;
        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
        {
          const int p = p0 + (lane & 15);
#pragma unroll
          for (int kd = 0; kd < DH / 32; ++kd) {
            const int sg = kd * 4 + lg;
            const f16x8 kf = *(const f16x8*)(sK + p * DH + ((sg ^ (p & 15)) & (KSEG - 1)) * 8);
            s0 = mfma_f16(kf, qf[q][kd], s0);
          }
        }
        if (has1) {
          const int p = p0 + 16 + (lane & 15);
#pragma unroll
          for (int kd = 0; kd < DH / 32; ++kd) {
            const int sg = kd * 4 + lg;
            const f16x8 kf = *(const f16x8*)(sK + p * DH + ((sg ^ (p & 15)) & (KSEG - 1)) * 8);
            s1 = mfma_f16(kf, qf[q][kd], s1);
          }
        }
        float sv[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int pa = p0 + lg * 4 + j, pb = pa + 16;
          sv[j] = (pa <= lim && pa < n_pos) ? s0[j] * a.scale_log2 : -INFINITY;
          sv[4 + j] = (pb <= lim && pb < n_pos) ? s1[j] * a.scale_log2 : -INFINITY;
        }
        float bm = sv[0];
#pragma unroll
        for (int j = 1; j < 8; ++j) bm = fmaxf(bm, sv[j]);
        bm = fmaxf(bm, __shfl_xor(bm, 16));
        bm = fmaxf(bm, __shfl_xor(bm, 32));
        const float mn = fmaxf(m[q], bm);
        const float alpha = (m[q] == -INFINITY) ? 0.f : exp2f(m[q] - mn);
        float pv[8];
        float ps = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          pv[j] = (sv[j] == -INFINITY) ? 0.f : exp2f(sv[j] - mn);
          ps += pv[j];
        }
        lsum[q] = lsum[q] * alpha + ps;
        m[q] = mn;
        f16x8 pf;
#pragma unroll
        for (int j = 0; j < 8; ++j) pf[j] = (_Float16)pv[j];
        const int ua = (p0 >> 2) + lg, ub = ua + 4;  // 8-byte units of positions 4lg.. and 16+4lg..
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) {
          o[q][dt] *= alpha;
          const int d = dt * 16 + (lane & 15);
          const uint2* row = (const uint2*)(sV + (size_t)d * CH);
          const uint2 va = row[(ua & ~15) | ((ua & 15) ^ (d & 15))];
          const uint2 vb = has1 ? row[(ub & ~15) | ((ub & 15) ^ (d & 15))] : uint2{0, 0};
          const u32x4 vv = {va.x, va.y, vb.x, vb.y};
          o[q][dt] = mfma_f16(__builtin_bit_cast(f16x8, vv), pf, o[q][dt]);
        }
      }
    }
  }

#pragma unroll
  for (int q = 0; q < 2; ++q) {
    if (!tile_on[q]) continue;
    float l = lsum[q];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int r = tile_row[q];
    const bool rvalid = r < R;
    if (it.nch == 1) {
      if (rvalid) {
        const int i = r / G, h = it.g * G + r % G;
        const float inv = l > 0.f ? 1.f / l : 0.f;
        const int row = it.cu + i;
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) {
          const int col = h * DH + dt * 16 + lg * 4;
          uint16_t hi[4], lo[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) split_bf16(o[q][dt][j] * inv, hi[j], lo[j]);
          const size_t off = afrag_off(row, col, a.MTtot);
          *(uint2*)(a.Ohi + off) = uint2{hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16)};
          *(uint2*)(a.Olo + off) = uint2{lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16)};
        }
      }
    } else {
      const int lr = (wave + 4 * q) * 16 + (lane & 15);
      const size_t slot = (size_t)it.part * 128 + lr;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt)
        *(float4*)(a.part_o + slot * DH + dt * 16 + lg * 4) =
            float4{o[q][dt][0], o[q][dt][1], o[q][dt][2], o[q][dt][3]};
      if (lg == 0) *(float2*)(a.part_ml + slot * 2) = float2{m[q], l};
    }
  }
}

// Merge the chunk partials of one (sequence, kv head, row group) in chunk
// order: O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c.  One block per
// (head entry, 16-row slice); one thread per (row, 8 output dims).
template <int DH>
__global__ __launch_bounds__(256) void attn_combine(CombineArgs a) {
  constexpr int OCT = DH / 8;
  constexpr int RPB = 256 / OCT;  // rows per block
  const AttnItem hd = a.heads[blockIdx.x / (128 / RPB)];
  if (hd.k < 0) return;  // grid padding
  const int slice = blockIdx.x % (128 / RPB);
  const int G = a.group;
  const int R = (hd.k + 1) * G;
  const int lr = slice * RPB + threadIdx.x / OCT, o8 = (threadIdx.x % OCT) * 8;
  const int r = hd.rg * 128 + lr;
  if (r >= R) return;
  const float* ml = a.part_ml + ((size_t)hd.part * 128 + lr) * 2;
  const float* po = a.part_o + ((size_t)hd.part * 128 + lr) * DH + o8;
  const size_t cstride_ml = (size_t)128 * 2, cstride_o = (size_t)128 * DH;
  float M = -INFINITY;
  for (int c = 0; c < hd.nch; ++c) M = fmaxf(M, ml[c * cstride_ml]);
  float L = 0.f, acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll 4
  for (int c = 0; c < hd.nch; ++c) {
    const float mc = ml[c * cstride_ml], lc = ml[c * cstride_ml + 1];
    const float w = (mc == -INFINITY) ? 0.f : exp2f(mc - M);
    L += w * lc;
    const float4 x0 = *(const float4*)(po + c * cstride_o);
    const float4 x1 = *(const float4*)(po + c * cstride_o + 4);
    acc[0] += w * x0.x; acc[1] += w * x0.y; acc[2] += w * x0.z; acc[3] += w * x0.w;
    acc[4] += w * x1.x; acc[5] += w * x1.y; acc[6] += w * x1.z; acc[7] += w * x1.w;
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const int i = r / G, h = hd.g * G + r % G;
  uint16_t hi[8], lo[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) split_bf16(acc[j] * inv, hi[j], lo[j]);
  const size_t off = afrag_off(hd.cu + i, h * DH + o8, a.MTtot);
  *(uint4*)(a.Ohi + off) = uint4{hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16),
                                 hi[4] | ((uint32_t)hi[5] << 16), hi[6] | ((uint32_t)hi[7] << 16)};
  *(uint4*)(a.Olo + off) = uint4{lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16),
                                 lo[4] | ((uint32_t)lo[5] << 16), lo[6] | ((uint32_t)lo[7] << 16)};
}

size_t attn_lds_bytes(int dh) { return (size_t)kAttnChunk * dh * 2 * 2; }

hipError_t launch_attn(const AttnArgs& a, int n_items, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  const size_t lds = attn_lds_bytes(a.dh);
  if (a.dh == 128)
    hipLaunchKernelGGL(verify_attn<128>, dim3(n_items), dim3(256), lds, s, a);
  else if (a.dh == 64)
    hipLaunchKernelGGL(verify_attn<64>, dim3(n_items), dim3(256), lds, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, int n_heads, hipStream_t s) {
  if (n_heads <= 0) return hipSuccess;
  if (a.dh == 128)
    hipLaunchKernelGGL(attn_combine<128>, dim3(n_heads * 8), dim3(256), 0, s, a);
  else if (a.dh == 64)
    hipLaunchKernelGGL(attn_combine<64>, dim3(n_heads * 4), dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t attn_set_lds_limit() {
  hipError_t e = hipFuncSetAttribute((const void*)verify_attn<128>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)attn_lds_bytes(128));
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void*)verify_attn<64>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)attn_lds_bytes(64));
}

}  // namespace hvd
