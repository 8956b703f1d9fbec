// Verify attention over the paged fp16 KV cache (gfx950, MFMA 16x16x32 f16).
//
// For one sequence, the (k+1) query rows of the verify step times the
// Hq/Hkv q-heads of one kv head g form R = (k+1)*group query vectors; row
// r = i*group + hh is draft row i (position ctx+i) of q-head g*group+hh and
// may attend to key positions 0..ctx+i.  A workgroup handles one KV chunk of
// one (sequence, kv head, row group of <= 128 rows).
//
// Scores are computed transposed, S^T = K Q^T, so the fp32 C fragment of a
// lane holds 4 key positions of one query row; the same registers, converted
// to fp16, are the B operand of O^T = V^T P^T with the contraction index
// permuted consistently on both operands (positions {4g..4g+3, 16+4g..16+4g+3}
// for lane group g).  V is stored transposed inside each 16-token page
// ([dh][16]) so that permuted V^T operand is two 8-byte loads per lane.
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
  const AttnItem it = a.items[blockIdx.x];
  const SeqMeta sq = a.seqs[it.b];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int G = a.group;
  const int R = (sq.k + 1) * G;
  const int T = sq.ctx + sq.k + 1;
  const int p_begin = it.c * a.chunk;
  const int p_end = min(T, p_begin + a.chunk);
  const int lg = lane >> 4;
  const int* ptrow = a.pt + (size_t)sq.slot * a.pt_stride;
  const size_t vhalf = (size_t)a.Hkv * kPage * DH;

  for (int tt = wave; tt < 8; tt += 4) {
    const int row_base = it.rg * 128 + tt * 16;
    if (row_base >= R) break;
    const int r = row_base + (lane & 15);
    const bool rvalid = r < R;
    const int i = rvalid ? r / G : sq.k;
    const int h = it.g * G + (rvalid ? r % G : 0);
    const int lim = sq.ctx + i;

    f16x8 qf[DH / 32];
#pragma unroll
    for (int kd = 0; kd < DH / 32; ++kd) {
      if (rvalid)
        qf[kd] = *(const f16x8*)(a.Q + ((size_t)(sq.cu + i) * a.Hq + h) * DH + kd * 32 + lg * 8);
      else
        qf[kd] = f16x8{0, 0, 0, 0, 0, 0, 0, 0};
    }

    float m = -INFINITY, lsum = 0.f;
    f32x4 o[DH / 16];
#pragma unroll
    for (int d = 0; d < DH / 16; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int p0 = p_begin; p0 < p_end; p0 += 32) {
      const int pg0 = ptrow[p0 >> 4];
      const bool has1 = p0 + 16 < p_end;
      const int pg1 = has1 ? ptrow[(p0 >> 4) + 1] : pg0;
      const _Float16* k0p = a.kv + (size_t)pg0 * a.page_stride + (size_t)it.g * kPage * DH;
      const _Float16* k1p = a.kv + (size_t)pg1 * a.page_stride + (size_t)it.g * kPage * DH;
      f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kd = 0; kd < DH / 32; ++kd) {
        f16x8 kf = *(const f16x8*)(k0p + (lane & 15) * DH + kd * 32 + lg * 8);
        s0 = mfma_f16(kf, qf[kd], s0);
      }
      if (has1) {
#pragma unroll
        for (int kd = 0; kd < DH / 32; ++kd) {
          f16x8 kf = *(const f16x8*)(k1p + (lane & 15) * DH + kd * 32 + lg * 8);
          s1 = mfma_f16(kf, qf[kd], s1);
        }
      }
      float sv[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int pa = p0 + lg * 4 + j, pb = pa + 16;
        sv[j] = (pa <= lim && pa < p_end) ? s0[j] * a.scale_log2 : -INFINITY;
        sv[4 + j] = (pb <= lim && pb < p_end) ? s1[j] * a.scale_log2 : -INFINITY;
      }
      float bm = sv[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) bm = fmaxf(bm, sv[j]);
      bm = fmaxf(bm, __shfl_xor(bm, 16));
      bm = fmaxf(bm, __shfl_xor(bm, 32));
      const float mn = fmaxf(m, bm);
      const float alpha = (m == -INFINITY) ? 0.f : exp2f(m - mn);
      float pv[8];
      float ps = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        pv[j] = (sv[j] == -INFINITY) ? 0.f : exp2f(sv[j] - mn);
        ps += pv[j];
      }
      lsum = lsum * alpha + ps;
      m = mn;
      f16x8 pf;
#pragma unroll
      for (int j = 0; j < 8; ++j) pf[j] = (_Float16)pv[j];

      const _Float16* v0p = a.kv + (size_t)pg0 * a.page_stride + vhalf + (size_t)it.g * DH * kPage;
      const _Float16* v1p = a.kv + (size_t)pg1 * a.page_stride + vhalf + (size_t)it.g * DH * kPage;
      const bool tail = p0 + lg * 4 + 3 >= p_end || p0 + 16 + lg * 4 + 3 >= p_end;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt) {
        o[dt] *= alpha;
        const int d = dt * 16 + (lane & 15);
        f16x4 va = *(const f16x4*)(v0p + (size_t)d * kPage + lg * 4);
        f16x4 vb = has1 ? *(const f16x4*)(v1p + (size_t)d * kPage + lg * 4) : f16x4{0, 0, 0, 0};
        if (tail) {  // keys past the end may hold stale values: zero them
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            if (p0 + lg * 4 + j >= p_end) va[j] = 0;
            if (p0 + 16 + lg * 4 + j >= p_end) vb[j] = 0;
          }
        }
        f16x8 vf = {va[0], va[1], va[2], va[3], vb[0], vb[1], vb[2], vb[3]};
        o[dt] = mfma_f16(vf, pf, o[dt]);
      }
    }
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);

    if (it.nch == 1) {
      if (rvalid) {
        const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
        const int row = sq.cu + i;
#pragma unroll
        for (int dt = 0; dt < DH / 16; ++dt) {
          const int col = h * DH + dt * 16 + lg * 4;
          uint16_t hi[4], lo[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) split_bf16(o[dt][j] * inv, hi[j], lo[j]);
          size_t off = afrag_off(row, col, a.MTtot);
          *(uint2*)(a.Ohi + off) = uint2{hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16)};
          *(uint2*)(a.Olo + off) = uint2{lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16)};
        }
      }
    } else {
      const int lr = tt * 16 + (lane & 15);
      const size_t slot = (size_t)it.part * 128 + lr;
#pragma unroll
      for (int dt = 0; dt < DH / 16; ++dt)
        *(float4*)(a.part_o + slot * DH + dt * 16 + lg * 4) = float4{o[dt][0], o[dt][1], o[dt][2], o[dt][3]};
      if (lg == 0) *(float2*)(a.part_ml + slot * 2) = float2{m, lsum};
    }
  }
}

// Merge the chunk partials of one (sequence, kv head, row group) in chunk
// order: O = sum_c 2^(m_c - M) O_c / sum_c 2^(m_c - M) l_c.
template <int DH>
__global__ __launch_bounds__(256) void attn_combine(CombineArgs a) {
  const AttnItem hd = a.heads[blockIdx.x];
  const SeqMeta sq = a.seqs[hd.b];
  const int G = a.group;
  const int R = (sq.k + 1) * G;
  constexpr int OCT = DH / 8;
  for (int e = threadIdx.x; e < 128 * OCT; e += 256) {
    const int lr = e / OCT, o8 = (e % OCT) * 8;
    const int r = hd.rg * 128 + lr;
    if (r >= R) continue;
    float M = -INFINITY;
    for (int c = 0; c < hd.nch; ++c) M = fmaxf(M, a.part_ml[((size_t)(hd.part + c) * 128 + lr) * 2]);
    float L = 0.f, acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int c = 0; c < hd.nch; ++c) {
      const size_t slot = (size_t)(hd.part + c) * 128 + lr;
      const float mc = a.part_ml[slot * 2], lc = a.part_ml[slot * 2 + 1];
      const float w = (mc == -INFINITY) ? 0.f : exp2f(mc - M);
      L += w * lc;
      const float4 x0 = *(const float4*)(a.part_o + slot * DH + o8);
      const float4 x1 = *(const float4*)(a.part_o + slot * DH + o8 + 4);
      acc[0] += w * x0.x; acc[1] += w * x0.y; acc[2] += w * x0.z; acc[3] += w * x0.w;
      acc[4] += w * x1.x; acc[5] += w * x1.y; acc[6] += w * x1.z; acc[7] += w * x1.w;
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const int i = r / G, h = hd.g * G + r % G;
    uint16_t hi[8], lo[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) split_bf16(acc[j] * inv, hi[j], lo[j]);
    const size_t off = afrag_off(sq.cu + i, h * DH + o8, a.MTtot);
    *(uint4*)(a.Ohi + off) = uint4{hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16),
                                   hi[4] | ((uint32_t)hi[5] << 16), hi[6] | ((uint32_t)hi[7] << 16)};
    *(uint4*)(a.Olo + off) = uint4{lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16),
                                   lo[4] | ((uint32_t)lo[5] << 16), lo[6] | ((uint32_t)lo[7] << 16)};
  }
}

hipError_t launch_attn(const AttnArgs& a, int n_items, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  if (a.dh == 128)
    hipLaunchKernelGGL(verify_attn<128>, dim3(n_items), dim3(256), 0, s, a);
  else if (a.dh == 64)
    hipLaunchKernelGGL(verify_attn<64>, dim3(n_items), dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, int n_heads, hipStream_t s) {
  if (n_heads <= 0) return hipSuccess;
  if (a.dh == 128)
    hipLaunchKernelGGL(attn_combine<128>, dim3(n_heads), dim3(256), 0, s, a);
  else if (a.dh == 64)
    hipLaunchKernelGGL(attn_combine<64>, dim3(n_heads), dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace hvd
