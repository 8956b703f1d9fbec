// Small kernels of the verify step: weight packing (load time), embedding
// gather with the first RMSNorm's operand, and the fused argmax finalize +
// greedy accept.
#include "common.h"
#include "kernels.h"

namespace hvd {

thread_local LaunchTiming tl_timing;

// dst fragment (strip s, K step kt), lane l, half j =
//   fp16(src[rowmap[16 s + l%16]][32 kt + 8 (l/16) + j])   (src bf16)
// stored at ((s/4 * KT + kt) * 4 + s%4) * 512 halves: the 4 strips of a
// 64-column block are contiguous for each K step.
__global__ void pack_weight(const uint16_t* __restrict__ src, const int32_t* __restrict__ rowmap,
                            uint16_t* __restrict__ dst, int N, int K) {
  const int KT = K >> 5;
  const size_t total = (size_t)(N >> 4) * KT * 64;
  for (size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (size_t)gridDim.x * blockDim.x) {
    const int l = (int)(t & 63);
    const size_t frag = t >> 6;           // in destination order
    const int ns = (int)(frag & 3);
    const int kt = (int)((frag >> 2) % KT);
    const int cb = (int)((frag >> 2) / KT);
    const int s = cb * 4 + ns;
    const int srow = rowmap[s * 16 + (l & 15)];
    // bf16 -> fp16: exact except magnitudes below 2^-17 (fp16 subnormals),
    // whose rounding error is below 2^-25
    const uint4 v = *(const uint4*)(src + (size_t)srow * K + kt * 32 + (l >> 4) * 8);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t h[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      h[j] = (uint32_t)f2h(bf2f((uint16_t)(w[j] & 0xFFFFu))) | ((uint32_t)f2h(bf2f((uint16_t)(w[j] >> 16))) << 16);
    *(uint4*)(dst + t * 8) = uint4{h[0], h[1], h[2], h[3]};
  }
}

hipError_t launch_pack(const uint16_t* src, const int32_t* rowmap, uint16_t* dst, int N, int K, hipStream_t s) {
  size_t total = (size_t)(N / 16) * (K / 32) * 64;
  int blocks = (int)((total + 255) / 256);
  if (blocks > 65535 * 8) blocks = 65535 * 8;
  hvd_launch(pack_weight, dim3(blocks), dim3(256), 0, s, src, rowmap, dst, N, K);
  return hipGetLastError();
}

// One block per (padded) row: X = fp32(E[tok]), the first norm's operand
// fp16 hi/lo split of X * gain, per-16-column sums of squares.  Block 0 first
// applies this step's page-table updates.
__global__ __launch_bounds__(256) void embed_rows(EmbedArgs a) {
  if (blockIdx.x == 0)
    for (int u = threadIdx.x, n = *a.n_upd; u < n; u += blockDim.x)
      a.pt[(size_t)a.upd[u * 3] * a.pt_stride + a.upd[u * 3 + 1]] = a.upd[u * 3 + 2];
  const int R = blockIdx.x;
  const bool valid = R < a.M;
  const uint16_t* er = valid ? a.E + (size_t)a.rows[R].tok * a.D : nullptr;
  const int noct = a.D >> 3;
  for (int base = 0; base < noct; base += 256) {
    const int o = base + threadIdx.x;
    const bool ok = o < noct;
    float x[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (ok && valid) {
      const uint4 v = *(const uint4*)(er + o * 8);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[2 * j] = __uint_as_float(w[j] << 16);
        x[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
      }
    }
    float sq = 0.f;
    if (ok) {
      const int C = o * 8;
      float* xp = a.X + (size_t)R * a.D + C;
      *(float4*)xp = float4{x[0], x[1], x[2], x[3]};
      *(float4*)(xp + 4) = float4{x[4], x[5], x[6], x[7]};
      uint16_t hi[8], lo[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        sq += x[j] * x[j];
        split_f16(x[j] * a.gain[C + j], hi[j], lo[j]);
      }
      const size_t off = afrag_off(R, C, a.MTtot);
      *(uint4*)(a.Nhi + off) = uint4{hi[0] | ((uint32_t)hi[1] << 16), hi[2] | ((uint32_t)hi[3] << 16),
                                     hi[4] | ((uint32_t)hi[5] << 16), hi[6] | ((uint32_t)hi[7] << 16)};
      *(uint4*)(a.Nlo + off) = uint4{lo[0] | ((uint32_t)lo[1] << 16), lo[2] | ((uint32_t)lo[3] << 16),
                                     lo[4] | ((uint32_t)lo[5] << 16), lo[6] | ((uint32_t)lo[7] << 16)};
    }
    const float other = __shfl_xor(sq, 1);
    if (ok && (o & 1) == 0) a.ss_out[(size_t)R * (a.D >> 4) + (o >> 1)] = sq + other;
  }
}

hipError_t launch_embed(const EmbedArgs& a, hipStream_t s) {
  hvd_launch(embed_rows, dim3(a.Mpad), dim3(256), 0, s, a);
  return hipGetLastError();
}

// One block per row: reduce the LM head's per-block (max, lowest argmax)
// partials to the row argmax g[r] (ties -> lowest token id).  The last block
// to finish applies the accept rule to every sequence: a = number of leading
// draft tokens equal to the target argmax of the row before them, next =
// argmax of row a.  It then resets the arrival counter.
__global__ __launch_bounds__(256) void argmax_accept(AcceptArgs a) {
  const int r = blockIdx.x;
  const float* pv = a.part_val + (size_t)r * a.n_part;
  const int32_t* pi = a.part_idx + (size_t)r * a.n_part;
  float best = -INFINITY;
  int bidx = 0x7fffffff;
  for (int j = threadIdx.x; j < a.n_part; j += 256) {
    const float v = pv[j];
    const int id = pi[j];
    if (v > best || (v == best && id < bidx)) { best = v; bidx = id; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(best, o);
    const int oi = __shfl_xor(bidx, o);
    if (ov > best || (ov == best && oi < bidx)) { best = ov; bidx = oi; }
  }
  __shared__ float sv[4];
  __shared__ int si[4];
  __shared__ bool last;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) { sv[wave] = best; si[wave] = bidx; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w)
      if (sv[w] > best || (sv[w] == best && si[w] < bidx)) { best = sv[w]; bidx = si[w]; }
    a.g[r] = bidx;
    __threadfence();
    const unsigned prev = atomicAdd(a.counter, 1u);
    last = (prev == (unsigned)a.M - 1);
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  for (int b = threadIdx.x; b < a.B; b += 256) {
    const SeqMeta sq = a.seqs[b];
    int acc = 0, last = 0;  // accepted count; row of the last accepted token
    if (!sq.tree) {
      while (acc < sq.k) {
        const int drafted = a.rows[sq.cu + acc + 1].tok;  // draft token acc
        const int target = __atomic_load_n(&a.g[sq.cu + acc], __ATOMIC_RELAXED);
        if (drafted != target) break;
        ++acc;
      }
      last = acc;
    } else {
      // from the pending token, move to the child (lowest node index) whose
      // token is the target's argmax of the current row, while one exists
      int cur = -1;
      for (;;) {
        const int target = __atomic_load_n(&a.g[sq.cu + cur + 1], __ATOMIC_RELAXED);
        int nxt = -1;
        for (int j = cur + 1; j < sq.k; ++j)  // children come after their parent
          if (a.tree_parent[sq.cu + 1 + j] == cur && a.rows[sq.cu + 1 + j].tok == target) {
            nxt = j;
            break;
          }
        if (nxt < 0) break;
        a.path[b * kMaxTreeNodes + acc] = nxt;
        ++acc;
        cur = nxt;
      }
      last = cur + 1;
    }
    a.out[2 * b] = acc;
    a.out[2 * b + 1] = __atomic_load_n(&a.g[sq.cu + last], __ATOMIC_RELAXED);
  }
  if (threadIdx.x == 0) *a.counter = 0u;
}

// After a tree verify: the accepted path's K/V moves from the nodes'
// positions ctx + 1 + node to the chain positions ctx + 1 .. ctx + a, so a
// commit keeps a prefix exactly as for a chain.  One block per (sequence,
// layer); each thread owns fixed (kv head, dims) across all positions and
// moves them in path order (target ctx + d never holds a later source:
// nodes follow their parents, so path node d - 1 has index >= d - 1).
__global__ __launch_bounds__(256) void tree_compact(CompactArgs a) {
  const int b = blockIdx.x, l = blockIdx.y;
  const SeqMeta sq = a.seqs[b];
  if (!sq.tree) return;
  const int acc = a.out[2 * b];
  const int32_t* ptrow = a.pt + (size_t)sq.slot * a.pt_stride;
  _Float16* lay = a.pool + (size_t)l * a.layer_stride;
  const size_t vhalf = (size_t)a.Hkv * kPage * a.dh;
  const int n_k = a.Hkv * a.dh / 8;  // 16-byte K units (8 dims) per position
  const int n_v = a.Hkv * a.dh;      // V elements per position
  for (int d = 1; d <= acc; ++d) {
    const int src = sq.ctx + 1 + a.path[b * kMaxTreeNodes + d - 1], dst = sq.ctx + d;
    if (src == dst) continue;
    const size_t ps = (size_t)ptrow[src / kPage] * a.page_stride, pd = (size_t)ptrow[dst / kPage] * a.page_stride;
    const int ts = src % kPage, td = dst % kPage;
    for (int u = threadIdx.x; u < n_k; u += 256) {
      const int g = u / (a.dh / 8), c8 = (u % (a.dh / 8)) * 8;
      *(uint4*)(lay + pd + ((size_t)g * kPage + td) * a.dh + c8) =
          *(const uint4*)(lay + ps + ((size_t)g * kPage + ts) * a.dh + c8);
    }
    for (int e = threadIdx.x; e < n_v; e += 256)  // V is [kv head][dim][16 positions] in a page
      lay[pd + vhalf + (size_t)e * kPage + td] = lay[ps + vhalf + (size_t)e * kPage + ts];
  }
}

hipError_t launch_compact(const CompactArgs& a, int B, hipStream_t s) {
  hvd_launch(tree_compact, dim3(B, a.n_layers), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs& a, hipStream_t s) {
  hvd_launch(argmax_accept, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace hvd
