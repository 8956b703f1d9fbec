// Small kernels of the verify step: weight packing (load time), embedding
// gather with the first RMSNorm's operand, and the fused argmax finalize +
// greedy accept.
#include "common.h"
#include <algorithm>

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
  for (int u = blockIdx.x * 256 + threadIdx.x; u < a.n_zero; u += gridDim.x * 256) a.zero[u] = 0u;
  const int R = blockIdx.x;
  const bool valid = R < a.M;
  int tok = valid ? a.rows[R].tok : 0;
  if ((unsigned)tok >= (unsigned)a.V) tok = 0;  // only a device-side drafter can pass one
  const uint16_t* er = valid ? a.E + (size_t)tok * a.D : nullptr;
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
  const int step = a.astate ? a.astate[2 * a.B] : 0;
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
    const int nxt = __atomic_load_n(&a.g[sq.cu + last], __ATOMIC_RELAXED);
    a.out[2 * b] = acc;
    a.out[2 * b + 1] = nxt;
    if (a.astate) {  // device-resident loop: commit the whole accepted block
      a.astate[b] += acc + 1;
      a.astate[a.B + b] = nxt;
      if (step < a.hist_cap) {
        a.hist[((size_t)step * a.B + b) * 2] = acc;
        a.hist[((size_t)step * a.B + b) * 2 + 1] = nxt;
      }
    }
  }
  __syncthreads();  // every thread has read the step count
  if (threadIdx.x == 0) {
    if (a.err_word) a.out[a.err_index] = (int32_t)*a.err_word;
    *a.counter = 0u;
    if (a.astate) a.astate[2 * a.B] = step + 1;
  }
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

// One workgroup: rows (token, position, pool slot), sequences (ctx) and the
// attention items and combine entries of this step of a device-resident
// loop.  Row i of sequence b is token pending[b] (i = 0) or draft i - 1, at
// position ctx[b] + i.  With the copy drafter, draft token i - 1 is the
// stream token at that position (-1 outside the stream: never accepted) and
// is also stored to the draft buffer.  Page indexes past a sequence's
// reserved list are clamped into it (the host reserves enough, so this only
// keeps a broken caller from faulting).
__global__ __launch_bounds__(512) void async_plan(AsyncPlanArgs a) {
  for (int r = threadIdx.x; r < a.M; r += blockDim.x) {
    const int b = a.row_seq[r];
    const SeqMeta sq = a.seq_static[b];
    const int ctx = a.state[b];
    const int i = r - sq.cu;
    int tok;
    if (i == 0) {
      tok = a.state[a.B + b];
    } else {
      const int d = sq.cu - b + i - 1;
      if (a.ref) {
        const int j = ctx + i - a.ref_start[b];
        tok = (j >= 0 && j < a.ref_len) ? a.ref[(size_t)b * a.ref_len + j] : -1;
        a.drafts[d] = tok;
      } else {
        tok = a.drafts[d];
      }
    }
    const int pos = ctx + i;
    const int p0 = a.page_off[b], np = a.page_off[b + 1] - p0;
    const int pi = min(pos / kPage, np - 1);
    a.rows[r] = RowMeta{tok, sq.slot, pos, a.pages[p0 + pi] * kPage + pos % kPage};
  }
  for (int b = threadIdx.x; b < a.B; b += blockDim.x) {
    SeqMeta sq = a.seq_static[b];
    sq.ctx = a.state[b];
    a.seqs[b] = sq;
  }
  // items: the live chunks of the unit at the current ctx
  for (int n = threadIdx.x; n < a.n_items + a.n_heads; n += blockDim.x) {
    const bool head = n >= a.n_items;
    const int e = head ? n - a.n_items : n;
    AttnItem it = head ? a.heads_static[e] : a.items_static[e];
    if (it.k >= 0) {
      const int ctx = a.state[it.pad1];
      const int nch = (ctx + it.pad2 + 1 + it.pad3 - 1) / it.pad3;  // pad3: the plan's chunk length
      if (head ? nch == 1 : it.c >= nch) {
        it.k = -1;  // no keys yet (item), or the only chunk writes O itself (combine entry)
      } else {
        it.ctx = ctx;
        it.nch = nch;
        it.p_end = min(ctx + it.k + 1, it.p_begin + it.pad3);
      }
    }
    if (head) a.heads[e] = it;
    else a.items[e] = it;
  }
}

// Page-table updates applied on their own (before a device-resident loop's
// captured steps, which then carry none).
__global__ __launch_bounds__(256) void pt_update(const int32_t* upd, const int32_t* n_upd, int32_t* pt, int pt_stride) {
  for (int u = threadIdx.x, n = *n_upd; u < n; u += blockDim.x)
    pt[(size_t)upd[u * 3] * pt_stride + upd[u * 3 + 1]] = upd[u * 3 + 2];
}

hipError_t launch_pt_update(const int32_t* upd, const int32_t* n_upd, int32_t* pt, int pt_stride, hipStream_t s) {
  hvd_launch(pt_update, dim3(1), dim3(256), 0, s, upd, n_upd, pt, pt_stride);
  return hipGetLastError();
}

// The step's metadata from pinned host memory into device memory, read by
// a kernel (16 bytes per lane): it starts a few microseconds after launch,
// where a DMA copy first waits for its copy engine.
__global__ __launch_bounds__(256) void copy_words(int32_t* __restrict__ dst, const int32_t* __restrict__ src, int n) {
  const int q = n >> 2;  // whole 16-byte units
  for (int i = blockIdx.x * 256 + threadIdx.x; i < q; i += gridDim.x * 256)
    ((uint4*)dst)[i] = ((const uint4*)src)[i];
  for (int i = 4 * q + blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) dst[i] = src[i];
}

hipError_t launch_copy_words(int32_t* dst, const int32_t* src, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (n > (size_t)INT32_MAX || ((uintptr_t)dst & 15) || ((uintptr_t)src & 15)) return hipErrorInvalidValue;
  const int blocks = (int)std::min<size_t>(64, (n / 4 + 255) / 256 + 1);
  hvd_launch(copy_words, dim3(blocks), dim3(256), 0, s, dst, src, (int)n);
  return hipGetLastError();
}

hipError_t launch_async_plan(const AsyncPlanArgs& a, hipStream_t s) {
  hvd_launch(async_plan, dim3(1), dim3(512), 0, s, a);
  return hipGetLastError();
}

}  // namespace hvd
