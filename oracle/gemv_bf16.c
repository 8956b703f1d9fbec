/*
 * TEST INFRASTRUCTURE ONLY (part of the CPU oracle; the GPU library never
 * links or calls it).
 *
 * y[m][n] = sum_k x[m][k] * w(n, k) for bf16 weights w given as bit patterns
 * W[n][k] (torch Linear layout [out, in], row-major) and float32 inputs x.
 *
 * This is the plain matrix product that the oracle's decoder forward takes
 * for every linear layer (Q/K/V/O projections, SwiGLU gate/up/down, LM head).
 * It exists only so that a model too large to hold in float32 on the host can
 * keep its weights as bf16 bits: each weight is widened exactly (bf16 -> fp32
 * is a 16-bit left shift of the bit pattern) and multiplied in float32 with a
 * float32 sum over k, in ascending k order within 16 interleaved partial
 * sums.  No blocking over k beyond that, no reordering of rows.
 *
 * Threads split the output columns n; every y[m][n] is computed by one thread
 * alone, so the result does not depend on the thread count.
 */
#include <stddef.h>
#include <stdint.h>
#include <string.h>

static inline float bf16_to_f32(uint16_t b) {
  uint32_t u = ((uint32_t)b) << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

void oracle_gemv_bf16(const float* x, int64_t M, const uint16_t* W, int64_t N, int64_t K, float* y) {
#pragma omp parallel
  {
    float* wrow = NULL;
    /* per-thread widened weight row (K floats) */
    float stack_row[16384];
    float* heap_row = NULL;
    if (K <= 16384) {
      wrow = stack_row;
    } else {
      heap_row = (float*)__builtin_malloc((size_t)K * sizeof(float));
      wrow = heap_row;
    }
#pragma omp for schedule(static)
    for (int64_t n = 0; n < N; ++n) {
      const uint16_t* wn = W + n * K;
      for (int64_t k = 0; k < K; ++k) wrow[k] = bf16_to_f32(wn[k]);
      for (int64_t m = 0; m < M; ++m) {
        const float* xm = x + m * K;
        float part[16] = {0};
        int64_t k = 0;
        for (; k + 16 <= K; k += 16)
          for (int j = 0; j < 16; ++j) part[j] += xm[k + j] * wrow[k + j];
        for (; k < K; ++k) part[k & 15] += xm[k] * wrow[k];
        float s = 0.f;
        for (int j = 0; j < 16; ++j) s += part[j];
        y[m * N + n] = s;
      }
    }
    if (heap_row) __builtin_free(heap_row);
  }
}
