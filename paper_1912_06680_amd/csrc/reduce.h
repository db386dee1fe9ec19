// Deterministic column reductions (fixed summation order, no atomics).
#pragma once

#include "common.h"

namespace o5 {

// part[c, n] = sum of src[r, n] over rows r in chunk c = [c*rows_per_chunk, ...).
static __global__ void __launch_bounds__(256) colsum_chunks(int R, int N, int rows_per_chunk, const float* __restrict__ src,
                                                           float* __restrict__ part) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  const int r0 = blockIdx.y * rows_per_chunk;
  const int r1 = min(R, r0 + rows_per_chunk);
  float s = 0.0f;
  for (int r = r0; r < r1; ++r) s += src[static_cast<size_t>(r) * N + n];
  part[static_cast<size_t>(blockIdx.y) * N + n] = s;
}

// out[n] = sum over the P rows of part (fixed order).
static __global__ void __launch_bounds__(256) colsum_rows(int P, int N, const float* __restrict__ part, float* __restrict__ out) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  float s = 0.0f;
  for (int p = 0; p < P; ++p) s += part[static_cast<size_t>(p) * N + n];
  out[n] = s;
}

// out[n] = sum over the P rows of part, one block of 256 threads per column:
// thread t sums rows t, t + 256, ... in order, then a fixed-shape tree in LDS.
// For short columns of many rows (where one thread per column would walk all
// P rows alone).
static __global__ void __launch_bounds__(256) colsum_tree(int P, int N, const float* __restrict__ part,
                                                        float* __restrict__ out) {
  __shared__ float red[256];
  const int n = blockIdx.x;
  float s = 0.0f;
  for (int p = threadIdx.x; p < P; p += 256) s += part[static_cast<size_t>(p) * N + n];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[n] = red[0];
}

}  // namespace o5
