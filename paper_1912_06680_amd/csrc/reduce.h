// Deterministic column reductions (fixed summation order, no atomics).
#pragma once

#include "common.h"

namespace o5 {

// at(0) + at(1) + ... + at(n - 1), added in that order onto 0; the terms'
// loads are issued eight at a time before their adds, so a run of eight
// waits on memory once.
template <class F>
__device__ __forceinline__ float ordered_sum(int n, F&& at) {
  float s = 0.0f;
  int p = 0;
  for (; p + 8 <= n; p += 8) {
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = at(p + q);
#pragma unroll
    for (int q = 0; q < 8; ++q) s += v[q];
  }
  for (; p < n; ++p) s += at(p);
  return s;
}

// part[c, n] = sum of src[r, n] over rows r in chunk c = [c*rows_per_chunk, ...).
static __global__ void __launch_bounds__(256) colsum_chunks(int R, int N, int rows_per_chunk, const float* __restrict__ src,
                                                           float* __restrict__ part) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  const int r0 = blockIdx.y * rows_per_chunk;
  const int r1 = min(R, r0 + rows_per_chunk);
  const float* col = src + static_cast<size_t>(r0) * N + n;
  part[static_cast<size_t>(blockIdx.y) * N + n] =
      ordered_sum(r1 - r0, [&](int i) { return col[static_cast<size_t>(i) * N]; });
}

// out[n] = sum over the P rows of part (fixed order).
static __global__ void __launch_bounds__(256) colsum_rows(int P, int N, const float* __restrict__ part, float* __restrict__ out) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  out[n] = ordered_sum(P, [&](int p) { return part[static_cast<size_t>(p) * N + n]; });
}

// out[n] = sum over the P rows of part for many rows and few columns: a
// block takes 64 columns; its 4 waves sum rows g, g + 4, g + 8, ... (g the
// wave), each in order, and the 4 sums are added in the order g = 0..3.
// Launch with cdiv(N, 64) blocks of 256 threads.
static __global__ void __launch_bounds__(256) colsum_rows4(int P, int N, const float* __restrict__ part,
                                                          float* __restrict__ out) {
  __shared__ float red[4][64];
  const int c = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + c;
  float s = 0.0f;
  if (n < N)
    s = ordered_sum((P - g + 3) / 4, [&](int i) { return part[static_cast<size_t>(g + 4 * i) * N + n]; });
  red[g][c] = s;
  __syncthreads();
  if (g == 0 && n < N) out[n] = ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
}

// out[n] = sum over the P rows of part, one block of 256 threads per column:
// thread t sums rows t, t + 256, ... in order, then a fixed-shape tree in LDS.
// For short columns of many rows (where one thread per column would walk all
// P rows alone).
static __global__ void __launch_bounds__(256) colsum_tree(int P, int N, const float* __restrict__ part,
                                                        float* __restrict__ out) {
  __shared__ float red[256];
  const int n = blockIdx.x;
  const int t = threadIdx.x;
  red[t] = ordered_sum((P - t + 255) / 256, [&](int i) { return part[static_cast<size_t>(t + 256 * i) * N + n]; });
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  if (t == 0) out[n] = red[0];
}

// ------------------------------------------------------ wave reductions

// v combined with the value DPP control CTRL moves into each lane; lanes of
// rows outside ROW_MASK take `id` instead.
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ float dpp(float id, float v) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(id), __float_as_int(v), CTRL, ROW_MASK, 0xf, false));
}

// Wave-wide reduction on the VALU's data-parallel lane moves: two quad
// swaps and two rotations within each row of 16 lanes leave every lane with
// its row's total, two row broadcasts carry them to lane 63, whose value is
// returned to every lane.  A fixed combination order, so the result is the
// same from call to call.
template <class Op>
__device__ __forceinline__ float wave_reduce(float v, float id, Op op) {
  v = op(v, dpp<0xB1>(id, v));        // quad_perm [1, 0, 3, 2]
  v = op(v, dpp<0x4E>(id, v));        // quad_perm [2, 3, 0, 1]
  v = op(v, dpp<0x124>(id, v));       // row_ror 4
  v = op(v, dpp<0x128>(id, v));       // row_ror 8
  v = op(v, dpp<0x142, 0xa>(id, v));  // row_bcast 15: rows 1 and 3 add rows 0 and 2
  v = op(v, dpp<0x143, 0xc>(id, v));  // row_bcast 31: rows 2 and 3 add rows 0 + 1
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
__device__ __forceinline__ float wave_max(float v) {
  return wave_reduce(v, -INFINITY, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ float wave_sum(float v) {
  return wave_reduce(v, 0.0f, [](float a, float b) { return a + b; });
}

// Column c (the same in every lane) of the row, held by lane c % 64 as its
// element c / 64.
template <int CPL>
__device__ __forceinline__ float column(const float (&z)[CPL], int c) {
  float v = z[0];
#pragma unroll
  for (int i = 1; i < CPL; ++i)
    if (c >> 6 == i) v = z[i];
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), c & 63));
}

}  // namespace o5
