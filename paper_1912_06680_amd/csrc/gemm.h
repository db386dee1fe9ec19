// GEMM engines of libo5:  C[i, j] = sum_k A(i, k) * B(j, k)  (+ epilogue).
//
// Operands are described by small loader structs instead of raw pointers so
// that one engine serves every contraction of the LSTM step:
//   forward  G_t   = [x_t | h~_{t-1}] . [W_x | W_h]^T      (A, B K-contiguous)
//   backward dh    = dG_t . W_h                             (B I-contiguous)
//   weights  dW    = dG^T . [x | h~_prev]                   (A, B I-contiguous)
//   input    dx    = dG . W_x                               (B I-contiguous)
// A loader reports whether its reduction index k is the contiguous one
// (kKMajor) and hands out elements (fp32 engine) or 8-element 16-byte
// vectors (bf16 MFMA engine), returning zeros outside the matrix.
//
// bf16 engine (gfx950 MFMA, v_mfma_f32_32x32x16_bf16, fp32 accumulate):
//  * block tile BM x BN, K tile 64, waves arranged (BM/WM) x (BN/WN), each
//    wave owning WM x WN = (WM/32) x (WN/32) MFMA blocks;
//  * both tiles staged in LDS as [row][64 k] bf16, double buffered, with the
//    16-byte chunk index XOR-swizzled by (row >> 1) & 7 so that the 16 lanes
//    of a fragment read (16 consecutive rows, same chunk) hit 16 distinct
//    16-byte bank groups;
//  * operands whose contiguous index is not k are loaded as 8x8 blocks and
//    transposed in registers (v_perm) before the LDS store, so the MFMA
//    fragment reads are always single 16-byte LDS reads;
//  * global loads of tile kt+1 are in flight while tile kt is multiplied;
//  * tiles are numbered so that the M-tiles sharing one B tile run
//    back-to-back on one XCD (blocks are dealt round-robin to the 8 XCDs),
//    which keeps the weight tile in that XCD's L2;
//  * optional split-K over gridDim.z; split z writes its partial sums to
//    its own slice (the caller reduces the slices in a fixed order).
#pragma once

#include "common.h"

namespace o5 {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// ------------------------------------------------------------------ loaders

// (i, k) -> K-contiguous rows, two segments along k: k < K0 reads p0[i*ld0 + k],
// k >= K0 reads p1[i*ld1 + k - K0].  A nonzero mask1[i] zeroes the p1 part
// of row i (the reset of the carried LSTM state).
template <typename E>
struct KRows2 {
  static constexpr bool kKMajor = true;
  const E* p0;
  const E* p1;
  const uint8_t* mask1;
  int ld0, ld1, K0, K, rows;

  __device__ __forceinline__ float at(int i, int k) const {
    if (i >= rows || k >= K) return 0.0f;
    if (k < K0) return elem<E>::to_f32(p0[static_cast<size_t>(i) * ld0 + k]);
    if (mask1 && mask1[i]) return 0.0f;
    return elem<E>::to_f32(p1[static_cast<size_t>(i) * ld1 + (k - K0)]);
  }
  // 8 consecutive k starting at k (k % 8 == 0, K0 % 8 == 0); bf16 only
  __device__ __forceinline__ uint4 vec(int i, int k) const {
    if (i >= rows || k >= K) return make_uint4(0, 0, 0, 0);
    if (k < K0) return *reinterpret_cast<const uint4*>(p0 + static_cast<size_t>(i) * ld0 + k);
    if (mask1 && mask1[i]) return make_uint4(0, 0, 0, 0);
    return *reinterpret_cast<const uint4*>(p1 + static_cast<size_t>(i) * ld1 + (k - K0));
  }
};

// (i, k) -> I-contiguous rows indexed by k, two segments along i:
//   i < I0 : p0[k*ld0 + i]
//   i >= I0: row k of the second source, column i - I0, where row k lives at
//            (k < kswitch ? p1a + k*ld1 : p1b + (k - kswitch)*ld1), zeroed when
//            mask1[k] != 0.
// This expresses [x | h~_prev] over the flattened (t, b) rows, where the
// previous hidden state of row (t, b) is h0[b] for t = 0 and h[t-1, b] after.
template <typename E>
struct ICols2 {
  static constexpr bool kKMajor = false;
  const E* p0;
  const E* p1a;
  const E* p1b;
  const uint8_t* mask1;
  int ld0, ld1, I0, I, K, kswitch;

  __device__ __forceinline__ const E* row1(int k) const {
    return k < kswitch ? p1a + static_cast<size_t>(k) * ld1 : p1b + static_cast<size_t>(k - kswitch) * ld1;
  }
  __device__ __forceinline__ float at(int i, int k) const {
    if (i >= I || k >= K) return 0.0f;
    if (i < I0) return elem<E>::to_f32(p0[static_cast<size_t>(k) * ld0 + i]);
    if (mask1 && mask1[k]) return 0.0f;
    return elem<E>::to_f32(row1(k)[i - I0]);
  }
  // 8 consecutive i starting at i (i % 8 == 0, I0 % 8 == 0); bf16 only
  __device__ __forceinline__ uint4 vec(int i, int k) const {
    if (i >= I || k >= K) return make_uint4(0, 0, 0, 0);
    if (i < I0) return *reinterpret_cast<const uint4*>(p0 + static_cast<size_t>(k) * ld0 + i);
    if (mask1 && mask1[k]) return make_uint4(0, 0, 0, 0);
    return *reinterpret_cast<const uint4*>(row1(k) + (i - I0));
  }
};

// ------------------------------------------------------------ epilogues

// Plain fp32 store of C (row-major, ldc) into slice `split` of a stack of
// M x N partial results (slice stride = sstride elements).
struct EpiStoreF32 {
  float* c;
  int ldc;
  size_t sstride;
  __device__ __forceinline__ void operator()(int i, int j, float v, int split) const {
    c[split * sstride + static_cast<size_t>(i) * ldc + j] = v;
  }
};

// Store into one of two fp32 matrices split by column: j < J0 -> c0[i*ld0 + j],
// else c1[i*ld1 + j - J0]  (dW = [dW_x | dW_h]).
struct EpiStoreF32Split2 {
  float* c0;
  float* c1;
  int ld0, ld1, J0;
  __device__ __forceinline__ void operator()(int i, int j, float v, int) const {
    if (j < J0)
      c0[static_cast<size_t>(i) * ld0 + j] = v;
    else
      c1[static_cast<size_t>(i) * ld1 + (j - J0)] = v;
  }
};

// Store converted to the element type E (dx in the GEMM input type).
template <typename E>
struct EpiStoreElem {
  E* c;
  int ldc;
  __device__ __forceinline__ void operator()(int i, int j, float v, int) const {
    c[static_cast<size_t>(i) * ldc + j] = elem<E>::from_f32(v);
  }
};

// ------------------------------------------------------ fp32 FMA engine
// 64 x 64 tile, K tile 16, 256 threads, 4 x 4 outputs per thread.
// Used for the fp32 path, where exactness matters more than speed.
template <class AL, class BL, class Epi>
__global__ void __launch_bounds__(256) gemm_f32_fma(AL al, BL bl, Epi epi, int M, int N, int K, int ktiles_per_split) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int split = blockIdx.z;
  const int nkt = (K + BK - 1) / BK;
  const int kt0 = split * ktiles_per_split;
  const int kt1 = min(nkt, kt0 + ktiles_per_split);
  float acc[4][4] = {};
  for (int kt = kt0; kt < kt1; ++kt) {
    const int k0 = kt * BK;
    // 64 x 16 elements per operand, 4 per thread; the contiguous index varies fastest
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + u * 256;
      int i, k;
      if (AL::kKMajor) { i = e / BK; k = e % BK; } else { k = e / BM; i = e % BM; }
      As[k][i] = al.at(m0 + i, k0 + k);
      if (BL::kKMajor) { i = e / BK; k = e % BK; } else { k = e / BN; i = e % BN; }
      Bs[k][i] = bl.at(n0 + i, k0 + k);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BK; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) a[r] = As[k][ty + 16 * r];
#pragma unroll
      for (int r = 0; r < 4; ++r) b[r] = Bs[k][tx + 16 * r];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int s = 0; s < 4; ++s) acc[r][s] = fmaf(a[r], b[s], acc[r][s]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int i = m0 + ty + 16 * r, j = n0 + tx + 16 * s;
      if (i < M && j < N) epi(i, j, acc[r][s], split);
    }
}

// ------------------------------------------------------ bf16 MFMA engine

// LDS byte offset of 16-byte chunk `chunk` (0..7) of tile row `row`
// (a row is 64 bf16 = 128 bytes).
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4);
}

// Transpose an 8 x 8 block of 16-bit values held as 8 rows of 4 dwords:
// in[r] = elements (r, 0..7) -> out[c] = elements (0..7, c).
__device__ __forceinline__ void transpose8x8_b16(const uint4 (&in)[8], uint4 (&out)[8]) {
  // v_perm_b32(hi_src, lo_src, sel): bytes 0-3 from lo_src, 4-7 from hi_src
  const uint32_t kLo = 0x05040100u;  // (lo.lo16, hi.lo16)
  const uint32_t kHi = 0x07060302u;  // (lo.hi16, hi.hi16)
#pragma unroll
  for (int c2 = 0; c2 < 4; ++c2) {  // pair of output columns 2*c2, 2*c2+1
    uint32_t w[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const uint4 v = in[r];
      w[r] = c2 == 0 ? v.x : c2 == 1 ? v.y : c2 == 2 ? v.z : v.w;
    }
    uint4 lo, hi;
    lo.x = __builtin_amdgcn_perm(w[1], w[0], kLo);
    lo.y = __builtin_amdgcn_perm(w[3], w[2], kLo);
    lo.z = __builtin_amdgcn_perm(w[5], w[4], kLo);
    lo.w = __builtin_amdgcn_perm(w[7], w[6], kLo);
    hi.x = __builtin_amdgcn_perm(w[1], w[0], kHi);
    hi.y = __builtin_amdgcn_perm(w[3], w[2], kHi);
    hi.z = __builtin_amdgcn_perm(w[5], w[4], kHi);
    hi.w = __builtin_amdgcn_perm(w[7], w[6], kHi);
    out[2 * c2] = lo;
    out[2 * c2 + 1] = hi;
  }
}

template <int ROWS, int NT, class L>
struct TileLoader {
  // K-major: ROWS rows x 8 chunks of 8 k = ROWS*8 vectors, kPer per thread.
  // I-major: (ROWS/8) x 8 blocks of 8 i x 8 k = ROWS blocks, kPer per thread
  // (threads past the last block idle when ROWS < NT).
  static constexpr int kItems = L::kKMajor ? ROWS * 8 : ROWS;
  static constexpr int kPer = kItems >= NT ? kItems / NT : 1;
  static constexpr int kVecs = L::kKMajor ? kPer : kPer * 8;
  static_assert(kItems >= NT ? kItems % NT == 0 : NT % kItems == 0, "tile/threads mismatch");
  uint4 r[kVecs];

  __device__ __forceinline__ bool active(int item) const { return kItems >= NT || item < kItems; }

  __device__ __forceinline__ void load(const L& l, int row0, int k0, int tid) {
    if constexpr (L::kKMajor) {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int v = tid + u * NT;
        if (active(v)) r[u] = l.vec(row0 + (v >> 3), k0 + ((v & 7) << 3));
      }
    } else {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int blk = tid + u * NT;
        const int kc = blk & 7, ic = blk >> 3;
        if (active(blk)) {
#pragma unroll
          for (int j = 0; j < 8; ++j) r[u * 8 + j] = l.vec(row0 + ic * 8, k0 + kc * 8 + j);
        }
      }
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) {
    if constexpr (L::kKMajor) {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int v = tid + u * NT;
        if (active(v)) *reinterpret_cast<uint4*>(lds + lds_off(v >> 3, v & 7)) = r[u];
      }
    } else {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int blk = tid + u * NT;
        const int kc = blk & 7, ic = blk >> 3;
        if (active(blk)) {
          uint4 in[8], out[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) in[j] = r[u * 8 + j];
          transpose8x8_b16(in, out);  // out[c] = the 8 k-values of tile row ic*8 + c
#pragma unroll
          for (int c = 0; c < 8; ++c) *reinterpret_cast<uint4*>(lds + lds_off(ic * 8 + c, kc)) = out[c];
        }
      }
    }
  }
};

// Map the linear block id to a (tile_m, tile_n) pair: blocks are dealt
// round-robin to the 8 XCDs, so give each XCD a contiguous run of tiles,
// M-tile fastest (consecutive tiles share the same B tile).
__device__ __forceinline__ void xcd_tile(int pid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nt = tiles_m * tiles_n;
  int tile = pid;
  if ((nt & 7) == 0) tile = (pid & 7) * (nt >> 3) + (pid >> 3);
  tm = tile % tiles_m;
  tn = tile / tiles_m;
}

template <int BM, int BN, int WM, int WN, class AL, class BL, class Epi>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
    gemm_bf16_mfma(AL al, BL bl, Epi epi, int M, int N, int K, int ktiles_per_split) {
  constexpr int BK = 64;
  constexpr int WAVES_N = BN / WN;
  constexpr int NT = (BM / WM) * WAVES_N * 64;
  constexpr int MB = WM / 32, NB = WN / 32;
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  __shared__ __attribute__((aligned(16))) char smem[2 * (A_BYTES + B_BYTES)];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / WAVES_N) * WM, wn0 = (wave % WAVES_N) * WN;
  int tm, tn;
  xcd_tile(blockIdx.x, (M + BM - 1) / BM, (N + BN - 1) / BN, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int split = blockIdx.z;
  const int nkt = (K + BK - 1) / BK;
  const int kt0 = split * ktiles_per_split;
  const int kt1 = min(nkt, kt0 + ktiles_per_split);

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.0f;

  TileLoader<BM, NT, AL> la;
  TileLoader<BN, NT, BL> lb;
  // buffer b of A at smem + b*A_BYTES, of B at smem + 2*A_BYTES + b*B_BYTES
  if (kt0 < kt1) {
    la.load(al, m0, kt0 * BK, tid);
    lb.load(bl, n0, kt0 * BK, tid);
    la.store(smem, tid);
    lb.store(smem + 2 * A_BYTES, tid);
  }
  __syncthreads();

  const int frow = lane & 31, fchunk = lane >> 5;
  for (int kt = kt0; kt < kt1; ++kt) {
    const int buf = (kt - kt0) & 1;
    const bool more = kt + 1 < kt1;
    if (more) {
      la.load(al, m0, (kt + 1) * BK, tid);
      lb.load(bl, n0, (kt + 1) * BK, tid);
    }
    const char* a_s = smem + buf * A_BYTES;
    const char* b_s = smem + 2 * A_BYTES + buf * B_BYTES;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8_t af[MB], bfr[NB];
#pragma unroll
      for (int a = 0; a < MB; ++a)
        af[a] = __builtin_bit_cast(bf16x8_t,
                                   *reinterpret_cast<const uint4*>(a_s + lds_off(wm0 + a * 32 + frow, kk * 2 + fchunk)));
#pragma unroll
      for (int b = 0; b < NB; ++b)
        bfr[b] = __builtin_bit_cast(bf16x8_t,
                                    *reinterpret_cast<const uint4*>(b_s + lds_off(wn0 + b * 32 + frow, kk * 2 + fchunk)));
#pragma unroll
      for (int a = 0; a < MB; ++a)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
    if (more) {
      la.store(smem + (buf ^ 1) * A_BYTES, tid);
      lb.store(smem + 2 * A_BYTES + (buf ^ 1) * B_BYTES, tid);
    }
    __syncthreads();
  }

  // accumulator layout of a 32 x 32 block: lane holds column (lane & 31);
  // register e holds row 8*(e/4) + 4*(lane/32) + (e%4)
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = m0 + wm0 + a * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int j = n0 + wn0 + b * 32 + (lane & 31);
        if (i < M && j < N) epi(i, j, acc[a][b][e], split);
      }
}

// ------------------------------------------------------------ launchers

template <class AL, class BL, class Epi>
inline void launch_gemm_f32(const AL& al, const BL& bl, const Epi& epi, int M, int N, int K, int splits,
                            hipStream_t s) {
  const int nkt = (K + 15) / 16;
  const int kps = (nkt + splits - 1) / splits;
  dim3 grid((M + 63) / 64, (N + 63) / 64, splits);
  hipLaunchKernelGGL((gemm_f32_fma<AL, BL, Epi>), grid, dim3(256), 0, s, al, bl, epi, M, N, K, kps);
}

// Tile configurations of the bf16 engine.
enum class BfTile { k256x256, k128x128 };

template <class AL, class BL, class Epi>
inline void launch_gemm_bf16(const AL& al, const BL& bl, const Epi& epi, int M, int N, int K, int splits,
                             BfTile tile, hipStream_t s) {
  const int nkt = (K + 63) / 64;
  const int kps = (nkt + splits - 1) / splits;
  if (tile == BfTile::k256x256) {
    const unsigned tiles = ((M + 255) / 256) * ((N + 255) / 256);
    hipLaunchKernelGGL((gemm_bf16_mfma<256, 256, 128, 128, AL, BL, Epi>), dim3(tiles, 1, splits), dim3(256), 0, s,
                       al, bl, epi, M, N, K, kps);
  } else {
    const unsigned tiles = ((M + 127) / 128) * ((N + 127) / 128);
    hipLaunchKernelGGL((gemm_bf16_mfma<128, 128, 64, 64, AL, BL, Epi>), dim3(tiles, 1, splits), dim3(256), 0, s, al,
                       bl, epi, M, N, K, kps);
  }
}

// --------------------------------------------------------------- planning

struct GemmPlan {
  bool bf16;
  BfTile tile;
  int splits;
};

inline int cdiv(long long a, long long b) { return static_cast<int>((a + b - 1) / b); }

// Choose tile shape and split-K so the launch has >= ~256 blocks (one per
// CU) while every split keeps a reasonable number of K tiles.
inline GemmPlan plan_gemm(bool bf16, int M, int N, int K) {
  GemmPlan p{bf16, BfTile::k256x256, 1};
  if (!bf16) {
    const int tiles = cdiv(M, 64) * cdiv(N, 64);
    const int nkt = cdiv(K, 16);
    int s = cdiv(512, tiles);
    s = std::min(s, std::max(1, nkt / 8));
    p.splits = std::max(1, std::min(s, 16));
    return p;
  }
  const int nkt = cdiv(K, 64);
  const int t256 = cdiv(M, 256) * cdiv(N, 256);
  if (t256 >= 64) {
    int s = cdiv(256, t256);
    s = std::min(s, std::max(1, nkt / 16));
    p.tile = BfTile::k256x256;
    p.splits = std::max(1, std::min(s, 8));
    return p;
  }
  const int t128 = cdiv(M, 128) * cdiv(N, 128);
  int s = cdiv(256, t128);
  s = std::min(s, std::max(1, nkt / 8));
  p.tile = BfTile::k128x128;
  p.splits = std::max(1, std::min(s, 8));
  return p;
}

template <class AL, class BL, class Epi>
inline void run_gemm(const GemmPlan& p, const AL& al, const BL& bl, const Epi& epi, int M, int N, int K,
                     hipStream_t s) {
  if (p.bf16)
    launch_gemm_bf16(al, bl, epi, M, N, K, p.splits, p.tile, s);
  else
    launch_gemm_f32(al, bl, epi, M, N, K, p.splits, s);
}

}  // namespace o5
