// GEMM engines of libo5:  C[i, j] = sum_k A(i, k) * B(j, k)  (+ epilogue).
//
// Operands are described by small loader structs instead of raw pointers so
// that one engine serves every contraction of the LSTM step:
//   forward  G_t   = [x_t | h~_{t-1}] . [W_x | W_h]^T      (A, B K-contiguous)
//   backward dh    = dG_t . W_h                             (B I-contiguous)
//   weights  dW    = dG^T . [x | h~_prev]                   (A, B I-contiguous)
//   input    dx    = dG . W_x                               (B I-contiguous)
// A loader reports whether its reduction index k is the contiguous one
// (kKMajor), hands out single elements to the fp32 engine (at) and, for
// the bf16 engine, has a per-thread Tile state that precomputes everything
// that does not change along K (row offsets, masks, sources) so that the
// K loop issues plain 16-byte loads with no branches.
//
// bf16 engine (gfx950 MFMA, v_mfma_f32_32x32x16_bf16, fp32 accumulate):
//  * block tile BM x BN, K tile 64, waves arranged (BM/WM) x (BN/WN), each
//    wave owning (WM/32) x (WN/32) MFMA blocks;
//  * both tiles staged in LDS as [row][64 k] bf16, double buffered, the
//    16-byte chunk index XOR-swizzled by (row >> 1) & 7 so that 16
//    consecutive rows read at one chunk hit 16 distinct 16-byte bank groups;
//  * operands whose contiguous index is not k are loaded as 8x8 blocks and
//    transposed in registers (v_perm) before the LDS store, so MFMA fragment
//    reads are always single 16-byte LDS reads;
//  * global loads of tile kt+1 are in flight while tile kt is multiplied,
//    and the fragments of k-step kk+1 are read from LDS while the MFMAs of
//    k-step kk run;
//  * blocks are dealt round-robin to the 8 XCDs; each XCD gets a contiguous
//    run of tiles ordered in groups of kGroupM = 4 M-tiles (M-tile fastest),
//    so the ~32 blocks an XCD runs at once cover 4 M-tiles x 8 N-tiles and
//    share both operands in that XCD's L2 (4 measured faster than 8 or 16
//    on the weight-gradient GEMM);
//  * optional split-K over gridDim.z; split z writes its partial sums to
//    its own slice (the caller reduces the slices in a fixed order).
#pragma once

#include <type_traits>

#include "common.h"

namespace o5 {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint4 zero4() { return make_uint4(0u, 0u, 0u, 0u); }
__device__ __forceinline__ uint4 sel4(bool keep, uint4 v) { return keep ? v : zero4(); }

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

// ------------------------------------------------------------------ loaders

// (i, k) -> K-contiguous rows, two segments along k: k < K0 reads p0[i*ld0 + k],
// k >= K0 reads p1[i*ld1 + k - K0].  A nonzero mask1[i] zeroes the p1 part
// of row i (the reset of the carried LSTM state).
template <typename E>
struct KRows2 {
  static constexpr bool kKMajor = true;
  static constexpr bool kBf16 = sizeof(E) == 2;
  const E* p0;
  const E* p1;
  const uint8_t* mask1;
  int ld0, ld1, K0, K, rows;
  // gate gathering (direct-to-LDS engine only): when gstride > 0, tile row r
  // of the block starting at row0 is source row (r / 64) * gstride +
  // row0 / 4 + r % 64, i.e. a 256-row tile holds the four gate blocks
  // (stride gstride = H) of 64 consecutive hidden units.
  int gstride = 0;

  __device__ __forceinline__ float at(int i, int k) const {
    if (i >= rows || k >= K) return 0.0f;
    if (k < K0) return elem<E>::to_f32(p0[static_cast<size_t>(i) * ld0 + k]);
    if (mask1 && mask1[i]) return 0.0f;
    return elem<E>::to_f32(p1[static_cast<size_t>(i) * ld1 + (k - K0)]);
  }

  // Per-thread state of the bf16 engine for a ROWS x 64 tile loaded by NT
  // threads: thread t always loads chunk (t & 7) of rows (t >> 3) + u*NT/8.
  // Requires K0 % 64 == 0 (a K tile never straddles the two sources),
  // K % 8 == 0 and rows * ld < 2^31; bf16 only.
  template <int ROWS, int NT>
  struct Tile {
    static constexpr int kPer = ROWS * 8 / NT;
    static constexpr int kVecs = kPer;
    static_assert(ROWS * 8 % NT == 0, "tile/threads mismatch");
    int off0[kPer], off1[kPer];  // element offset of each row in p0 / p1; < 0 -> zeros
    int chunk;

    __device__ __forceinline__ void init(const KRows2& l, int row0, int tid) {
      chunk = (tid & 7) * 8;
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int row = row0 + (tid >> 3) + u * (NT / 8);
        const bool valid = row < l.rows;
        const bool masked = valid && l.mask1 != nullptr && l.mask1[row] != 0;
        off0[u] = valid ? row * l.ld0 : -1;
        off1[u] = (valid && !masked) ? row * l.ld1 : -1;
      }
    }
    __device__ __forceinline__ void load(const KRows2& l, int k0, uint4 (&r)[kVecs]) const {
      const bool seg0 = k0 < l.K0;  // uniform over the block
      const bool kok = k0 + chunk < l.K;
      const E* base = seg0 ? l.p0 + k0 : l.p1 + (k0 - l.K0);
      const int kc = kok ? chunk : 0;  // k0 itself is always inside the row
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int off = seg0 ? off0[u] : off1[u];
        const uint4 v = *reinterpret_cast<const uint4*>(base + (off < 0 ? 0 : off) + kc);
        r[u] = sel4(off >= 0 && kok, v);
      }
    }
    __device__ __forceinline__ void store(char* lds, int tid, const uint4 (&r)[kVecs]) const {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int row = (tid >> 3) + u * (NT / 8);
        *reinterpret_cast<uint4*>(lds + lds_off(row, tid & 7)) = r[u];
      }
    }
  };
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
  static constexpr bool kBf16 = sizeof(E) == 2;
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

  // Per-thread state of the bf16 engine for a ROWS x 64 tile: the tile holds
  // (ROWS/8) x 8 blocks of 8 i x 8 k; thread t loads block (i-chunk t >> 3,
  // k-chunk t & 7) (+ NT/8 i-chunks per extra block), i.e. 8 rows k of 8
  // consecutive i, and transposes them before the LDS store.  Requires
  // I0 % 8 == 0 and I % 8 == 0; bf16 only.
  template <int ROWS, int NT>
  struct Tile {
    static constexpr int kBlocks = ROWS;  // (ROWS/8) i-chunks x 8 k-chunks
    static constexpr int kPer = kBlocks >= NT ? kBlocks / NT : 1;
    static constexpr int kVecs = kPer * 8;
    static_assert(kBlocks >= NT ? kBlocks % NT == 0 : NT % kBlocks == 0, "tile/threads mismatch");
    int col[kPer];   // column inside its source (0 when the block is idle or out of range)
    uint32_t flags;  // bit u: block u active and in range; bit 8+u: block u reads the second source
    int kc;

    __device__ __forceinline__ void init(const ICols2& l, int row0, int tid) {
      kc = (tid & 7) * 8;
      flags = 0;
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int blk = tid + u * NT;
        const int i = row0 + (blk >> 3) * 8;
        const bool ok = blk < kBlocks && i < l.I;
        const bool second = ok && i >= l.I0;
        col[u] = ok ? (second ? i - l.I0 : i) : 0;
        flags |= (ok ? 1u : 0u) << u;
        flags |= (second ? 1u : 0u) << (8 + u);
      }
    }
    __device__ __forceinline__ void load(const ICols2& l, int k0, uint4 (&r)[kVecs]) const {
      if constexpr (kBlocks < NT) {
        if ((flags & 1u) == 0u) return;  // idle or out-of-range block: store() skips it too
      }
      const int kb = k0 + kc;  // first of this thread's 8 rows k
      // reset mask of the 8 rows (applies to the second source only)
      uint32_t mlo = 0, mhi = 0;
      if (l.mask1 != nullptr) {
        if (kb + 8 <= l.K) {
          const uint2 m = *reinterpret_cast<const uint2*>(l.mask1 + kb);
          mlo = m.x;
          mhi = m.y;
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const uint32_t b = (kb + j < l.K) ? l.mask1[kb + j] : 0u;
            if (j < 4)
              mlo |= b << (8 * j);
            else
              mhi |= b << (8 * (j - 4));
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const bool ok = (flags >> u) & 1u;
        const bool second = (flags >> (8 + u)) & 1u;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int k = kb + j;
          const bool kin = k < l.K;
          const int kk = kin ? k : l.K - 1;  // clamped row: always a valid address
          const E* p;
          if (!second) {
            p = l.p0 + static_cast<size_t>(kk) * l.ld0 + col[u];
          } else {
            p = (kk < l.kswitch ? l.p1a + static_cast<size_t>(kk) * l.ld1
                                : l.p1b + static_cast<size_t>(kk - l.kswitch) * l.ld1) + col[u];
          }
          const uint32_t mb = (j < 4 ? mlo >> (8 * j) : mhi >> (8 * (j - 4))) & 0xffu;
          const bool keep = ok && kin && !(second && mb != 0u);
          r[u * 8 + j] = sel4(keep, *reinterpret_cast<const uint4*>(p));
        }
      }
    }
    __device__ __forceinline__ void store(char* lds, int tid, const uint4 (&r)[kVecs]) const {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int blk = tid + u * NT;
        if (blk < kBlocks) {
          if constexpr (kBlocks < NT) {
            if ((flags & 1u) == 0u) continue;  // not loaded: leave the rows as they are
          }
          uint4 in[8], out[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) in[j] = r[u * 8 + j];
          transpose8x8_b16(in, out);  // out[c] = the 8 k-values of tile row (blk>>3)*8 + c
#pragma unroll
          for (int c = 0; c < 8; ++c)
            *reinterpret_cast<uint4*>(lds + lds_off((blk >> 3) * 8 + c, blk & 7)) = out[c];
        }
      }
    }
  };
};

// ------------------------------------------------------------ epilogues

// Plain fp32 store of C (row-major, ldc) into slice `split` of a stack of
// M x N partial results (slice stride = sstride elements).
struct EpiStoreF32 {
  static constexpr int kTileSmem = 0;
  float* c;
  int ldc;
  size_t sstride;
  __device__ __forceinline__ void operator()(int i, int j, float v, int split) const {
    c[split * sstride + static_cast<size_t>(i) * ldc + j] = v;
  }
  // where the 32-column block from (i0, j0) goes and its row pitch
  __device__ __forceinline__ bool blocks_ok() const { return true; }
  __device__ __forceinline__ float* block(int i0, int j0, int split, int& ld) const {
    ld = ldc;
    return c + split * sstride + static_cast<size_t>(i0) * ldc + j0;
  }
};

// Store into one of two fp32 matrices split by column: j < J0 -> c0[i*ld0 + j],
// else c1[i*ld1 + j - J0]  (dW = [dW_x | dW_h]).
struct EpiStoreF32Split2 {
  static constexpr int kTileSmem = 0;
  float* c0;
  float* c1;
  int ld0, ld1, J0;
  __device__ __forceinline__ void operator()(int i, int j, float v, int) const {
    if (j < J0)
      c0[static_cast<size_t>(i) * ld0 + j] = v;
    else
      c1[static_cast<size_t>(i) * ld1 + (j - J0)] = v;
  }
  // (a 32-column block lies in one matrix when J0 is a multiple of 32)
  __device__ __forceinline__ bool blocks_ok() const { return J0 % 32 == 0; }
  __device__ __forceinline__ float* block(int i0, int j0, int, int& ld) const {
    ld = j0 < J0 ? ld0 : ld1;
    return j0 < J0 ? c0 + static_cast<size_t>(i0) * ld0 + j0 : c1 + static_cast<size_t>(i0) * ld1 + (j0 - J0);
  }
};

// Store converted to the element type E (dx in the GEMM input type).
template <typename E>
struct EpiStoreElem {
  static constexpr int kTileSmem = 0;
  E* c;
  int ldc;
  __device__ __forceinline__ void operator()(int i, int j, float v, int) const {
    c[static_cast<size_t>(i) * ldc + j] = elem<E>::from_f32(v);
  }
};

// Epilogues that store 32 x 32 accumulator blocks row by row (block(),
// blocks_ok()): the stores of a full tile take a uniform block base and a
// per-lane 32-bit offset, with no per-element bounds test or 64-bit index.
template <class Epi, class = void>
struct HasBlockStore : std::false_type {};
template <class Epi>
struct HasBlockStore<Epi, std::void_t<decltype(&Epi::blocks_ok)>> : std::true_type {};

// The element epilogue of an MB x NB set of 32 x 32 MFMA accumulator blocks
// at (i0, j0) of an M x N result.  Accumulator layout of a block: lane holds
// column (lane & 31); register e holds row 8*(e/4) + 4*(lane/32) + (e%4).
// `full`: the block tile lies inside M x N.
template <int MB, int NB, class Epi>
__device__ __forceinline__ void store_acc(const Epi& epi, const f32x16_t (&acc)[MB][NB], int i0, int j0, int lane,
                                          int split, int M, int N, bool full) {
  if constexpr (HasBlockStore<Epi>::value) {
    if (full && epi.blocks_ok()) {
#pragma unroll
      for (int a = 0; a < MB; ++a)
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          int ld;
          float* base = epi.block(i0 + a * 32, j0 + b * 32, split, ld);
          const int lo = 4 * (lane >> 5) * ld + (lane & 31);
#pragma unroll
          for (int e = 0; e < 16; ++e) base[lo + (8 * (e >> 2) + (e & 3)) * ld] = acc[a][b][e];
        }
      return;
    }
  }
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = i0 + a * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int j = j0 + b * 32 + (lane & 31);
        if (full || (i < M && j < N)) epi(i, j, acc[a][b][e], split);
      }
}

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

constexpr int kGroupM = 4;

// Map the linear block id to a (tile_m, tile_n) pair.  Blocks are dealt
// round-robin to the 8 XCDs, so each XCD first gets a contiguous run of
// tiles (when the tile count is a multiple of 8); tiles are then numbered in
// groups of kGroupM M-tiles with the M-tile fastest.
__device__ __forceinline__ void group_tile(int tile, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int gsz = kGroupM * tiles_n;
  const int g = tile / gsz;
  const int first_m = g * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int in = tile - g * gsz;
  tm = first_m + in % gm;
  tn = in / gm;
}

__device__ __forceinline__ void xcd_tile(int pid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nt = tiles_m * tiles_n;
  int tile = pid;
  if ((nt & 7) == 0) tile = (pid & 7) * (nt >> 3) + (pid >> 3);
  group_tile(tile, tiles_m, tiles_n, tm, tn);
}

// The same for a grid of S K splits, block (x, z) = tile x of split z
// (dispatched as linear id x + gridDim.x * z).  When S divides 8 the 8 / S
// XCDs of one split take its tiles in contiguous runs, so the blocks an XCD
// holds read the same K range and share operand panels in its L2 (with the
// plain mapping each XCD would hold every split of fewer tiles); otherwise
// xcd_tile with split z.
__device__ __forceinline__ void xcd_tile_split(int x, int z, int S, int tiles_m, int tiles_n, int& tm, int& tn,
                                               int& split) {
  const int nt = tiles_m * tiles_n;
  if (S > 1 && 8 % S == 0 && nt % (8 / S) == 0) {
    const int xs = 8 / S;           // XCDs per split
    const int L = x + nt * z;       // the dispatch order; XCD = L % 8
    const int xcd = L & 7, slot = L >> 3;
    split = xcd / xs;
    group_tile((xcd % xs) * (nt / xs) + slot, tiles_m, tiles_n, tm, tn);
  } else {
    split = z;
    xcd_tile(x, tiles_m, tiles_n, tm, tn);
  }
}

template <int MB, int NB>
__device__ __forceinline__ void read_frags(const char* a_s, const char* b_s, int wm0, int wn0, int frow, int fchunk,
                                           bf16x8_t (&af)[MB], bf16x8_t (&bfr)[NB]) {
#pragma unroll
  for (int a = 0; a < MB; ++a)
    af[a] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(a_s + lds_off(wm0 + a * 32 + frow, fchunk)));
#pragma unroll
  for (int b = 0; b < NB; ++b)
    bfr[b] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(b_s + lds_off(wn0 + b * 32 + frow, fchunk)));
}

template <int MB, int NB>
__device__ __forceinline__ void mfma_block(const bf16x8_t (&af)[MB], const bf16x8_t (&bfr)[NB],
                                           f32x16_t (&acc)[MB][NB]) {
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
}

template <int BM, int BN, int WM, int WN, class AL, class BL, class Epi>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64, 1)
    gemm_bf16_mfma(AL al, BL bl, Epi epi, int M, int N, int K, int ktiles_per_split) {
  constexpr int BK = 64;
  constexpr int WAVES_N = BN / WN;
  constexpr int NT = (BM / WM) * WAVES_N * 64;
  constexpr int MB = WM / 32, NB = WN / 32;
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  __shared__ __attribute__((aligned(16))) char smem[2 * (A_BYTES + B_BYTES)];
  using ATile = typename AL::template Tile<BM, NT>;
  using BTile = typename BL::template Tile<BN, NT>;

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

  ATile ta;
  BTile tb;
  // the B operand uses a rotated thread index, so that when a tile has fewer
  // 8x8 blocks than threads the A and B loads land on different waves
  const int tidb = (tid + NT / 2) % NT;
  ta.init(al, m0, tid);
  tb.init(bl, n0, tidb);
  uint4 ra[ATile::kVecs], rb[BTile::kVecs];

  // buffer b of A at smem + b*A_BYTES, of B at smem + 2*A_BYTES + b*B_BYTES
  if (kt0 < kt1) {
    ta.load(al, kt0 * BK, ra);
    tb.load(bl, kt0 * BK, rb);
    ta.store(smem, tid, ra);
    tb.store(smem + 2 * A_BYTES, tidb, rb);
  }
  __syncthreads();

  const int frow = lane & 31, fhalf = lane >> 5;
  for (int kt = kt0; kt < kt1; ++kt) {
    const int buf = (kt - kt0) & 1;
    const bool more = kt + 1 < kt1;
    if (more) {
      ta.load(al, (kt + 1) * BK, ra);
      tb.load(bl, (kt + 1) * BK, rb);
    }
    const char* a_s = smem + buf * A_BYTES;
    const char* b_s = smem + 2 * A_BYTES + buf * B_BYTES;
    bf16x8_t af0[MB], bf0[NB], af1[MB], bf1[NB];
    // fragments of k-step kk+1 are read while the MFMAs of k-step kk run
    read_frags<MB, NB>(a_s, b_s, wm0, wn0, frow, 0 + fhalf, af0, bf0);
    read_frags<MB, NB>(a_s, b_s, wm0, wn0, frow, 2 + fhalf, af1, bf1);
    mfma_block<MB, NB>(af0, bf0, acc);
    read_frags<MB, NB>(a_s, b_s, wm0, wn0, frow, 4 + fhalf, af0, bf0);
    mfma_block<MB, NB>(af1, bf1, acc);
    read_frags<MB, NB>(a_s, b_s, wm0, wn0, frow, 6 + fhalf, af1, bf1);
    mfma_block<MB, NB>(af0, bf0, acc);
    mfma_block<MB, NB>(af1, bf1, acc);
    if (more) {
      ta.store(smem + (buf ^ 1) * A_BYTES, tid, ra);
      tb.store(smem + 2 * A_BYTES + (buf ^ 1) * B_BYTES, tidb, rb);
    }
    __syncthreads();
  }

  // accumulator layout of a 32 x 32 block: lane holds column (lane & 31);
  // register e holds row 8*(e/4) + 4*(lane/32) + (e%4)
  const bool full = m0 + BM <= M && n0 + BN <= N;
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = m0 + wm0 + a * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int j = n0 + wn0 + b * 32 + (lane & 31);
        if (full || (i < M && j < N)) epi(i, j, acc[a][b][e], split);
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

// Tile configurations of the bf16 engines: block tile, waves (x 64 threads).
//   kDma256    256 x 256, 8 waves, buffer loads straight to LDS (gemm_kk.h for
//              two K-contiguous operands, else gemm_dma.h)
//   k256x256w8 256 x 256, 8 waves of 128 x 64, register-staged (operands the
//              direct-to-LDS engines cannot take: a masked second source)
//   k128x128   128 x 128, 4 waves of 64 x 64, register-staged (small grids)
enum class BfTile { kDma256, k256x256w8, k128x128 };

template <class AL, class BL, class Epi>
inline void launch_gemm_bf16(const AL& al, const BL& bl, const Epi& epi, int M, int N, int K, int splits,
                             BfTile tile, hipStream_t s) {
  const int nkt = (K + 63) / 64;
  const int kps = (nkt + splits - 1) / splits;
  if (tile == BfTile::k256x256w8) {
    const unsigned tiles = ((M + 255) / 256) * ((N + 255) / 256);
    hipLaunchKernelGGL((gemm_bf16_mfma<256, 256, 128, 64, AL, BL, Epi>), dim3(tiles, 1, splits), dim3(512), 0, s,
                       al, bl, epi, M, N, K, kps);
  } else {
    const unsigned tiles = ((M + 127) / 128) * ((N + 127) / 128);
    hipLaunchKernelGGL((gemm_bf16_mfma<128, 128, 64, 64, AL, BL, Epi>), dim3(tiles, 1, splits), dim3(256), 0, s, al,
                       bl, epi, M, N, K, kps);
  }
}

}  // namespace o5
