// bf16 MFMA GEMM fed by direct-to-LDS loads (gfx950):
//   C[i, j] = sum_k A(i, k) * B(j, k)  (+ epilogue), fp32 accumulate.
//
// Pipeline: the K loop runs over tiles of 32 k held in a ring of STAGES (5)
// LDS stages.  Tiles are copied global -> LDS by global_load_lds_dwordx4 (16
// bytes per lane, written at M0 + 16 * lane), so no registers stage the
// operands and STAGES - 1 tiles are in flight while one is multiplied: each
// iteration waits (vmcnt) for its own tile only, meets the other waves at one
// barrier, issues the copy of the tile STAGES - 1 steps ahead into the stage
// that was just freed, and runs its MFMAs.  The stages are distinct LDS
// arrays and the loop is unrolled by STAGES, so the compiler can see that the
// copies in flight never alias the LDS reads (it would otherwise wait for
// every copy before each read); the barrier is a bare s_barrier (a fence
// would also wait for the copies).
//
// Operand layouts in LDS (one stage; 256 rows/columns x 32 k):
//  * K-contiguous operand: [row][32 k] bf16 = 64 bytes per row, 16-byte
//    chunk c of row r stored at slot c ^ ((r >> 2) & 3).  A fragment read
//    (16 consecutive rows, one chunk) then touches 16 distinct 16-byte bank
//    groups.  Fragments are single ds_read_b128.
//  * I-contiguous operand (the reduction index k is the row): [32 k][256 i]
//    bf16 = 512 bytes per k row, 16-byte unit u of row k stored at position
//    u ^ (4 * (k & 3)).  Fragments are two ds_read_b64_tr_b16: within each
//    16-lane group the 16 lanes' 4-element reads form a 64-element sequence
//    S and lane i receives S[i], S[16+i], S[32+i], S[48+i]; when lane j reads
//    row k0 + j/4, columns n0 + 4(j%4) .. +3, lane i receives k0..k0+3 of
//    column n0 + i -- an MFMA operand slice.  The swizzle keeps the 4 rows x
//    4 eight-byte pieces of a 32-lane half on distinct banks.
// MFMA v_mfma_f32_32x32x16_bf16: lane l supplies row/column (l & 31) and the
// k slice 8*(l >> 5) .. +7 of a 16-wide k step, for both operands alike.
//
// Block tile 256 x 256, 8 waves (2 x 4) of 128 x 64, two waves per SIMD.
// Rows or k beyond the matrix read a static zero row, so every address the
// copies use is inside a buffer.
#pragma once

#include <type_traits>

#include "gemm.h"

namespace o5 {

namespace dma {

constexpr int BM = 256, BN = 256, BK = 32, STAGES = 5;  // 5 x 32 KB: dW of the pre-LSTM layer 1.20 against 1.23 ms with 4
static_assert(STAGES >= 3 && STAGES <= 5, "3..5 stages fit in 160 KB of LDS");
// 8 waves (2 x 4) of 128 x 64, two waves per SIMD
constexpr int WM = 128, WN = 64;
constexpr int WAVES_M = BM / WM, WAVES_N = BN / WN;
constexpr int NWAVES = WAVES_M * WAVES_N;
constexpr int NT = NWAVES * 64;
constexpr int TILE_BYTES = 256 * BK * 2;   // 16 KB per operand per stage
constexpr int COPIES = TILE_BYTES / 1024 / NWAVES;  // 1 KB copies per wave per operand per tile

// 1 KB of zeros: the source of every copy that falls outside a matrix.
__device__ __attribute__((aligned(16))) const uint16_t kZeroRow[512] = {};

// One wave-wide copy of 64 x 16 bytes into LDS at lds_wave_base + 16 * lane.
// Written as inline asm so that the compiler's wait-count pass neither tracks
// these copies (it would wait for all of them before every LDS read) nor
// edits the explicit waits below; ordering against the LDS reads is kept by
// wait_copies + wave_barrier.
__device__ __forceinline__ void copy16(const void* g, char* lds_wave_base) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<size_t>((__attribute__((address_space(3))) char*)(lds_wave_base))));
  // one wait state between the M0 write and the LDS DMA that reads it (a
  // hazard the compiler would handle for instructions it can see)
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}

// ------------------------------------------------- K-contiguous operand
// Rows i of the operand are K-contiguous; two sources along k (split at K0,
// a multiple of 32): k < K0 -> p0[i*ld0 + k], else p1[i*ld1 + k - K0].
// mask1[i] != 0 zeroes the second source for row i.
template <typename E, int NC = COPIES>
struct KTile {
  const char* ptr0[NC];  // row start in source 0 (bytes), or nullptr = zero row
  const char* ptr1[NC];  // row start in source 1
  int koff;                  // byte offset of this lane's 16-byte chunk within a tile

  __device__ __forceinline__ void init(const KRows2<E>& l, int row0, int wave, int lane) {
    const int slot = lane & 3;
#pragma unroll
    for (int q = 0; q < NC; ++q) {
      const int r = (wave * NC + q) * 16 + (lane >> 2);  // tile row this lane fills
      const int row = l.gstride > 0 ? (r >> 6) * l.gstride + (row0 >> 2) + (r & 63) : row0 + r;
      const int chunk = slot ^ ((r >> 2) & 3);
      koff = chunk * 16;
      const bool valid = row < l.rows;
      const bool masked = valid && l.mask1 != nullptr && l.mask1[row] != 0;
      ptr0[q] = valid ? reinterpret_cast<const char*>(l.p0 + static_cast<size_t>(row) * l.ld0) : nullptr;
      ptr1[q] = (valid && !masked && l.p1 != nullptr)
                    ? reinterpret_cast<const char*>(l.p1 + static_cast<size_t>(row) * l.ld1)
                    : nullptr;
    }
  }
  // copy piece q of the tile starting at k0 into `stage`
  __device__ __forceinline__ void issue_one(const KRows2<E>& l, int k0, char* stage, int wave, int q) const {
    const bool seg0 = k0 < l.K0;
    const int kb = seg0 ? k0 : k0 - l.K0;  // element offset inside the source row
    const bool kin = k0 + koff / 2 < l.K;
    const char* p = seg0 ? ptr0[q] : ptr1[q];
    const void* g = (p != nullptr && kin) ? static_cast<const void*>(p + kb * 2 + koff)
                                          : static_cast<const void*>(kZeroRow);
    copy16(g, stage + (wave * NC + q) * 1024);
  }
  // copy tile starting at k0 into `stage` (this wave's 1 KB pieces)
  __device__ __forceinline__ void issue(const KRows2<E>& l, int k0, char* stage, int wave) const {
#pragma unroll
    for (int q = 0; q < NC; ++q) issue_one(l, k0, stage, wave, q);
  }
};

// LDS byte offset of chunk c (0..3) of K-contiguous tile row r.
__device__ __forceinline__ int koffset(int r, int c) { return r * 64 + ((c ^ ((r >> 2) & 3)) << 4); }

template <int NBLK>
__device__ __forceinline__ void read_k(const char* stage, int row0, int lane, int kk, bf16x8_t (&f)[NBLK]) {
  const int c = kk * 2 + (lane >> 5);
#pragma unroll
  for (int b = 0; b < NBLK; ++b) {
    const int r = row0 + b * 32 + (lane & 31);
    f[b] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(stage + koffset(r, c)));
  }
}

// ------------------------------------------------- I-contiguous operand
// Element (i, k) at row k of the source: i < I0 -> p0[k*ld0 + i]; i >= I0 ->
// (k < kswitch ? p1a + k*ld1 : p1b + (k - kswitch)*ld1)[i - I0].  No mask.
template <typename E>
struct ITile {
  int col[COPIES];   // element column of this lane's 16 bytes inside its source row
  int kl[COPIES];    // tile k row this copy fills
  uint32_t second;   // bit q: the lane's columns come from the second source
  uint32_t ok;       // bit q: the lane's columns are inside the matrix

  __device__ __forceinline__ void init(const ICols2<E>& l, int row0, int wave, int lane) {
    second = 0;
    ok = 0;
#pragma unroll
    for (int q = 0; q < COPIES; ++q) {
      const int piece = wave * COPIES + q;  // 1 KB piece = 2 k rows of 512 bytes
      const int k = piece * 2 + (lane >> 5);
      const int u = (lane & 31) ^ (4 * (k & 3));
      const int i = row0 + u * 8;
      kl[q] = k;
      const bool in = i < l.I;
      const bool sec = i >= l.I0;
      ok |= (in ? 1u : 0u) << q;
      second |= (sec ? 1u : 0u) << q;
      col[q] = sec ? i - l.I0 : i;
    }
  }
  __device__ __forceinline__ void issue(const ICols2<E>& l, int k0, char* stage, int wave) const {
#pragma unroll
    for (int q = 0; q < COPIES; ++q) {
      const int k = k0 + kl[q];
      const bool valid = ((ok >> q) & 1u) && k < l.K;
      const E* row;
      if ((second >> q) & 1u)
        row = k < l.kswitch ? l.p1a + static_cast<size_t>(k) * l.ld1
                            : l.p1b + static_cast<size_t>(k - l.kswitch) * l.ld1;
      else
        row = l.p0 + static_cast<size_t>(k) * l.ld0;
      const void* g = valid ? static_cast<const void*>(row + col[q]) : static_cast<const void*>(kZeroRow);
      copy16(g, stage + (wave * COPIES + q) * 1024);
    }
  }
};

typedef short v4s_t __attribute__((ext_vector_type(4)));

// Two transpose reads give lane (l & 31)'s 8 k values (8*(l>>5) .. +7 of k
// step kk) for 32-wide block b of an I-contiguous stage.
template <int NBLK>
__device__ __forceinline__ void read_i(const char* stage, int col0, int lane, int kk, bf16x8_t (&f)[NBLK]) {
  const int g = lane >> 4, j = lane & 15;
  const int kg = kk * 16 + 8 * (g >> 1);
#pragma unroll
  for (int b = 0; b < NBLK; ++b) {
    const int nb = col0 + b * 32 + 16 * (g & 1) + 4 * (j & 3);  // first column this lane reads
    v4s_t h[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int k = kg + 4 * r + (j >> 2);
      const int u = nb >> 3;
      const int off = k * 512 + ((u ^ (4 * (k & 3))) << 4) + ((nb & 7) << 1);
      h[r] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s_t*)(stage + off));
    }
    struct {
      v4s_t a, b;
    } pair{h[0], h[1]};
    f[b] = __builtin_bit_cast(bf16x8_t, pair);
  }
}

// operand traits
template <class L>
struct Op;
template <typename E>
struct Op<KRows2<E>> {
  using Tile = KTile<E>;
  template <int NBLK>
  __device__ __forceinline__ static void read(const char* s, int r0, int lane, int kk, bf16x8_t (&f)[NBLK]) {
    read_k<NBLK>(s, r0, lane, kk, f);
  }
};
template <typename E>
struct Op<ICols2<E>> {
  using Tile = ITile<E>;
  template <int NBLK>
  __device__ __forceinline__ static void read(const char* s, int r0, int lane, int kk, bf16x8_t (&f)[NBLK]) {
    read_i<NBLK>(s, r0, lane, kk, f);
  }
};

__device__ __forceinline__ void wave_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Wait until at most `tiles_after` tiles' copies (PER_TILE per wave each)
// are still in flight.
template <int PER_TILE>
__device__ __forceinline__ void wait_copies_n(int tiles_after) {
  __builtin_amdgcn_sched_barrier(0);
  if (tiles_after >= 3)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * PER_TILE) : "memory");
  else if (tiles_after == 2)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * PER_TILE) : "memory");
  else if (tiles_after == 1)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(PER_TILE) : "memory");
  else
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}
__device__ __forceinline__ void wait_copies(int tiles_after) { wait_copies_n<2 * COPIES>(tiles_after); }

// s_waitcnt vmcnt(N) between scheduling barriers.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Calls f(integral_constant<int, I>) for I = 0 .. N-1 (compile-time unroll).
template <int I, int N, class F>
__device__ __forceinline__ void unroll(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    unroll<I + 1, N>(f);
  }
}

}  // namespace dma

// Registers that an epilogue staging its tile through LDS loads ahead of the
// tile (prefetch, before the last K tile where the engine allows); nothing
// for the element-wise epilogues.
template <class Epi, bool = (Epi::kTileSmem > 0)>
struct EpiPre {
  struct type {};
};
template <class Epi>
struct EpiPre<Epi, true> {
  static_assert(Epi::kThreads == dma::NT, "the tile epilogue maps the engines' 8 waves");
  using type = typename Epi::Pre;
};

template <class AL, class BL, class Epi>
__global__ void __launch_bounds__(dma::NT, 1)
    gemm_bf16_dma(AL al, BL bl, Epi epi, int M, int N, int K, int ktiles_per_split) {
  using namespace dma;
  constexpr int MB = WM / 32, NB = WN / 32;
  // stage s: A tile at s * TILE_BYTES, B tile at (STAGES + s) * TILE_BYTES;
  // a tile epilogue may reuse the whole array after the K loop.
  constexpr int SMEM = Epi::kTileSmem > 2 * STAGES * TILE_BYTES ? Epi::kTileSmem : 2 * STAGES * TILE_BYTES;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  using ATile = typename Op<AL>::Tile;
  using BTile = typename Op<BL>::Tile;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / WAVES_N) * WM, wn0 = (wave % WAVES_N) * WN;
  int tm, tn, split;
  xcd_tile_split(blockIdx.x, blockIdx.z, gridDim.z, (M + BM - 1) / BM, (N + BN - 1) / BN, tm, tn, split);
  const int m0 = tm * BM, n0 = tn * BN;
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
  ta.init(al, m0, wave, lane);
  tb.init(bl, n0, wave, lane);

  // prologue: tiles kt0 .. kt0 + STAGES - 2 into stages 0 .. STAGES - 2
  unroll<0, STAGES - 1>([&](auto I) {
    constexpr int st = decltype(I)::value;
    if (kt0 + st < kt1) {
      ta.issue(al, (kt0 + st) * BK, smem + st * TILE_BYTES, wave);
      tb.issue(bl, (kt0 + st) * BK, smem + (STAGES + st) * TILE_BYTES, wave);
    }
  });

  // one K tile: wait for its copies, barrier, refill the freed stage, multiply
  auto step = [&](int kt, const char* as, const char* bs, char* an, char* bn) {
    wait_copies(min(kt + STAGES - 2, kt1 - 1) - kt);
    wave_barrier();
    if (kt + STAGES - 1 < kt1) {
      ta.issue(al, (kt + STAGES - 1) * BK, an, wave);
      tb.issue(bl, (kt + STAGES - 1) * BK, bn, wave);
    }
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8_t af[MB], bfr[NB];
      Op<AL>::template read<MB>(as, wm0, lane, kk, af);
      Op<BL>::template read<NB>(bs, wn0, lane, kk, bfr);
#pragma unroll
      for (int a = 0; a < MB; ++a)
#pragma unroll
        for (int b = 0; b < NB; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
  };
  // the stage of tile kt is (kt - kt0) % STAGES; unrolling by STAGES keeps
  // every stage address a compile-time constant
  for (int kt = kt0; kt < kt1; kt += STAGES) {
    unroll<0, STAGES>([&](auto I) {
      constexpr int st = decltype(I)::value;
      constexpr int nx = (st + STAGES - 1) % STAGES;  // stage refilled during this step
      if (kt + st < kt1)
        step(kt + st, smem + st * TILE_BYTES, smem + (STAGES + st) * TILE_BYTES, smem + nx * TILE_BYTES,
             smem + (STAGES + nx) * TILE_BYTES);
    });
  }

  if constexpr (Epi::kTileSmem > 0) {
    typename EpiPre<Epi>::type pre;
    epi.prefetch(pre, m0, n0, tid, M);
    wave_barrier();  // every wave is done with the stages
    epi.template tile<MB, NB>(acc, smem, m0, n0, wave / WAVES_N, wn0, lane, tid, M, pre);
  } else {
    store_acc<MB, NB>(epi, acc, m0 + wm0, n0 + wn0, lane, split, M, N, m0 + BM <= M && n0 + BN <= N);
  }
}

template <class AL, class BL, class Epi>
inline void launch_gemm_bf16_dma(const AL& al, const BL& bl, const Epi& epi, int M, int N, int K, int splits,
                                 hipStream_t s) {
  const int nkt = (K + dma::BK - 1) / dma::BK;
  const int kps = (nkt + splits - 1) / splits;
  const unsigned tiles = ((M + 255) / 256) * ((N + 255) / 256);
  hipLaunchKernelGGL((gemm_bf16_dma<AL, BL, Epi>), dim3(tiles, 1, splits), dim3(dma::NT), 0, s, al, bl, epi, M, N,
                     K, kps);
}

}  // namespace o5
