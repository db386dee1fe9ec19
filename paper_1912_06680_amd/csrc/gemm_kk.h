// bf16 MFMA GEMM for two K-contiguous operands (gfx950):
//   C[i, j] = sum_k A(i, k) * B(j, k)  (+ epilogue), fp32 accumulate.
//
// Block tile 256 x BN (BN = 256, or 128 where 256 x 256 tiles would need a
// K split to fill the chip), one block per CU, 8 waves, two per SIMD, so one
// wave's MFMAs run while the other issues copies or waits at a barrier: 2 x 4
// waves of 128 x 64 for BN = 256, 4 x 2 waves of 64 x 64 for BN = 128.  (4
// waves of 128 x 128, one per SIMD, each fragment read from LDS feeding four
// MFMAs, measured a few percent slower overall.)
//
// Operands go global -> LDS by buffer loads with the LDS flag (16 bytes per
// lane, written at M0 + 16 * lane) through stages of BK = 64 k (for 256 x
// 256 tiles two of A and three of B, 32 KB each; for 256 x 128 tiles three
// of each): a copy
// instruction moves 8 rows x 128 bytes, i.e. whole cache lines (stages of 32
// k move 16 half lines, which halves the rate at which the L2 feeds the CU;
// a ring of more, smaller slots measured slower).  Each lane's byte offset
// into its operand is fixed for the whole K loop and the tile's k travels in
// the scalar offset, so a copy is one s_mov to M0 and one load; rows outside
// the operand get an offset past the buffer and read zeros.
//
// The wave software-pipelines its fragments: those of k step s + 1 are read
// while the MFMAs of step s run.  Before the last k step of tile r the wave
// waits for its own copies of tile r + 1 (those of later tiles may stay in
// flight), meets the other waves at the barrier (after which the stages of
// tile r are free: every wave has finished reading them), reads the first
// fragments of tile r + 1, and then issues the copies that refill them with
// A tile r + NSA and B tile r + NSB, interleaved with the MFMAs of that last
// k step.  The copies are inline asm, so the compiler neither waits for them
// before LDS reads nor edits the explicit waits; copies past the K range
// re-read the last tile into stages no one reads again.
//
// LDS layout of one operand stage: [rows][64 k] bf16, the 16-byte chunk c of
// row r stored at slot c ^ ((r / 2) % 8), so the 16 rows of a fragment read
// fall on 16 distinct 16-byte bank groups.
#pragma once

#include "gemm_dma.h"

namespace o5 {

namespace kk {

constexpr int BK = 64;                 // k per stage
constexpr int KSTEPS = BK / 16;        // MFMA k steps per stage
constexpr int ROW_BYTES = BK * 2;      // one stage row
constexpr int CPR = BK / 8;            // 16-byte chunks per row
constexpr int RPI = 1024 / ROW_BYTES;  // rows per 1 KB copy
constexpr int R256 = 256 / ROW_BYTES;  // rows per 256 bytes
constexpr int NWAVES = 8;              // two per SIMD
constexpr int NT = NWAVES * 64;

// Block and wave tiling of a 256 x BN block tile: 256 x 256 (2 x 4 waves of
// 128 x 64) or 256 x 128 (4 x 2 waves of 64 x 64).
template <int BN_>
struct Shape {
  static_assert(BN_ == 256 || BN_ == 128, "BN is 256 or 128");
  static_assert(NWAVES == 8, "8 waves");
  static constexpr int BM = 256, BN = BN_;
  static constexpr int WAVES_M = BN == 128 ? 4 : 2;
  static constexpr int WAVES_N = NWAVES / WAVES_M;
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int MB = WM / 32, NB = WN / 32;  // 32 x 32 MFMA blocks per wave
  static constexpr int TA = BM * ROW_BYTES;        // A stage bytes
  static constexpr int TB = BN * ROW_BYTES;        // B stage bytes
  static constexpr int NCA = TA / 1024 / NWAVES;   // copies per wave per A tile
  static constexpr int NCB = TB / 1024 / NWAVES;   // copies per wave per B tile
  // stages per operand: with NS of them, NS - 1 tiles' copies are in
  // flight while one is read.  256 x 128 tiles: three of each (48 KB per
  // stage pair); 256 x 256 tiles: two of A and three of B, 32 KB each,
  // which fills the 160 KB (a third B stage: forward GEMM 471 against 478
  // us, weight gradient 6.69 against 6.76 ms)
  static constexpr int NSA = BN == 128 ? 3 : 2;
  static constexpr int NSB = 3;
  static_assert(NSB >= NSA && NSB <= NSA + 1, "the wait below assumes NSA <= NSB <= NSA + 1");
  static constexpr int SMEM = NSA * TA + NSB * TB;
  static_assert(SMEM <= 160 * 1024, "LDS");
};

__device__ __forceinline__ int slot(int r, int c) { return c ^ ((r / R256) % CPR); }

typedef int rsrc_t __attribute__((ext_vector_type(4)));

// Buffer resource for bytes [base, base + bytes): raw (stride 0), 32-bit
// words, out-of-range reads return zero.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  rsrc_t r;
  r.x = static_cast<int>(static_cast<uint32_t>(b));
  r.y = static_cast<int>(static_cast<uint32_t>(b >> 32) & 0xffffu);
  r.z = static_cast<int>(bytes);
  r.w = 0x00020000;
  return r;
}

constexpr uint32_t kOutOfRange = 0xfffffff0u;  // a byte offset past every operand buffer

// Per-lane state for copying one operand's tiles with buffer loads to LDS,
// NC copies of 1 KB per wave and tile: copy q of wave w fills tile rows (w *
// NC + q) * RPI .. + RPI - 1; the lane fetches the chunk that belongs at slot
// (lane % CPR) of row (lane / CPR).  The lane's byte offset into each source
// is fixed; the tile's k moves in the scalar offset.  Rows past the operand,
// and masked rows of the second source, get an offset past the buffer and so
// read zeros.  Requires K0 and K multiples of BK (no tile straddles a source
// boundary or the end) and sources below 2^31 bytes.
template <typename E, int NC, bool TWO>
struct Tile {
  rsrc_t rs0, rs1;
  uint32_t voff0[NC], voff1[TWO ? NC : 1];  // (TWO: the operand has a second source)
  int K0, kmax;

  __device__ __forceinline__ void init(const KRows2<E>& l, int row0, int wave, int lane) {
    K0 = l.K0;
    kmax = l.K - BK;
    rs0 = make_rsrc(l.p0, static_cast<uint32_t>(static_cast<size_t>(l.rows) * l.ld0 * sizeof(E)));
    if constexpr (TWO)
      rs1 = make_rsrc(l.p1 != nullptr ? l.p1 : l.p0,
                      l.p1 != nullptr ? static_cast<uint32_t>(static_cast<size_t>(l.rows) * l.ld1 * sizeof(E)) : 0u);
#pragma unroll
    for (int q = 0; q < NC; ++q) {
      const int r = (wave * NC + q) * RPI + lane / CPR;  // tile row this lane fills
      const int row = l.gstride > 0 ? (r >> 6) * l.gstride + (row0 >> 2) + (r & 63) : row0 + r;
      const uint32_t koff = slot(r, lane % CPR) * 16;
      const bool valid = row < l.rows;
      voff0[q] = valid ? static_cast<uint32_t>(row) * l.ld0 * sizeof(E) + koff : kOutOfRange;
      if constexpr (TWO) {
        const bool masked = valid && l.mask1 != nullptr && l.mask1[row] != 0;
        voff1[q] = (valid && !masked && l.p1 != nullptr) ? static_cast<uint32_t>(row) * l.ld1 * sizeof(E) + koff
                                                          : kOutOfRange;
      }
    }
  }
  // copy q of the tile starting at k0 into the stage at LDS address `stage`;
  // a tile past the end re-reads the last tile
  __device__ __forceinline__ void issue_one(int k0, uint32_t stage, int wave, int q) const {
    k0 = min(k0, kmax);
    uint32_t soff, voff;
    rsrc_t rs;
    if constexpr (TWO) {
      const bool seg0 = k0 < K0;
      soff = static_cast<uint32_t>(seg0 ? k0 : k0 - K0) * sizeof(E);
      voff = seg0 ? voff0[q] : voff1[q];
      rs = seg0 ? rs0 : rs1;
    } else {
      soff = static_cast<uint32_t>(k0) * sizeof(E);
      voff = voff0[q];
      rs = rs0;
    }
    const uint32_t lds = stage + (wave * NC + q) * 1024;
    // (s_nop: one wait state between the M0 write and the LDS DMA reading it)
    asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(voff), "s"(rs),
                 "s"(soff), "s"(lds)
                 : "memory", "m0");
  }
  __device__ __forceinline__ void issue(int k0, uint32_t stage, int wave) const {
#pragma unroll
    for (int q = 0; q < NC; ++q) issue_one(k0, stage, wave, q);
  }
};

template <int MB, int NB>
struct Frags {
  bf16x8_t a[MB], b[NB];
};

// The fragment of k step s (16 k) for the 32-row block at row0: lane l holds
// row row0 + (l & 31) and the 8 k values 8 * (l >> 5) .. + 7 of the step.
__device__ __forceinline__ bf16x8_t read_frag(const char* stage, int row0, int lane, int s) {
  const int c = s * 2 + (lane >> 5);
  const int r = row0 + (lane & 31);
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(stage + r * ROW_BYTES + slot(r, c) * 16));
}

// The same for NBLK 32-row blocks from row0.
template <int NBLK>
__device__ __forceinline__ void read_rows(const char* stage, int row0, int lane, int s, bf16x8_t (&f)[NBLK]) {
#pragma unroll
  for (int b = 0; b < NBLK; ++b) f[b] = read_frag(stage, row0 + b * 32, lane, s);
}

template <int MB, int NB>
__device__ __forceinline__ void read(const char* as, const char* bs, int wm0, int wn0, int lane, int s,
                                     Frags<MB, NB>& f) {
  read_rows<MB>(as, wm0, lane, s, f.a);
  read_rows<NB>(bs, wn0, lane, s, f.b);
}

// Fragment I alone of the same: A block I for I < MB, else B block I - MB.
template <int I, int MB, int NB>
__device__ __forceinline__ void read_one(const char* as, const char* bs, int wm0, int wn0, int lane, int s,
                                         Frags<MB, NB>& f) {
  if constexpr (I < MB)
    f.a[I] = read_frag(as, wm0 + I * 32, lane, s);
  else
    f.b[I - MB] = read_frag(bs, wn0 + (I - MB) * 32, lane, s);
}

template <int MB, int NB>
__device__ __forceinline__ void mfma_all(const Frags<MB, NB>& f, f32x16_t (&acc)[MB][NB]) {
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[a], f.b[b], acc[a][b], 0, 0, 0);
}

// The same MFMAs with the wave's copies of one A and one B tile (k0, stages
// as and bs) spread evenly among them, and after each of the first MB + NB
// MFMAs one LDS read of the next tile's first fragments (from na and nb into
// nf; forward GEMM 446 against 451 us with those reads ahead of the MFMAs);
// the order is pinned by scheduling barriers.
template <typename E, int MB, int NB, int NCA, int NCB, bool TWO>
__device__ __forceinline__ void mfma_copies(const Frags<MB, NB>& f, f32x16_t (&acc)[MB][NB],
                                            const Tile<E, NCA, TWO>& ta, const Tile<E, NCB, TWO>& tb, int k0a,
                                            int k0b, uint32_t as, uint32_t bs, int wave, const char* na,
                                            const char* nb, int wm0, int wn0, int lane, Frags<MB, NB>& nf) {
  constexpr int NQ = NCA + NCB;
  dma::unroll<0, MB * NB>([&](auto I) {
    constexpr int m = decltype(I)::value;
    constexpr int a = m / NB, b = m % NB;
    acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[a], f.b[b], acc[a][b], 0, 0, 0);
    if constexpr (m < MB + NB) read_one<m>(na, nb, wm0, wn0, lane, 0, nf);
    // copies after MFMA m: those q with floor(q * MB * NB / NQ) == m
    dma::unroll<0, NQ>([&](auto J) {
      constexpr int q = decltype(J)::value;
      if constexpr (q * MB * NB / NQ == m) {
        if constexpr (q < NCA)
          ta.issue_one(k0a, as, wave, q);
        else
          tb.issue_one(k0b, bs, wave, q - NCA);
      }
    });
    __builtin_amdgcn_sched_barrier(0);
  });
}

}  // namespace kk

template <int BN, bool TWO, class Epi, typename E>
__global__ void __launch_bounds__(kk::NT, 1)
    gemm_kk(KRows2<E> al, KRows2<E> bl, Epi epi, int M, int N, int K, int ktiles_per_split) {
  using namespace kk;
  using S = Shape<BN>;
  constexpr int BM = S::BM, MB = S::MB, NB = S::NB, WM = S::WM, WN = S::WN, WAVES_N = S::WAVES_N;
  constexpr int TA = S::TA, TB = S::TB;
  static_assert(sizeof(E) == 2, "bf16 operands only");
  static_assert(NT == dma::NT, "tile epilogues assume the 8 waves of both engines");
  static_assert(KSTEPS % 2 == 0, "the fragment double buffer assumes an even number of k steps");
  static_assert(MB * NB >= MB + NB, "a wave's MFMAs of a k step outnumber its fragment reads");
  constexpr int SMEM = Epi::kTileSmem > S::SMEM ? Epi::kTileSmem : S::SMEM;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / WAVES_N) * WM, wn0 = (wave % WAVES_N) * WN;
  int tm, tn, split;
  xcd_tile_split(blockIdx.x, blockIdx.z, gridDim.z, (M + BM - 1) / BM, (N + BN - 1) / BN, tm, tn, split);
  const int m0 = tm * BM, n0 = tn * BN;
  const int nkt = (K + BK - 1) / BK;
  const int kt0 = split * ktiles_per_split;
  const int n = min(nkt, kt0 + ktiles_per_split) - kt0;  // K tiles of this split

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.0f;
  typename EpiPre<Epi>::type pre;  // what the epilogue loads ahead

  if (n > 0) {
    Tile<E, S::NCA, TWO> ta;
    Tile<E, S::NCB, TWO> tb;
    ta.init(al, m0, wave, lane);
    tb.init(bl, n0, wave, lane);
    // stage t % NSA of A at (t % NSA) * TA, of B at NSA * TA + (t % NSB) * TB
    constexpr int NSA = S::NSA, NSB = S::NSB;
    // copies a wave may leave in flight when it waits for a tile: those of
    // the NSA - 2 A tiles and NSB - 2 B tiles issued after it (each
    // iteration issues its A copies, then its B copies)
    constexpr int AHEAD = (NSA - 2) * S::NCA + (NSB - 2) * S::NCB;
    auto aoff = [&](int t) { return (t % NSA) * TA; };
    auto boff = [&](int t) { return NSA * TA + (t % NSB) * TB; };
    // the same memory as an LDS address, for the copies' M0
    const uint32_t l0 = static_cast<uint32_t>(reinterpret_cast<size_t>((__attribute__((address_space(3))) char*)smem));

    // prologue: A tiles 0 .. NSA - 2 and B tiles 0 .. NSB - 2 (A, then B,
    // per tile), wait for tile 0, barrier, A tile NSA - 1 and B tile
    // NSB - 1, first fragments
#pragma unroll
    for (int t = 0; t + 1 < NSB; ++t) {
      if (t + 1 < NSA) ta.issue((kt0 + t) * BK, l0 + aoff(t), wave);
      tb.issue((kt0 + t) * BK, l0 + boff(t), wave);
    }
    dma::vm_wait<AHEAD>();
    dma::wave_barrier();
    ta.issue((kt0 + NSA - 1) * BK, l0 + aoff(NSA - 1), wave);
    tb.issue((kt0 + NSB - 1) * BK, l0 + boff(NSB - 1), wave);
    Frags<MB, NB> f[2];
    read(smem + aoff(0), smem + boff(0), wm0, wn0, lane, 0, f[0]);

    for (int r = 0; r < n - 1; ++r) {
      const int ao = aoff(r), bo = boff(r);
      // k steps 0 .. KSTEPS-2 of tile r, each with the next step's fragments in flight
      dma::unroll<0, KSTEPS - 1>([&](auto Sx) {
        constexpr int s = decltype(Sx)::value;
        read(smem + ao, smem + bo, wm0, wn0, lane, s + 1, f[(s + 1) & 1]);
        // one MFMA, then one of the next step's LDS reads, in turn (forward
        // GEMM 451 against 458 us with all reads ahead of the MFMAs), then
        // the remaining MFMAs
        dma::unroll<0, MB + NB>([&](auto) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        });
        if constexpr (MB * NB > MB + NB) __builtin_amdgcn_sched_group_barrier(0x008, MB * NB - (MB + NB), 0);
        mfma_all(f[s & 1], acc);
        __builtin_amdgcn_sched_barrier(0);
      });
      // every wave done reading tile r; tile r + 1 landed (the copies of
      // later tiles may still be in flight)
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      dma::vm_wait<AHEAD>();
      dma::wave_barrier();
      __builtin_amdgcn_sched_barrier(0);
      // last k step of tile r, reading tile r + 1's first fragments; its
      // stages refill with A tile r + NSA and B tile r + NSB
      mfma_copies<E>(f[1], acc, ta, tb, (kt0 + r + NSA) * BK, (kt0 + r + NSB) * BK, l0 + ao, l0 + bo, wave,
                     smem + aoff(r + 1), smem + boff(r + 1), wm0, wn0, lane, f[0]);
    }
    // the epilogue's own loads overlap the last tile's MFMAs (the wait
    // below covers them)
    if constexpr (Epi::kTileSmem > 0) epi.prefetch(pre, m0, n0, tid, M);
    {
      // the last tile; its first fragments are in f[0]
      const int ao = aoff(n - 1), bo = boff(n - 1);
      dma::unroll<0, KSTEPS>([&](auto Sx) {
        constexpr int s = decltype(Sx)::value;
        if constexpr (s + 1 < KSTEPS) read(smem + ao, smem + bo, wm0, wn0, lane, s + 1, f[(s + 1) & 1]);
        mfma_all(f[s & 1], acc);
      });
    }
    dma::vm_wait<0>();  // no copy outlives the loop
  } else if constexpr (Epi::kTileSmem > 0) {
    epi.prefetch(pre, m0, n0, tid, M);
  }

  if constexpr (Epi::kTileSmem > 0) {
    dma::wave_barrier();  // every wave is done with the stages
    epi.template tile<MB, NB>(acc, smem, m0, n0, wave / WAVES_N, wn0, lane, tid, M, pre);
  } else {
    store_acc<MB, NB>(epi, acc, m0 + wm0, n0 + wn0, lane, split, M, N, m0 + BM <= M && n0 + BN <= N);
  }
}

template <int BN = 256, class Epi, typename E>
inline void launch_gemm_kk(const KRows2<E>& al, const KRows2<E>& bl, const Epi& epi, int M, int N, int K, int splits,
                           hipStream_t s) {
  const int nkt = (K + kk::BK - 1) / kk::BK;
  const int kps = (nkt + splits - 1) / splits;
  const unsigned tiles = ((M + 255) / 256) * ((N + BN - 1) / BN);
  // operands with a second source (or a row mask) take the two-source copies
  if (al.p1 != nullptr || bl.p1 != nullptr || al.mask1 != nullptr || bl.mask1 != nullptr)
    hipLaunchKernelGGL((gemm_kk<BN, true, Epi, E>), dim3(tiles, 1, splits), dim3(kk::NT), 0, s, al, bl, epi, M, N, K,
                       kps);
  else
    hipLaunchKernelGGL((gemm_kk<BN, false, Epi, E>), dim3(tiles, 1, splits), dim3(kk::NT), 0, s, al, bl, epi, M, N, K,
                       kps);
}

// Operands the buffer-load copies can take: K and the source split K0 whole
// tiles, every source below 2^31 bytes.
template <typename E>
inline bool kk_fits(const KRows2<E>& l) {
  const size_t b0 = static_cast<size_t>(l.rows) * l.ld0 * sizeof(E);
  const size_t b1 = l.p1 != nullptr ? static_cast<size_t>(l.rows) * l.ld1 * sizeof(E) : 0;
  return l.K >= kk::BK && l.K % kk::BK == 0 && l.K0 % kk::BK == 0 && b0 < (size_t{1} << 31) &&
         b1 < (size_t{1} << 31);
}

}  // namespace o5
