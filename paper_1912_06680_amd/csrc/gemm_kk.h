// bf16 MFMA GEMM for two K-contiguous operands (gfx950):
//   C[i, j] = sum_k A(i, k) * B(j, k)  (+ epilogue), fp32 accumulate.
//
// Block tile 256 x 256, one block per CU.  By default 8 waves (2 x 4) of
// 128 x 64, two per SIMD, so one wave's MFMAs run while the other issues
// copies or waits at a barrier; the alternative of 4 waves of 128 x 128 (one
// per SIMD, each fragment read from LDS feeding four MFMAs) measured a few
// percent slower overall.
//
// Operands go global -> LDS by buffer loads with the LDS flag (16 bytes per
// lane, written at M0 + 16 * lane) through a ring of STAGES stages of BK k.
// With BK = 64 a copy instruction moves 8 rows x 128 bytes, i.e. whole cache
// lines; with BK = 32 it moves 16 half lines, which halves the rate at which
// the L2 feeds the CU.  BK = 64 leaves room for two stages only.  Each lane's
// byte offset into its operand is fixed for the whole K loop and the tile's
// k travels in the scalar offset, so a copy is one s_mov to M0 and one load;
// rows outside the operand get an offset past the buffer and read zeros.
//
// The wave software-pipelines its fragments: those of k step s + 1 are read
// while the MFMAs of step s run.  Before the last k step of tile r the wave
// waits for its own copies of tile r + 1, meets the other waves at the
// barrier (after which the stage of tile r is free: every wave has finished
// reading it), reads the first fragments of tile r + 1, and then issues the
// copies that refill stage r interleaved with its MFMAs (with SPREAD > 1
// also over the first SPREAD - 1 k steps of the next tile; one step measured
// best with two waves per SIMD, two steps with one).  The copies are inline asm, so
// the compiler neither waits for them before LDS reads nor edits the explicit
// waits; each wave issues copies for tiles 0 .. n + STAGES - 2 (those past
// the K range re-read the last tile into a stage no one reads again), so the
// wait counts are constants.
//
// LDS layout of one operand stage: [256 rows][BK k] bf16, the 16-byte chunk
// c of row r stored at slot c ^ ((r / R) % C) with C = BK / 8 chunks per row
// and R = 128 / BK rows per 256 bytes, so the 16 rows of a fragment read
// fall on 16 distinct 16-byte bank groups.
#pragma once

#include "gemm_dma.h"

#ifndef O5_KK_BK
#define O5_KK_BK 64
#endif
#ifndef O5_KK_RING
#define O5_KK_RING 0  // measured a little slower than two stages
#endif

namespace o5 {

namespace kk {

constexpr int BM = 256, BN = 256;
#ifndef O5_KK_WAVES
#define O5_KK_WAVES 8
#endif
// 8 waves (2 x 4) of 128 x 64, two per SIMD (default); or 4 waves (2 x 2) of
// 128 x 128, one per SIMD
constexpr int NWAVES = O5_KK_WAVES;
constexpr int WM = 128, WN = NWAVES == 4 ? 128 : 64, WAVES_N = BN / WN, NT = NWAVES * 64;
constexpr int MB = WM / 32, NB = WN / 32;

template <int BK>
struct Cfg {
  static_assert(BK == 32 || BK == 64, "BK is 32 or 64");
  static constexpr int STAGES = BK == 64 ? 2 : 4;
  // BK = 64 with O5_KK_RING: the operand tiles A_t, B_t take turns in one
  // ring of 5 slots of 32 KB (A_t in slot 2t % 5, B_t in slot (2t + 1) % 5):
  // the barrier of tile t frees the slots of A_t and B_t, which receive
  // B_{t+2} and A_{t+3}, so about one and a half tiles are in flight
  // instead of one, in all 160 KB of LDS
  static constexpr bool RING = BK == 64 && O5_KK_RING;
  static constexpr int ROW_BYTES = BK * 2;
  static constexpr int CPR = BK / 8;                     // 16-byte chunks per row
  static constexpr int RPI = 1024 / ROW_BYTES;           // rows per 1 KB copy
  static constexpr int R256 = 256 / ROW_BYTES;           // rows per 256 bytes
  static constexpr int TILE_BYTES = 256 * ROW_BYTES;     // one operand, one stage
  static constexpr int NC = TILE_BYTES / 1024 / NWAVES;  // copies per wave per operand per tile
  static constexpr int KSTEPS = BK / 16;
  static constexpr int SMEM = RING ? 5 * TILE_BYTES : 2 * STAGES * TILE_BYTES;
};

template <int BK>
__device__ __forceinline__ int slot(int r, int c) {
  using C = Cfg<BK>;
  return c ^ ((r / C::R256) % C::CPR);
}

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

// Per-lane state for copying one operand's 256-row tiles with buffer loads to
// LDS: copy q of wave w fills tile rows (w * NC + q) * RPI .. + RPI - 1; the
// lane fetches the chunk that belongs at slot (lane % CPR) of row (lane /
// CPR).  The lane's byte offset into each source is fixed; the tile's k moves
// in the scalar offset, so a copy is one s_mov and one buffer load.  Rows past
// the operand, and masked rows of the second source, get an offset past the
// buffer and so read zeros.  Requires K0 and K multiples of BK (no tile
// straddles a source boundary or the end) and sources below 2^31 bytes.
template <typename E, int BK>
struct Tile {
  using C = Cfg<BK>;
  rsrc_t rs0, rs1;
  uint32_t voff0[C::NC], voff1[C::NC];
  int K0, kmax;

  __device__ __forceinline__ void init(const KRows2<E>& l, int row0, int wave, int lane) {
    K0 = l.K0;
    kmax = l.K - BK;
    rs0 = make_rsrc(l.p0, static_cast<uint32_t>(static_cast<size_t>(l.rows) * l.ld0 * sizeof(E)));
    rs1 = make_rsrc(l.p1 != nullptr ? l.p1 : l.p0,
                    l.p1 != nullptr ? static_cast<uint32_t>(static_cast<size_t>(l.rows) * l.ld1 * sizeof(E)) : 0u);
#pragma unroll
    for (int q = 0; q < C::NC; ++q) {
      const int r = (wave * C::NC + q) * C::RPI + lane / C::CPR;  // tile row this lane fills
      const int row = l.gstride > 0 ? (r >> 6) * l.gstride + (row0 >> 2) + (r & 63) : row0 + r;
      const uint32_t koff = slot<BK>(r, lane % C::CPR) * 16;
      const bool valid = row < l.rows;
      const bool masked = valid && l.mask1 != nullptr && l.mask1[row] != 0;
      voff0[q] = valid ? static_cast<uint32_t>(row) * l.ld0 * sizeof(E) + koff : kOutOfRange;
      voff1[q] = (valid && !masked && l.p1 != nullptr) ? static_cast<uint32_t>(row) * l.ld1 * sizeof(E) + koff
                                                        : kOutOfRange;
    }
  }
  // copy q of the tile starting at k0 into the stage at LDS address `stage`;
  // tiles past the end (the ring's trailing copies) re-read the last tile into
  // a stage no one reads
  __device__ __forceinline__ void issue_one(int k0, uint32_t stage, int wave, int q) const {
    k0 = min(k0, kmax);
    const bool seg0 = k0 < K0;
    const uint32_t soff = static_cast<uint32_t>(seg0 ? k0 : k0 - K0) * sizeof(E);
    const uint32_t voff = seg0 ? voff0[q] : voff1[q];
    const rsrc_t rs = seg0 ? rs0 : rs1;
    const uint32_t lds = stage + (wave * C::NC + q) * 1024;
    // (s_nop: one wait state between the M0 write and the LDS DMA reading it)
    asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(voff), "s"(rs), "s"(soff),
                 "s"(lds)
                 : "memory", "m0");
  }
  __device__ __forceinline__ void issue(int k0, uint32_t stage, int wave) const {
#pragma unroll
    for (int q = 0; q < C::NC; ++q) issue_one(k0, stage, wave, q);
  }
};

struct Frags {
  bf16x8_t a[MB], b[NB];
};

// Fragments of k step s (16 k) for the wave's 128 x 128 tile: lane l holds row
// (l & 31) of each 32-row block and the 8 k values 8 * (l >> 5) .. + 7.
template <int BK, int NBLK>
__device__ __forceinline__ void read_rows(const char* stage, int row0, int lane, int s, bf16x8_t (&f)[NBLK]) {
  const int c = s * 2 + (lane >> 5);
#pragma unroll
  for (int b = 0; b < NBLK; ++b) {
    const int r = row0 + b * 32 + (lane & 31);
    f[b] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(stage + r * (BK * 2) + slot<BK>(r, c) * 16));
  }
}

template <int BK>
__device__ __forceinline__ void read(const char* as, const char* bs, int wm0, int wn0, int lane, int s, Frags& f) {
  read_rows<BK, MB>(as, wm0, lane, s, f.a);
  read_rows<BK, NB>(bs, wn0, lane, s, f.b);
}

__device__ __forceinline__ void mfma_all(const Frags& f, f32x16_t (&acc)[MB][NB]) {
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[a], f.b[b], acc[a][b], 0, 0, 0);
}

// The same MFMAs with the wave's copies of a B tile (k kb, LDS address bs)
// and then an A tile (ka, as) spread evenly among them (the order is pinned
// by scheduling barriers; the waits count on B's copies being older).
template <typename E, int BK>
__device__ __forceinline__ void mfma_copies(const Frags& f, f32x16_t (&acc)[MB][NB], const Tile<E, BK>& ta,
                                            const Tile<E, BK>& tb, int ka, uint32_t as, int kb, uint32_t bs,
                                            int wave) {
  constexpr int NC = Cfg<BK>::NC;
  constexpr int NQ = 2 * NC;
  dma::unroll<0, MB * NB>([&](auto I) {
    constexpr int m = decltype(I)::value;
    constexpr int a = m / NB, b = m % NB;
    acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[a], f.b[b], acc[a][b], 0, 0, 0);
    // copies after MFMA m: those q with floor(q * MB * NB / NQ) == m
    dma::unroll<0, NQ>([&](auto J) {
      constexpr int q = decltype(J)::value;
      if constexpr (q * MB * NB / NQ == m) {
        if constexpr (q < NC)
          tb.issue_one(kb, bs, wave, q);
        else
          ta.issue_one(ka, as, wave, q - NC);
      }
    });
    __builtin_amdgcn_sched_barrier(0);
  });
}

}  // namespace kk

template <int BK, class Epi, typename E>
__global__ void __launch_bounds__(kk::NT, 1)
    gemm_kk(KRows2<E> al, KRows2<E> bl, Epi epi, int M, int N, int K, int ktiles_per_split) {
  using namespace kk;
  using C = Cfg<BK>;
  constexpr int STAGES = C::STAGES, TB = C::TILE_BYTES, KS = C::KSTEPS, NC = C::NC;
  constexpr bool RING = C::RING;
  static_assert(sizeof(E) == 2, "bf16 operands only");
  static_assert(KS % 2 == 0, "the fragment double buffer assumes an even number of k steps");
  constexpr int SMEM = Epi::kTileSmem > C::SMEM ? Epi::kTileSmem : C::SMEM;
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / WAVES_N) * WM, wn0 = (wave % WAVES_N) * WN;
  int tm, tn;
  xcd_tile(blockIdx.x, (M + BM - 1) / BM, (N + BN - 1) / BN, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int split = blockIdx.z;
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

  if (n > 0) {
    Tile<E, BK> ta, tb;
    ta.init(al, m0, wave, lane);
    tb.init(bl, n0, wave, lane);
    // LDS byte offset of A_t and B_t (t relative to the split's first tile)
    auto aoff = [&](int t) { return RING ? ((2 * t) % 5) * TB : (t % STAGES) * TB; };
    auto boff = [&](int t) { return RING ? ((2 * t + 1) % 5) * TB : (STAGES + t % STAGES) * TB; };
    // the same memory as an LDS address, for the copies' M0
    const uint32_t l0 = static_cast<uint32_t>(reinterpret_cast<size_t>((__attribute__((address_space(3))) char*)smem));
    auto copy_a = [&](int t) { ta.issue((kt0 + t) * BK, l0 + aoff(t), wave); };
    auto copy_b = [&](int t) { tb.issue((kt0 + t) * BK, l0 + boff(t), wave); };

    // Prologue.  Stages: tiles 0 .. STAGES-2, wait for tile 0, tile
    // STAGES-1.  Ring: A0 B0 A1 B1 A2, wait for B0.  In both cases the copies
    // still allowed in flight at every later wait are a fixed count: WAIT.
    constexpr int WAIT = RING ? NC : (STAGES - 2) * 2 * NC;
    if constexpr (RING) {
      copy_a(0);
      copy_b(0);
      copy_a(1);
      copy_b(1);
      copy_a(2);
      dma::wait_copies_n<NC>(3);
      dma::wave_barrier();
    } else {
#pragma unroll
      for (int t = 0; t < STAGES - 1; ++t) {
        copy_a(t);
        copy_b(t);
      }
      dma::wait_copies_n<2 * NC>(STAGES - 2);
      dma::wave_barrier();
      copy_a(STAGES - 1);
      copy_b(STAGES - 1);
    }
    Frags f[2];
    read<BK>(smem + aoff(0), smem + boff(0), wm0, wn0, lane, 0, f[0]);

    for (int r = 0; r < n - 1; ++r) {
      const int ao = aoff(r), bo = boff(r);
      // k steps 0 .. KS-2 of tile r, each with the next step's fragments in flight
      dma::unroll<0, KS - 1>([&](auto S) {
        constexpr int s = decltype(S)::value;
        read<BK>(smem + ao, smem + bo, wm0, wn0, lane, s + 1, f[(s + 1) & 1]);
        __builtin_amdgcn_sched_group_barrier(0x100, MB + NB, 0);  // the LDS reads first
        __builtin_amdgcn_sched_group_barrier(0x008, MB * NB, 0);  // then the MFMAs
        mfma_all(f[s & 1], acc);
        __builtin_amdgcn_sched_barrier(0);
      });
      // every wave done reading tile r; tile r + 1 landed
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      dma::vm_wait<WAIT>();
      dma::wave_barrier();
      read<BK>(smem + aoff(r + 1), smem + boff(r + 1), wm0, wn0, lane, 0, f[0]);
      __builtin_amdgcn_sched_barrier(0);
      // last k step of tile r; the slots of tile r refill (stages: with tile
      // r + STAGES; ring: with B_{r+2} and A_{r+3})
      if constexpr (RING)
        mfma_copies<E, BK>(f[1], acc, ta, tb, (kt0 + r + 3) * BK, l0 + aoff(r + 3), (kt0 + r + 2) * BK,
                           l0 + boff(r + 2), wave);
      else
        mfma_copies<E, BK>(f[1], acc, ta, tb, (kt0 + r + STAGES) * BK, l0 + aoff(r + STAGES),
                           (kt0 + r + STAGES) * BK, l0 + boff(r + STAGES), wave);
    }
    {
      // the last tile; its first fragments are in f[0]
      const int ao = aoff(n - 1), bo = boff(n - 1);
      dma::unroll<0, KS>([&](auto S) {
        constexpr int s = decltype(S)::value;
        if constexpr (s + 1 < KS) read<BK>(smem + ao, smem + bo, wm0, wn0, lane, s + 1, f[(s + 1) & 1]);
        mfma_all(f[s & 1], acc);
      });
    }
    dma::vm_wait<0>();  // no copy outlives the loop
  }

  if constexpr (Epi::kTileSmem > 0) {
    dma::wave_barrier();  // every wave is done with the stages
    epi.template tile<MB, NB>(acc, smem, m0, n0, wave / WAVES_N, wn0, lane, tid, M);
  } else {
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
}

template <class Epi, typename E>
inline void launch_gemm_kk(const KRows2<E>& al, const KRows2<E>& bl, const Epi& epi, int M, int N, int K, int splits,
                           hipStream_t s) {
  constexpr int BK = O5_KK_BK;
  const int nkt = (K + BK - 1) / BK;
  const int kps = (nkt + splits - 1) / splits;
  const unsigned tiles = ((M + kk::BM - 1) / kk::BM) * ((N + kk::BN - 1) / kk::BN);
  hipLaunchKernelGGL((gemm_kk<BK, Epi, E>), dim3(tiles, 1, splits), dim3(kk::NT), 0, s, al, bl, epi, M, N, K, kps);
}

// Operands the buffer-load copies can take: K and the source split K0 whole
// tiles, every source below 2^31 bytes.
template <typename E>
inline bool kk_fits(const KRows2<E>& l) {
  constexpr int BK = O5_KK_BK;
  const size_t b0 = static_cast<size_t>(l.rows) * l.ld0 * sizeof(E);
  const size_t b1 = l.p1 != nullptr ? static_cast<size_t>(l.rows) * l.ld1 * sizeof(E) : 0;
  return l.K >= BK && l.K % BK == 0 && l.K0 % BK == 0 && b0 < (size_t{1} << 31) && b1 < (size_t{1} << 31);
}

// The K-contiguous engine is the default for two K-contiguous bf16 operands;
// O5_GEMM_ENGINE=dma selects the 8-wave direct-to-LDS engine instead.
inline bool kk_engine_enabled() {
  static const bool v = [] {
    const char* e = std::getenv("O5_GEMM_ENGINE");
    return !(e && e[0] == 'd');
  }();
  return v;
}

}  // namespace o5
