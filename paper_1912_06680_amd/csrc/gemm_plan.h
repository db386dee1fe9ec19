// GEMM planning and dispatch: engine, tile and split-K for a problem shape.
#pragma once

#include <type_traits>

#include "gemm_kk.h"

namespace o5 {

// --------------------------------------------------------------- planning

struct GemmPlan {
  bool bf16;
  BfTile tile;
  int splits;
  int bn;  // column tile of the K-contiguous engine: 256 or 128
};

inline int cdiv(long long a, long long b) { return static_cast<int>((a + b - 1) / b); }

// Choose engine, tile and split-K so the launch has >= ~256 blocks (one per
// CU) while every split keeps a reasonable number of K tiles.  256 x 128
// tiles replace 256 x 256 ones where half of a 256-wide column tile would be
// padding.  (They do not replace a K split: at M = 2048, N = 4096, K = 16384,
// 256 x 128 tiles without a split ran at 0.88 PFLOP/s against 1.21 for 256 x
// 256 tiles split in two, the narrower tile needing 1.5x the operand bytes
// per MFMA.)
inline GemmPlan plan_gemm(bool bf16, int M, int N, int K) {
  GemmPlan p{bf16, BfTile::kDma256, 1, 256};
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
    const bool narrow = N % 256 != 0 && N % 256 <= 128;
    p.bn = narrow ? 128 : 256;
    const int t = p.bn == 128 ? cdiv(M, 256) * cdiv(N, 128) : t256;
    int s = cdiv(256, t);
    s = std::min(s, std::max(1, nkt / 16));
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

// The direct-to-LDS engine takes I-contiguous operands without a mask only.
template <class L>
inline bool dma_ok(const L&) { return true; }
template <typename E>
inline bool dma_ok(const ICols2<E>& l) { return l.mask1 == nullptr; }

template <class AL, class BL, class Epi>
inline void run_gemm(const GemmPlan& p, const AL& al, const BL& bl, const Epi& epi, int M, int N, int K,
                     hipStream_t s) {
  if constexpr (AL::kBf16 && BL::kBf16) {
    if (p.bf16) {
      if constexpr (std::is_same_v<AL, KRows2<uint16_t>> && std::is_same_v<BL, KRows2<uint16_t>>) {
        if (p.tile == BfTile::kDma256 && kk_fits(al) && kk_fits(bl)) {
          if (p.bn == 128)
            launch_gemm_kk<128>(al, bl, epi, M, N, K, p.splits, s);
          else
            launch_gemm_kk<256>(al, bl, epi, M, N, K, p.splits, s);
          return;
        }
      }
      if (p.tile == BfTile::kDma256 && dma_ok(al) && dma_ok(bl)) {
        launch_gemm_bf16_dma(al, bl, epi, M, N, K, p.splits, s);
        return;
      }
      launch_gemm_bf16(al, bl, epi, M, N, K, p.splits,
                       p.tile == BfTile::kDma256 ? BfTile::k256x256w8 : p.tile, s);
      return;
    }
  }
  launch_gemm_f32(al, bl, epi, M, N, K, p.splits, s);
}

}  // namespace o5
