// Policy and value heads, PPO clipped-surrogate loss, value loss and entropy
// bonus, and their gradients (appendix "Neural Network Architecture":
// linear projections of the LSTM state for the action logits and the value,
// sharing the network and its gradients; appendix "Action Space": factorised
// action, ignored parameter heads masked out of the optimisation;
// subsection "Optimizing the Policy" and Table "Hyperparameters": clip 0.2,
// value loss weight 1.0; appendix "Exploration": entropy bonus 0.01).
//
//   z   = h Wp^T                        GEMM  (M = N rows, N = A+1, K = H)
//   row kernel (one wave per row): + bp, per-head log-softmax over the
//        available logits, joint log-ratio, clipped surrogate, value error,
//        entropy -> dz [N, A+1],
//        and per-block partial sums of dz (for dbp) and of the row stats
//   dh  = dz Wp                         GEMM  (M = N, N = H, K = A+1)
//   dWp = dz^T h                        GEMM  (M = A+1, N = H, K = N), split-K
//   dbp, stats: fixed-order sums of the block partials.
// On the bf16 path the two gradient products run on the MFMA engine: dz is
// written as a pair of bf16 terms hi = bf16(dz), lo = bf16(dz - hi) (relative
// error ~2^-16) laid side by side along K, against the bf16 operand repeated
// twice, so the product keeps nearly fp32 accuracy.  For dWp the row kernel
// also writes the pair transposed ([hi rows; lo rows] x N, K-contiguous), so h
// is read once: dWp = sum of the hi and lo halves of [hi; lo] h.
// Every reduction has a fixed order, so results are bitwise reproducible.
#include "gemm_plan.h"
#include "heads.h"
#include "reduce.h"

namespace o5 {

constexpr int kStatCols = 8;

// The logits store: an EpiStoreF32 under its own type name, so the heads
// GEMM is a kernel symbol of its own in profiles.
struct EpiLogits : EpiStoreF32 {};

constexpr int kRowsPerWave = 4;
constexpr int kWavesPerBlock = 8;
constexpr int kRowsPerBlock = kRowsPerWave * kWavesPerBlock;

// Read in place of an absent availability mask, head mask and unit-head
// logits.
__device__ const uint8_t kAllAvailable = 1;
__device__ const float kNoLogit = 0.0f;

// The head of each logit column a lane holds (columns l + 64 i), -1 for the
// value column and beyond.
template <int CPL>
__device__ __forceinline__ void column_heads(const HeadsMeta& hm, int lane, int (&head)[CPL]) {
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int a = lane + 64 * i;
    head[i] = -1;
    for (int k = 0; k < hm.K; ++k)
      if (a >= hm.off[k] && a < hm.off[k + 1]) head[i] = k;
  }
}

// The loss terms of one row and their gradient with respect to its logits,
// computed by one wave.  Lane l holds columns a = l + 64 i: the logit z[i]
// (bias added; the unit head's own logit for its columns), the availability
// byte avb[i] as read, and the column's head.  Lane k < K holds head k's
// action `actl` and mask byte `mkl`.  Writes d[i] = dL/dz for each column
// held (0 where a logit does not count) and adds the row's surrogate,
// squared value error, entropy, clip indicator, approx-KL term, ratio and
// non-finite indicator to st.  An unavailable logit is left out of its
// head's softmax and gets no gradient; a head with no available logit adds
// nothing; an unavailable taken action has log-probability -inf.  All
// reductions over the wave run in a fixed order.
template <int CPL>
__device__ __forceinline__ void ppo_row(const float (&z)[CPL], const uint32_t (&avb)[CPL], const int (&head)[CPL],
                                        int lane, int actl, uint32_t mkl, float Ad, float R, float lpo,
                                        const HeadsMeta& hm, float clip_eps, float vf_coef, float ent_coef,
                                        float invN, float (&d)[CPL], float (&st)[kStatCols]) {
  const int K = hm.K, A = hm.A;
  bool av[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) av[i] = lane + 64 * i >= A || avb[i] != 0;
  float lse[kMaxHeads], zbar[kMaxHeads];
  bool mk[kMaxHeads], some[kMaxHeads];
  int ak[kMaxHeads];
  float logpi = 0.0f, ent = 0.0f;
  // per head: the maximum over its available logits; then one exponential
  // per column; then the sums of e and e z per head
  float mx[kMaxHeads];
#pragma unroll
  for (int k = 0; k < kMaxHeads; ++k) {
    mx[k] = -INFINITY;
    if (k < K) {
      float m = -INFINITY;
#pragma unroll
      for (int i = 0; i < CPL; ++i)
        if (head[i] == k && av[i]) m = fmaxf(m, z[i]);
      mx[k] = wave_max(m);
    }
  }
  float e[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    float m = 0.0f;
#pragma unroll
    for (int k = 0; k < kMaxHeads; ++k)
      if (k < K && head[i] == k) m = mx[k];
    e[i] = (head[i] >= 0 && av[i]) ? expf(z[i] - m) : 0.0f;
  }
  float inv_se[kMaxHeads];
#pragma unroll
  for (int k = 0; k < kMaxHeads; ++k) {
    inv_se[k] = 0.0f;
    some[k] = false;
    mk[k] = false;
    ak[k] = 0;
    if (k < K) {
      float se = 0.0f, sez = 0.0f;
#pragma unroll
      for (int i = 0; i < CPL; ++i)
        if (head[i] == k) {
          se += e[i];
          sez += e[i] * z[i];
        }
      se = wave_sum(se);
      sez = wave_sum(sez);
      some[k] = se > 0.0f;  // the maximum contributes e = 1
      lse[k] = some[k] ? mx[k] + logf(se) : 0.0f;
      zbar[k] = some[k] ? sez / se : 0.0f;
      inv_se[k] = some[k] ? 1.0f / se : 0.0f;
      ak[k] = __builtin_amdgcn_readlane(actl, k);
      mk[k] = __builtin_amdgcn_readlane(static_cast<int>(mkl), k) != 0;
      const int nk = hm.off[k + 1] - hm.off[k];
      const int a_sel = min(max(ak[k], 0), nk - 1);
      const int c_sel = hm.off[k] + a_sel;
      const float z_sel = column(z, c_sel);
      uint32_t tb = avb[0];
#pragma unroll
      for (int i = 1; i < CPL; ++i)
        if (c_sel >> 6 == i) tb = avb[i];
      const bool taken = __builtin_amdgcn_readlane(static_cast<int>(tb), c_sel & 63) != 0;
      if (mk[k] && some[k]) {
        logpi += taken ? z_sel - lse[k] : -INFINITY;
        ent += lse[k] - zbar[k];
      }
    }
  }
  const float dlog = logpi - lpo;
  const float ratio = expf(dlog);
  const float rc = fminf(fmaxf(ratio, 1.0f - clip_eps), 1.0f + clip_eps);
  const float surr = fminf(ratio * Ad, rc * Ad);
  const float V = column(z, A);
  const float verr = V - R;
  const bool flow = (Ad >= 0.0f && ratio <= 1.0f + clip_eps) || (Ad < 0.0f && ratio >= 1.0f - clip_eps);
  const float g_logpi = flow ? -ratio * Ad * invN : 0.0f;
  const float ent_scale = ent_coef * invN;
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int a = lane + 64 * i;
    float di = 0.0f;
    if (a == A) di = 2.0f * vf_coef * verr * invN;
    // this column's head: its softmax normaliser, mean logit, taken action
    bool use = false;
    float is = 0.0f, zb = 0.0f;
    int act_col = -1;
#pragma unroll
    for (int k = 0; k < kMaxHeads; ++k)
      if (k < K && head[i] == k) {
        use = mk[k] && some[k];
        is = inv_se[k];
        zb = zbar[k];
        act_col = hm.off[k] + ak[k];
      }
    if (use && av[i]) {
      const float p = e[i] * is;
      const float onehot = a == act_col ? 1.0f : 0.0f;
      di = g_logpi * (onehot - p) + ent_scale * p * (z[i] - zb);
    }
    d[i] = di;
  }
  const float row_loss = -surr + vf_coef * verr * verr - ent_coef * ent;
  st[0] += surr;
  st[1] += verr * verr;
  st[2] += ent;
  st[3] += fabsf(ratio - 1.0f) > clip_eps ? 1.0f : 0.0f;
  st[4] += expm1f(dlog) - dlog;  // (r - 1) - log r without the cancellation in r - 1
  st[5] += ratio;
  st[6] += isfinite(row_loss) ? 0.0f : 1.0f;
}

// Where the gradient of row n (from ppo_row) goes: the unit head's columns
// to dzext [N][nke] (and 0 in every other output), the rest to dz [N][A1]
// (if set) and to the column sums csum; on the bf16 path the pair hi =
// bf16(d), lo = bf16(d - hi) to dz_hi, dz_lo [N][ld_hilo] (if set).
template <int CPL>
__device__ __forceinline__ void ppo_row_store(float (&d)[CPL], const int (&head)[CPL], int lane, int n,
                                              const HeadsMeta& hm, int kext, int nke, int A1, float* dzext, float* dz,
                                              float (&csum)[CPL], uint16_t* dz_hi, uint16_t* dz_lo, int ncol_hilo,
                                              int ld_hilo) {
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int a = lane + 64 * i;
    if (head[i] >= 0 && head[i] == kext) {
      dzext[static_cast<size_t>(n) * nke + (a - hm.off[kext])] = d[i];
      d[i] = 0.0f;  // these logits do not depend on Wp, bp
    }
    if (dz != nullptr && a < A1) dz[static_cast<size_t>(n) * A1 + a] = d[i];
    csum[i] += d[i];
    if (dz_hi != nullptr && a < ncol_hilo) {
      const uint16_t hb = f32_to_bf16_bits(d[i]);
      const uint16_t lb = f32_to_bf16_bits(d[i] - bf16_bits_to_f32(hb));
      dz_hi[static_cast<size_t>(n) * ld_hilo + a] = hb;
      dz_lo[static_cast<size_t>(n) * ld_hilo + a] = lb;
    }
  }
}

// The block's column sums of dz and its row statistics, reduced over its
// waves in a fixed order through red [waves][CPL 64 + kStatCols] in LDS,
// then written as row `prow` of part: the A1 column sums, then the
// kStatCols statistics.
template <int CPL, int NW>
__device__ __forceinline__ void block_partials(const float (&csum)[CPL], const float (&st)[kStatCols], float* red,
                                               int wave, int lane, int A1, float* part, int prow) {
  constexpr int RW = CPL * 64 + kStatCols;
#pragma unroll
  for (int i = 0; i < CPL; ++i) red[wave * RW + 64 * i + lane] = csum[i];
  if (lane < kStatCols) {
    float v = 0.0f;
#pragma unroll
    for (int q = 0; q < kStatCols; ++q)
      if (q == lane) v = st[q];
    red[wave * RW + CPL * 64 + lane] = v;
  }
  __syncthreads();
  const int W = A1 + kStatCols;
  for (int t = threadIdx.x; t < W; t += blockDim.x) {
    const int c = t < A1 ? t : CPL * 64 + (t - A1);
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) v += red[w * RW + c];
    part[static_cast<size_t>(prow) * W + t] = v;
  }
}

// One wave per row, kRowsPerWave consecutive rows per wave; lane l holds
// logit columns l + 64 i (i < CPL).  zpart: [S][N][A1] partial logits (bias
// not added).  avail [N][A] (or null = all available).  Head kext (or none,
// -1) takes its logits from zext [N][n_kext] (the unit-selection head) and
// returns their gradient in dzext instead of dz and its sums.  Writes dz
// [N][A1] (if set); on the bf16 path the (hi, lo) pair in row layout
// [N][ld_hilo].  Each block writes row blockIdx.x of part (see
// block_partials).
template <int CPL, int SMAX>
__global__ void __launch_bounds__(kWavesPerBlock * 64) ppo_rows(
    int N, int A1, int S, const float* __restrict__ zpart, const float* __restrict__ bp,
    const int32_t* __restrict__ act, const float* __restrict__ logp_old, const float* __restrict__ adv,
    const float* __restrict__ ret, const uint8_t* __restrict__ mask, const uint8_t* __restrict__ avail, HeadsMeta hm,
    const float* __restrict__ zext, float* __restrict__ dzext, int kext, float clip_eps, float vf_coef,
    float ent_coef, float invN, float* __restrict__ dz, float* __restrict__ part, uint16_t* __restrict__ dz_hi,
    uint16_t* __restrict__ dz_lo, int ncol_hilo, int ld_hilo) {
  __shared__ float red[kWavesPerBlock * (CPL * 64 + kStatCols)];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int K = hm.K, A = hm.A;
  int head[CPL];
  column_heads(hm, lane, head);
  float csum[CPL] = {};
  float st[kStatCols] = {};
  const size_t sstride = static_cast<size_t>(N) * A1;
  const int n0 = (blockIdx.x * kWavesPerBlock + wave) * kRowsPerWave;
  // the logits and availability of the wave's rows, every request issued
  // before the first row's reductions (rows past N read row N - 1, unused)
  const int nke = kext >= 0 ? hm.off[kext + 1] - hm.off[kext] : 0;
  float zr[kRowsPerWave][CPL];
  uint32_t avr[kRowsPerWave][CPL];  // availability bytes as read (tested at use)
  // per row: lane k < K holds head k's action and mask byte; the row's
  // advantage, return and behaviour log-probability
  int actr[kRowsPerWave];
  uint32_t mkr[kRowsPerWave];
  float advr[kRowsPerWave], retr[kRowsPerWave], lpor[kRowsPerWave];
  const uint8_t* mkp = mask ? mask : &kAllAvailable;
  const size_t mks = mask ? 1 : 0;
  const int kl = min(lane, K - 1);
  // (branch-free: every load reads a valid address, selects drop the ones
  // not wanted, so no wait sits between two loads)
  const uint8_t* avp = avail ? avail : &kAllAvailable;
  const size_t avs = avail ? 1 : 0;
  const float* zep = zext ? zext : &kNoLogit;
  const size_t zes = zext ? 1 : 0;
#pragma unroll
  for (int rr = 0; rr < kRowsPerWave; ++rr) {
    const size_t nc = static_cast<size_t>(min(n0 + rr, N - 1));
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int a = lane + 64 * i;
      const bool ext = head[i] >= 0 && head[i] == kext;
      const int ac = min(a, A1 - 1);
      float p[SMAX];
#pragma unroll
      for (int s2 = 0; s2 < SMAX; ++s2) p[s2] = zpart[min(s2, S - 1) * sstride + nc * A1 + ac];
      const float ze = zep[(nc * nke + (ext ? a - hm.off[kext] : 0)) * zes];
      float v = bp[ac];
#pragma unroll
      for (int s2 = 0; s2 < SMAX; ++s2)
        if (s2 < S) v += p[s2];
      zr[rr][i] = ext ? ze : a < A1 ? v : 0.0f;
      avr[rr][i] = avp[(nc * A + min(a, A - 1)) * avs];
    }
    actr[rr] = act[nc * K + kl];
    mkr[rr] = mkp[(nc * K + kl) * mks];
    advr[rr] = adv[nc];
    retr[rr] = ret[nc];
    lpor[rr] = logp_old[nc];
  }
  for (int rr = 0; rr < kRowsPerWave; ++rr) {
    const int n = n0 + rr;
    if (n >= N) break;
    float d[CPL];
    ppo_row<CPL>(zr[0], avr[0], head, lane, actr[0], mkr[0], advr[0], retr[0], lpor[0], hm, clip_eps, vf_coef,
                 ent_coef, invN, d, st);
    ppo_row_store<CPL>(d, head, lane, n, hm, kext, nke, A1, dzext, dz, csum, dz_hi, dz_lo, ncol_hilo, ld_hilo);
    // the next row's inputs move to slot 0 (constant indices keep the
    // prefetched values in registers)
#pragma unroll
    for (int q = 0; q + 1 < kRowsPerWave; ++q) {
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        zr[q][i] = zr[q + 1][i];
        avr[q][i] = avr[q + 1][i];
      }
      actr[q] = actr[q + 1];
      mkr[q] = mkr[q + 1];
      advr[q] = advr[q + 1];
      retr[q] = retr[q + 1];
      lpor[q] = lpor[q + 1];
    }
  }
  block_partials<CPL, kWavesPerBlock>(csum, st, red, wave, lane, A1, part, blockIdx.x);
}

// The row kernel with one thread per row, for up to MAXC logit columns: the
// block's 64 rows of logits (the GEMM's partial sums plus bias, or the unit
// head's own logits) and availability bytes are staged in LDS by all 256
// threads with coalesced loads; then, one row per lane, the same definition
// as ppo_row in three passes: each wave takes whole heads (max,
// exponentials and sums, the taken action's log-probability), the first
// wave the row (joint ratio, clipped surrogate, value error, entropy), and
// the waves their heads again for dL/dz per column, written back over the
// row's logits; finally the block writes the gradient rows (dz, the (hi,
// lo) pair, the unit head's columns) and its column sums with coalesced
// stores.  No cross-lane operation; every sum in a fixed order.
// the mask byte read where no mask is given
__device__ const uint8_t kMaskOn = 1;

// Writes row blockIdx.x of part (64 rows per partial).
constexpr int kRtRows = 64;
constexpr int kRtThreads = 256;

template <int MAXC>
__global__ void __launch_bounds__(kRtThreads) ppo_rows_t(
    int N, int A1, int S, const float* __restrict__ zpart, const float* __restrict__ bp,
    const int32_t* __restrict__ act, const float* __restrict__ logp_old, const float* __restrict__ adv,
    const float* __restrict__ ret, const uint8_t* __restrict__ mask, const uint8_t* __restrict__ avail, HeadsMeta hm,
    const float* __restrict__ zext, float* __restrict__ dzext, int kext, float clip_eps, float vf_coef,
    float ent_coef, float invN, float* __restrict__ dz, float* __restrict__ part, uint16_t* __restrict__ dz_hi,
    uint16_t* __restrict__ dz_lo, int ncol_hilo, int ld_hilo) {
  constexpr int ZP = MAXC + 1;  // floats per staged row (odd: a column read hits distinct banks)
  constexpr int AP = MAXC + 4;  // bytes per availability row (an odd number of dwords, for the same reason)
  __shared__ float zs[kRtRows][ZP];
  __shared__ uint8_t avs[kRtRows][AP];
  __shared__ float st_red[kStatCols][kRtRows];
  __shared__ float hd_mx[kMaxHeads][kRtRows], hd_inv[kMaxHeads][kRtRows], hd_zbar[kMaxHeads][kRtRows];
  __shared__ float hd_lp[kMaxHeads][kRtRows], hd_ent[kMaxHeads][kRtRows], row_g[kRtRows];
  __shared__ int hd_act[kMaxHeads][kRtRows], hd_use[kMaxHeads][kRtRows];
  // the byte the head loops read in place of an availability byte when no
  // availability is given (avs is then never written)
  __shared__ uint8_t av_all;
  const int t = threadIdx.x;
  const int n0 = blockIdx.x * kRtRows;
  const int rows = min(kRtRows, N - n0);
  const int K = hm.K, A = hm.A;
  const size_t sstride = static_cast<size_t>(N) * A1;
  const int nke = kext >= 0 ? hm.off[kext + 1] - hm.off[kext] : 0;
  const int e0 = kext >= 0 ? hm.off[kext] : 0;
  const int r = t & (kRtRows - 1), w0 = t / kRtRows;
  // the per-row inputs are loaded first, so their latency overlaps the
  // staging below: the taken action and mask of each head this lane takes
  // (heads w0, w0 + 4, ...) and, for the row threads, logp_old, A and R
  constexpr int kHpl = kMaxHeads / (kRtThreads / kRtRows);  // heads per lane
  // (every load here and in the staging is unconditional, its index clamped
  // into range, so none waits behind a branch; values of clamped indices
  // are never used)
  int act_r[kHpl];
  uint32_t mk_r[kHpl];
  {
    const int rc = min(r, rows - 1);
    const uint8_t* mp = mask != nullptr ? mask : &kMaskOn;
    const size_t ms = mask != nullptr ? 1 : 0;
#pragma unroll
    for (int i = 0; i < kHpl; ++i) {
      const size_t nk = static_cast<size_t>(n0 + rc) * K + min(w0 + i * (kRtThreads / kRtRows), K - 1);
      act_r[i] = act[nk];
      mk_r[i] = mp[nk * ms];
    }
  }
  const int tc = n0 + min(t, rows - 1);
  const float lpo_r = logp_old[tc], adv_r = adv[tc], ret_r = ret[tc];
  // stage the rows: element e = (r, a) of the block's [rows x A1] slice
  // (the block's rows are contiguous in every source), kGrp elements per
  // thread at a time: the bias and split 0 of all of them, then each further
  // split, each split's loads all issued before its adds (the sum is bias +
  // split 0 + split 1 + ... in that order)
  {
    constexpr int kGrp = 16;
    const int ne = rows * A1;
    const float* zp = zpart + static_cast<size_t>(n0) * A1;
    // (r, a) of e advances by (dr, dc) per kRtThreads elements
    const int dr = kRtThreads / A1, dc = kRtThreads - dr * A1;
    for (int e0g = 0; e0g < ne; e0g += kGrp * kRtThreads) {
      const int r0 = (e0g + t) / A1, c0 = e0g + t - r0 * A1;
      int ix[kGrp];
#pragma unroll
      for (int q = 0; q < kGrp; ++q) ix[q] = min(e0g + t + q * kRtThreads, ne - 1);
      float v[kGrp], b[kGrp], w[kGrp];
      {
        int c = c0;
#pragma unroll
        for (int q = 0; q < kGrp; ++q) {
          b[q] = bp[c];
          c += dc;
          if (c >= A1) c -= A1;
        }
      }
#pragma unroll
      for (int q = 0; q < kGrp; ++q) v[q] = zp[ix[q]];
      if (S > 1) {
#pragma unroll
        for (int q = 0; q < kGrp; ++q) w[q] = zp[sstride + ix[q]];
      }
      // (keeps the adds below every load above)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < kGrp; ++q) v[q] = b[q] + v[q];
      if (S > 1) {
#pragma unroll
        for (int q = 0; q < kGrp; ++q) v[q] += w[q];
      }
      for (int s2 = 2; s2 < S; ++s2) {
#pragma unroll
        for (int q = 0; q < kGrp; ++q) w[q] = zp[s2 * sstride + ix[q]];
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < kGrp; ++q) v[q] += w[q];
      }
      // (the unit head's columns come from zext below, written by other
      // threads: no store here may race with those)
      int rq = r0, c = c0;
#pragma unroll
      for (int q = 0; q < kGrp; ++q) {
        const int e = e0g + t + q * kRtThreads;
        if (e < ne && (c < e0 || c >= e0 + nke)) zs[rq][c] = v[q];
        rq += dr;
        c += dc;
        if (c >= A1) {
          c -= A1;
          ++rq;
        }
      }
    }
    for (int e = t; e < rows * nke; e += kRtThreads) {
      const int r = e / nke, u = e - r * nke;
      zs[r][e0 + u] = zext[static_cast<size_t>(n0) * nke + e];
    }
    if (avail != nullptr) {
#pragma unroll 4
      for (int e = t; e < rows * A; e += kRtThreads) {
        const int r = e / A, a = e - r * A;
        avs[r][a] = avail[static_cast<size_t>(n0) * A + e];
      }
    } else if (t == 0) {
      av_all = 1;
    }
  }
  __syncthreads();
  // heads: wave w takes heads w, w + 4, ... of every row (lane = row): the
  // head's maximum, normaliser, mean logit and the taken action's
  // log-probability, kept in LDS per (head, row).  A lane reads a head's
  // columns kCh at a time, every read of a chunk issued before its first
  // use (indices past the head repeat its last column and are not used), so
  // a chunk waits on LDS once; the sums keep column order.
  constexpr int kCh = 8;
  const bool all_av = avail == nullptr;  // uniform: no availability bytes read
  auto chunk = [&](const float* z, const uint8_t* av, int o, int nk, int a0, float (&v)[kCh], bool (&ok)[kCh]) {
#pragma unroll
    for (int q = 0; q < kCh; ++q) {
      const int a = o + min(a0 + q, nk - 1);
      v[q] = z[a];
      // (a byte is read either way, without a branch: the column's, or
      // av_all = 1 when no availability is given)
      ok[q] = (a0 + q < nk) & (*(all_av ? &av_all : av + a) != 0);
    }
  };
  if (r < rows) {
    const float* z = zs[r];
    const uint8_t* av = avs[r];
#pragma unroll
    for (int i = 0; i < kHpl; ++i) {
      const int k = w0 + i * (kRtThreads / kRtRows);
      if (k >= K) continue;
      const int o = hm.off[k], nk = hm.off[k + 1] - o;
      float m = -INFINITY;
      for (int a0 = 0; a0 < nk; a0 += kCh) {
        float v[kCh];
        bool ok[kCh];
        chunk(z, av, o, nk, a0, v, ok);
#pragma unroll
        for (int q = 0; q < kCh; ++q)
          if (ok[q]) m = fmaxf(m, v[q]);
      }
      float sum = 0.0f, sz = 0.0f;
      for (int a0 = 0; a0 < nk; a0 += kCh) {
        float v[kCh];
        bool ok[kCh];
        chunk(z, av, o, nk, a0, v, ok);
#pragma unroll
        for (int q = 0; q < kCh; ++q)
          if (ok[q]) {
            const float e = expf(v[q] - m);
            sum += e;
            sz += e * v[q];
          }
      }
      const bool some = sum > 0.0f;  // the maximum contributes e = 1
      const float lse = some ? m + logf(sum) : 0.0f;
      const float zb = some ? sz / sum : 0.0f;
      const int ak = act_r[i];
      const bool use = mk_r[i] != 0 && some;
      float lp = 0.0f, en = 0.0f;
      if (use) {
        const int a_sel = min(max(ak, 0), nk - 1);
        lp = (all_av || av[o + a_sel]) ? z[o + a_sel] - lse : -INFINITY;
        en = lse - zb;
      }
      hd_mx[k][r] = m;
      hd_inv[k][r] = some ? 1.0f / sum : 0.0f;
      hd_zbar[k][r] = zb;
      hd_lp[k][r] = lp;
      hd_ent[k][r] = en;
      hd_act[k][r] = ak;
      hd_use[k][r] = use;
    }
  }
  __syncthreads();
  // the row: joint ratio (log-probabilities summed over heads in order),
  // clipped surrogate, value error, entropy, the scale of the log-probability
  // gradient; the value column's gradient and the padding columns
  if (t < kRtRows) {
    float st[kStatCols] = {};
    if (t < rows) {
      float* z = zs[t];
      float logpi = 0.0f, ent = 0.0f;
      for (int k = 0; k < K; ++k)
        if (hd_use[k][t]) {
          logpi += hd_lp[k][t];
          ent += hd_ent[k][t];
        }
      const float Ad = adv_r, R = ret_r;
      const float dlog = logpi - lpo_r;
      const float ratio = expf(dlog);
      const float rc = fminf(fmaxf(ratio, 1.0f - clip_eps), 1.0f + clip_eps);
      const float surr = fminf(ratio * Ad, rc * Ad);
      const float verr = z[A] - R;
      const bool flow = (Ad >= 0.0f && ratio <= 1.0f + clip_eps) || (Ad < 0.0f && ratio >= 1.0f - clip_eps);
      row_g[t] = flow ? -ratio * Ad * invN : 0.0f;
      z[A] = 2.0f * vf_coef * verr * invN;
      for (int a = A1; a < MAXC; ++a) z[a] = 0.0f;
      const float row_loss = -surr + vf_coef * verr * verr - ent_coef * ent;
      st[0] = surr;
      st[1] = verr * verr;
      st[2] = ent;
      st[3] = fabsf(ratio - 1.0f) > clip_eps ? 1.0f : 0.0f;
      st[4] = expm1f(dlog) - dlog;  // (r - 1) - log r without the cancellation in r - 1
      st[5] = ratio;
      st[6] = isfinite(row_loss) ? 0.0f : 1.0f;
    } else {
      for (int a = 0; a < MAXC; ++a) zs[t][a] = 0.0f;  // rows past N: defined, never stored
    }
#pragma unroll
    for (int q = 0; q < kStatCols; ++q) st_red[q][t] = st[q];
  }
  __syncthreads();
  // dL/dz of every head column, written back over the row's logits (same
  // head-to-wave assignment as above)
  if (r < rows) {
    float* z = zs[r];
    const uint8_t* av = avs[r];
    const float g_logpi = row_g[r];
    const float ent_scale = ent_coef * invN;
    for (int k = w0; k < K; k += kRtThreads / kRtRows) {
      const int o = hm.off[k], nk = hm.off[k + 1] - o;
      const int ak = hd_act[k][r];
      const bool use = hd_use[k][r] != 0;
      const float mx = hd_mx[k][r], inv = hd_inv[k][r], zbar = hd_zbar[k][r];
      // (the chunk's reads stay inside this head's columns, which only this
      // lane writes)
      for (int a0 = 0; a0 < nk; a0 += kCh) {
        float v[kCh];
        bool ok[kCh];
        chunk(z, av, o, nk, a0, v, ok);
#pragma unroll
        for (int q = 0; q < kCh; ++q) {
          const int a = a0 + q;
          float d = 0.0f;
          if (use && ok[q]) {
            const float p = expf(v[q] - mx) * inv;
            const float onehot = a == ak ? 1.0f : 0.0f;
            d = g_logpi * (onehot - p) + ent_scale * p * (v[q] - zbar);
          }
          if (a < nk) z[o + a] = d;
        }
      }
    }
  }
  __syncthreads();
  // the unit head's gradient leaves; its columns are 0 in every other output
  if (nke > 0) {
    for (int e = t; e < rows * nke; e += kRtThreads) {
      const int r = e / nke, u = e - r * nke;
      dzext[static_cast<size_t>(n0) * nke + e] = zs[r][e0 + u];
    }
    __syncthreads();
    for (int e = t; e < kRtRows * nke; e += kRtThreads) zs[e / nke][e0 + e % nke] = 0.0f;
    __syncthreads();
  }
  if (dz != nullptr)
    for (int e = t; e < rows * A1; e += kRtThreads) dz[static_cast<size_t>(n0) * A1 + e] = zs[e / A1][e % A1];
  if (dz_hi != nullptr) {
    // 8 columns of one row per item: two 16-byte stores (hi, lo)
    const int cpr = ncol_hilo / 8;  // ncol_hilo is a multiple of 64
    for (int c = t; c < rows * cpr; c += kRtThreads) {
      const int r = c / cpr, a0 = (c - r * cpr) * 8;
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float d0 = zs[r][a0 + 2 * j], d1 = zs[r][a0 + 2 * j + 1];
        const uint16_t h0 = f32_to_bf16_bits(d0), h1 = f32_to_bf16_bits(d1);
        const uint16_t l0 = f32_to_bf16_bits(d0 - bf16_bits_to_f32(h0));
        const uint16_t l1 = f32_to_bf16_bits(d1 - bf16_bits_to_f32(h1));
        hw[j] = h0 | (static_cast<uint32_t>(h1) << 16);
        lw[j] = l0 | (static_cast<uint32_t>(l1) << 16);
      }
      const size_t o = static_cast<size_t>(n0 + r) * ld_hilo + a0;
      *reinterpret_cast<uint4*>(dz_hi + o) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
      *reinterpret_cast<uint4*>(dz_lo + o) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
    }
  }
  // column sums over the block's rows, then its statistics, in row order
  const int W = A1 + kStatCols;
  for (int c = t; c < W; c += kRtThreads) {
    float v = 0.0f;
    if (c < A1) {
#pragma unroll 8
      for (int r = 0; r < rows; ++r) v += zs[r][c];
    } else {
#pragma unroll 8
      for (int r = 0; r < rows; ++r) v += st_red[c - A1][r];
    }
    part[static_cast<size_t>(blockIdx.x) * W + c] = v;
  }
}

// The weights of the dh product, transposed and repeated for the (hi, lo)
// pair: row j of wT [H][2 ldh] is [w(0..ldh) | w(0..ldh)] with w(k) = Wp[k][j]
// for k < A1, Wq[k - A1p][j] for A1p <= k < A1p + d (the unit head's query
// weights, if any) and 0 elsewhere.  One 64 x 64 tile per block through LDS.
__global__ void __launch_bounds__(256) pair_weights_t(int A1, int A1p, int ldh, int H, const uint16_t* __restrict__ Wp,
                                                      const uint16_t* __restrict__ Wq, int d,
                                                      uint16_t* __restrict__ wT) {
  __shared__ uint16_t t[64][66];
  const int j0 = blockIdx.x * 64, k0 = blockIdx.y * 64;
  // every load unconditional (rows outside both sources read row 0 of Wp
  // and are replaced by 0), so all 16 of a thread's loads are in flight
  // together
  constexpr int kPer = 64 * 64 / 256;
  const bool hasq = Wq != nullptr;
  uint16_t v[kPer];
  bool in[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int e = threadIdx.x + 256 * i, kk = e >> 6, jj = e & 63, k = k0 + kk;
    const bool inp = k < A1;
    const bool inq = hasq & (k >= A1p) & (k < A1p + d);
    in[i] = inp | inq;
    const uint16_t* base = inq ? Wq : Wp;
    const int row = inp ? k : inq ? k - A1p : 0;
    v[i] = base[static_cast<size_t>(row) * H + j0 + jj];
  }
  // (keeps the LDS stores below every load above)
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int e = threadIdx.x + 256 * i;
    t[e >> 6][e & 63] = in[i] ? v[i] : static_cast<uint16_t>(0);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 64 * 64; e += 256) {
    const int jj = e >> 6, kk = e & 63;
    const size_t row = static_cast<size_t>(j0 + jj) * 2 * ldh;
    wT[row + k0 + kk] = t[kk][jj];
    wT[row + ldh + k0 + kk] = t[kk][jj];
  }
}

// stats from the summed block partials (sums = [dz column sums (A1) | row
// stat sums (kStatCols)]); also copies the bias gradient out.
__global__ void ppo_finalize(int A1, const float* __restrict__ sums, float invN, float vf_coef, float ent_coef,
                             float* __restrict__ stats, float* __restrict__ dbp) {
  for (int a = threadIdx.x; a < A1; a += blockDim.x) dbp[a] = sums[a];
  if (threadIdx.x != 0) return;
  const float* ss = sums + A1;
  const float pg = -ss[0] * invN, vf = ss[1] * invN, ent = ss[2] * invN;
  stats[0] = pg + vf_coef * vf - ent_coef * ent;
  stats[1] = pg;
  stats[2] = vf;
  stats[3] = ent;
  stats[4] = ss[3] * invN;
  stats[5] = ss[4] * invN;
  stats[6] = ss[5] * invN;
  stats[7] = ss[6];
}

struct PpoWs {
  size_t zpart, dz, part, sums, wpart, dzp, wT, unit, total;
  UnitWs uw;  // the unit-selection head's scratch, at offset unit (if any)
  GemmPlan plan_z, plan_w, plan_h;
  int nblk, A1, A1p, ldh, wsplits;  // ldh: row length of the (hi, lo) pair, A1p + the unit head's dp
  bool rows_t;  // the row kernel with one thread per row (ppo_rows_t)
  int nblk_t;   // its blocks (= partial rows)
};

static PpoWs ppo_ws(o5_dtype dt, int N, int H, int A1, int unit_nk = 0, int unit_d = 0) {
  PpoWs w{};
  const bool bf = dt == O5_BF16;
  w.A1 = A1;
  w.A1p = cdiv(A1, 64) * 64;  // padded logit count: a multiple of the K tile
  w.ldh = w.A1p + (unit_d > 0 ? cdiv(unit_d, 64) * 64 : 0);
  w.nblk = cdiv(N, kRowsPerBlock);
  // the thread-per-row kernel takes up to 256 logit columns; where a unit
  // head widens the pair past 256 columns its long head (one lane runs a
  // head's columns serially) made it slower than the wave-per-row kernel
  // (1.61 against 1.50 ms for the call with 189 units)
  w.rows_t = w.ldh <= 256;
  w.nblk_t = cdiv(N, kRtRows);
  w.plan_z = plan_gemm(bf, N, A1, H);
  w.plan_w = plan_gemm(false, A1, H, N);  // fp32 dWp (bf16: the pair product below)
  w.plan_h = plan_gemm(bf, N, H, 2 * w.ldh);
  w.plan_h.splits = 1;
  w.wsplits = 1;
  if (bf) {
    // dWp: M = 2 A1p, N = H, K = N: split K so the grid has about 256
    // blocks, each with at least 8 K tiles of 32
    const int tiles = cdiv(2 * w.A1p, 256) * cdiv(H, 256);
    w.wsplits = std::max(1, std::min(cdiv(256, tiles), cdiv(N, 32) / 8));
  }
  size_t o = 0;
  w.zpart = o;
  o += align_up(static_cast<size_t>(w.plan_z.splits) * N * A1 * 4);
  w.dz = o;
  o += align_up(static_cast<size_t>(N) * A1 * 4);
  w.part = o;
  o += align_up(static_cast<size_t>(w.nblk) * (A1 + kStatCols) * 4);
  w.sums = o;
  o += align_up(static_cast<size_t>(A1 + kStatCols) * 4);
  w.wpart = o;
  o += align_up(bf ? static_cast<size_t>(w.wsplits) * 2 * w.A1p * H * 4
                        : static_cast<size_t>(w.plan_w.splits) * A1 * H * 4);
  w.dzp = w.wT = 0;
  if (bf) {
    // the (hi, lo) pair, row n = [hi (ldh) | lo (ldh)], and the weights
    // transposed and repeated for it, row j = [W[., j] | W[., j]]
    w.dzp = o;
    o += align_up(static_cast<size_t>(N) * 2 * w.ldh * 2);
    w.wT = o;
    o += align_up(static_cast<size_t>(H) * 2 * w.ldh * 2);
  }
  w.unit = o;
  if (unit_d > 0) {
    w.uw = unit_ws(dt, N, H, unit_nk, unit_d, true);
    o += align_up(w.uw.total);
  }
  w.total = o;
  return w;
}

int check_heads(const char* fn, o5_dtype dt, int N, int H, int K, const int* head_sizes, HeadsMeta* hm) {
  O5_CHECK(dt == O5_F32 || dt == O5_BF16, O5_E_DTYPE, "%s: unknown dtype %d", fn, static_cast<int>(dt));
  O5_CHECK(N >= 1 && H >= 64 && H % 64 == 0 && H <= 65536, O5_E_SHAPE,
           "%s: need N >= 1 and H a positive multiple of 64 (N=%d H=%d)", fn, N, H);
  O5_CHECK(K >= 1 && K <= kMaxHeads, O5_E_SHAPE, "%s: K=%d heads must be in 1..%d", fn, K, kMaxHeads);
  O5_CHECK(head_sizes != nullptr, O5_E_NULL, "%s: head_sizes is NULL", fn);
  hm->K = K;
  hm->off[0] = 0;
  for (int k = 0; k < K; ++k) {
    O5_CHECK(head_sizes[k] >= 1, O5_E_SHAPE, "%s: head_sizes[%d]=%d must be >= 1", fn, k, head_sizes[k]);
    hm->off[k + 1] = hm->off[k] + head_sizes[k];
    O5_CHECK(hm->off[k + 1] + 1 <= kMaxA1, O5_E_SHAPE, "%s: total logits + 1 must be <= %d", fn, kMaxA1);
  }
  for (int k = K + 1; k <= kMaxHeads; ++k) hm->off[k] = hm->off[K];
  hm->A = hm->off[K];
  O5_CHECK(static_cast<long long>(N) * H < (1ll << 31), O5_E_SHAPE, "%s: N*H must stay below 2^31", fn);
  return O5_OK;
}

template <int CPL, int SMAX>
static void launch_rows_s(const PpoWs& w, int N, int A1, int S, const float* zpart, const float* bp,
                          const int32_t* act, const float* logp_old, const float* adv, const float* ret, const uint8_t* mask,
                        const uint8_t* avail, const HeadsMeta& hm, const float* zext, float* dzext, int kext,
                        o5_ppo_hp hp, float invN, float* dz, float* part, uint16_t* dzhi, uint16_t* dzlo,
                        hipStream_t s) {
  hipLaunchKernelGGL((ppo_rows<CPL, SMAX>), dim3(w.nblk), dim3(kWavesPerBlock * 64), 0, s, N, A1, S, zpart, bp, act,
                     logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp.clip_eps, hp.vf_coef, hp.ent_coef, invN,
                     dz, part, dzhi, dzlo, w.A1p, 2 * w.ldh);
}

// The row kernel unrolls its reads of the logits GEMM's split partials up
// to SMAX (2 covers the usual split, 16 every plan).
template <int CPL>
static void launch_rows(const PpoWs& w, int N, int A1, int S, const float* zpart, const float* bp, const int32_t* act,
                        const float* logp_old, const float* adv, const float* ret, const uint8_t* mask,
                        const uint8_t* avail, const HeadsMeta& hm, const float* zext, float* dzext, int kext,
                        o5_ppo_hp hp, float invN, float* dz, float* part, uint16_t* dzhi, uint16_t* dzlo,
                        hipStream_t s) {
  if (S <= 2)
    launch_rows_s<CPL, 2>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp,
                          invN, dz, part, dzhi, dzlo, s);
  else
    launch_rows_s<CPL, 16>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp,
                           invN, dz, part, dzhi, dzlo, s);
}

template <typename E>
static int ppo_impl(int N, int H, const HeadsMeta& hm, const E* h, const E* Wp, const float* bp, const int32_t* act,
                    const float* logp_old, const float* adv, const float* ret, const uint8_t* mask,
                    const uint8_t* avail, const o5_unit_head* unit, o5_ppo_hp hp,
                    float* stats, float* dh, float* dWp, float* dbp, char* ws, const PpoWs& w, hipStream_t s,
                    uint16_t* P_out = nullptr, uint16_t* W_out = nullptr) {
  // bf16 path: the (hi, lo) pair and its repeated weights go to P_out and
  // W_out when given (then dh may be null and is not formed)
  const int A1 = hm.A + 1;
  float* zpart = reinterpret_cast<float*>(ws + w.zpart);
  float* dz = reinterpret_cast<float*>(ws + w.dz);
  float* part = reinterpret_cast<float*>(ws + w.part);
  float* sums = reinterpret_cast<float*>(ws + w.sums);
  float* wpart = reinterpret_cast<float*>(ws + w.wpart);
  const float invN = 1.0f / static_cast<float>(N);
  uint16_t* dzhi = nullptr;
  uint16_t* dzlo = nullptr;
  if constexpr (sizeof(E) == 2) {
    dzhi = P_out != nullptr ? P_out : reinterpret_cast<uint16_t*>(ws + w.dzp);
    dzlo = dzhi + w.ldh;
    dz = nullptr;  // the bf16 products read the (hi, lo) pair only
  }
  const float* zext = nullptr;
  float* dzext = nullptr;
  int kext = -1;
  char* uws = ws + w.unit;
  constexpr o5_dtype dt = sizeof(E) == 2 ? O5_BF16 : O5_F32;
  if (unit != nullptr) {  // the unit-selection head's logits
    kext = unit->head;
    unit_forward(dt, N, H, w.uw.nk, *unit, h, uws, w.uw, s);
    zext = reinterpret_cast<const float*>(uws + w.uw.zext);
    dzext = reinterpret_cast<float*>(uws + w.uw.dzext);
  }
  {  // z = h Wp^T
    KRows2<E> hl{h, nullptr, nullptr, H, 0, H, H, N};
    KRows2<E> wl{Wp, nullptr, nullptr, H, 0, H, H, A1};
    EpiLogits epi{{zpart, A1, static_cast<size_t>(N) * A1}};
    run_gemm(w.plan_z, hl, wl, epi, N, A1, H, s);
  }
  const int S = w.plan_z.splits;
  const int cpl = cdiv(A1, 64);
  if (w.rows_t && w.A1p <= 128)
    hipLaunchKernelGGL(ppo_rows_t<128>, dim3(w.nblk_t), dim3(kRtThreads), 0, s, N, A1, S, zpart, bp, act, logp_old,
                       adv, ret, mask, avail, hm, zext, dzext, kext, hp.clip_eps, hp.vf_coef, hp.ent_coef, invN, dz,
                       part, dzhi, dzlo, w.A1p, 2 * w.ldh);
  else if (w.rows_t)
    hipLaunchKernelGGL(ppo_rows_t<256>, dim3(w.nblk_t), dim3(kRtThreads), 0, s, N, A1, S, zpart, bp, act, logp_old,
                       adv, ret, mask, avail, hm, zext, dzext, kext, hp.clip_eps, hp.vf_coef, hp.ent_coef, invN, dz,
                       part, dzhi, dzlo, w.A1p, 2 * w.ldh);
  else if (cpl <= 1)
    launch_rows<1>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz,
                   part, dzhi, dzlo, s);
  else if (cpl <= 2)
    launch_rows<2>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz,
                   part, dzhi, dzlo, s);
  else if (cpl <= 4)
    launch_rows<4>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz,
                   part, dzhi, dzlo, s);
  else if (cpl <= 8)
    launch_rows<8>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz,
                   part, dzhi, dzlo, s);
  else
    launch_rows<16>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz,
                    part, dzhi, dzlo, s);
  if constexpr (sizeof(E) == 2) {
    const int A1p = w.A1p, ldh = w.ldh;
    uint16_t* wT = W_out != nullptr ? W_out : reinterpret_cast<uint16_t*>(ws + w.wT);
    const uint16_t* Wq = nullptr;
    int d = 0;
    if (unit != nullptr) {
      // dq (hi, lo) into columns A1p .. ldh - 1 of the pair, Wq into the same columns of wT
      unit_grad(dt, N, H, w.uw.nk, *unit, h, uws, w.uw, dzhi, dzlo, A1p, 2 * ldh, s);
      Wq = static_cast<const uint16_t*>(unit->Wq);
      d = unit->d;
    }
    hipLaunchKernelGGL(pair_weights_t, dim3(H / 64, ldh / 64), dim3(256), 0, s, A1, A1p, ldh, H, Wp, Wq, d, wT);
    if (dh != nullptr) {  // dh = [dz_hi dq_hi | dz_lo dq_lo] . [Wp Wq ; Wp Wq]  (K = 2 ldh), both K-contiguous
      KRows2<uint16_t> al{dzhi, nullptr, nullptr, 2 * ldh, 0, 2 * ldh, 2 * ldh, N};
      KRows2<uint16_t> bl{wT, nullptr, nullptr, 2 * ldh, 0, 2 * ldh, 2 * ldh, H};
      EpiStoreF32 epi{dh, H, 0};
      run_gemm(w.plan_h, al, bl, epi, N, H, 2 * ldh, s);
    }
    {
      // [dWp_hi ; dWp_lo] = [dz_hi | dz_lo]^T . h  (M = 2 A1p rows: the hi
      // logit columns of the pair, then its lo logit columns (a unit head's
      // dq columns in between are skipped); N = H, K = N), both operands read
      // I-contiguous (the row layouts of the pair and of h, h read once),
      // split over K; then hi + lo per split
      ICols2<uint16_t> al{dzhi, dzlo, dzlo, nullptr, 2 * ldh, 2 * ldh, A1p, 2 * A1p, N, N};
      ICols2<uint16_t> bl{h, nullptr, nullptr, nullptr, H, 0, H, H, N, 0};
      EpiStoreF32 epi{wpart, H, static_cast<size_t>(2) * A1p * H};
      launch_gemm_bf16_dma(al, bl, epi, 2 * A1p, H, N, w.wsplits, s);
      hipLaunchKernelGGL(sum_hilo_splits, dim3(cdiv(static_cast<long long>(A1) * H, 256)), dim3(256), 0, s,
                         w.wsplits, A1, A1p, H, wpart, dWp);
    }
  } else {
    if (unit == nullptr) {  // dh = dz Wp  (fp32 FMA engine)
      KRows2<float> al{dz, nullptr, nullptr, A1, 0, A1, A1, N};
      ICols2<E> bl{Wp, nullptr, nullptr, nullptr, H, 0, H, H, A1, 0};
      EpiStoreF32 epi{dh, H, 0};
      launch_gemm_f32(al, bl, epi, N, H, A1, 1, s);
    } else {  // dh = [dz | dq] . [Wp ; Wq]
      unit_grad(dt, N, H, w.uw.nk, *unit, h, uws, w.uw, nullptr, nullptr, 0, 0, s);
      const int d = unit->d;
      const float* dq = reinterpret_cast<const float*>(uws + w.uw.dq);
      KRows2<float> al{dz, dq, nullptr, A1, d, A1, A1 + d, N};
      ICols2<E> bl{Wp, Wp, static_cast<const E*>(unit->Wq), nullptr, H, H, 0, H, A1 + d, A1};
      EpiStoreF32 epi{dh, H, 0};
      launch_gemm_f32(al, bl, epi, N, H, A1 + d, 1, s);
    }
    {  // dWp = dz^T h, split over rows
      ICols2<float> al{dz, nullptr, nullptr, nullptr, A1, 0, A1, A1, N, 0};
      ICols2<E> bl{h, nullptr, nullptr, nullptr, H, 0, H, H, N, 0};
      EpiStoreF32 epi{wpart, H, static_cast<size_t>(A1) * H};
      launch_gemm_f32(al, bl, epi, A1, H, N, w.plan_w.splits, s);
    }
    hipLaunchKernelGGL(colsum_rows, dim3(cdiv(static_cast<long long>(A1) * H, 256)), dim3(256), 0, s, w.plan_w.splits,
                       A1 * H, wpart, dWp);
  }
  hipLaunchKernelGGL(colsum_tree, dim3(A1 + kStatCols), dim3(256), 0, s, w.rows_t ? w.nblk_t : w.nblk,
                     A1 + kStatCols, part, sums);
  hipLaunchKernelGGL(ppo_finalize, dim3(1), dim3(256), 0, s, A1, sums, invN, hp.vf_coef, hp.ent_coef, stats, dbp);
  return check_launch("o5_ppo_loss_grad");
}

}  // namespace o5

using namespace o5;

extern "C" size_t o5_ppo_loss_grad_workspace_bytes(o5_dtype dt, int N, int H, int K, const int* head_sizes,
                                                   const o5_unit_head* unit) {
  HeadsMeta hm;
  if (check_heads("o5_ppo_loss_grad_workspace_bytes", dt, N, H, K, head_sizes, &hm) != O5_OK) return 0;
  if (unit != nullptr && (unit->head < 0 || unit->head >= K || unit->d < 8 || unit->d > 512 || (unit->d & (unit->d - 1)) != 0)) return 0;
  return unit ? ppo_ws(dt, N, H, hm.A + 1, hm.off[unit->head + 1] - hm.off[unit->head], unit->d).total
              : ppo_ws(dt, N, H, hm.A + 1).total;
}

// Validation shared by the two loss calls (everything but the gradient
// outputs that differ); fills hm and w.
static int ppo_check(const char* fn, o5_dtype dt, int N, int H, int K, const int* head_sizes, const void* h,
                     const void* Wp, const float* bp, const int32_t* act, const float* logp_old, const float* adv,
                     const float* ret, const uint8_t* head_mask, const uint8_t* avail, const o5_unit_head* unit,
                     o5_ppo_hp hp, float* stats, float* dWp, float* dbp, void* ws, size_t ws_bytes, HeadsMeta* hm,
                     PpoWs* w) {
  int st = check_heads(fn, dt, N, H, K, head_sizes, hm);
  if (st != O5_OK) return st;
  O5_CHECK(hp.clip_eps >= 0.0f && hp.clip_eps < 1.0f, O5_E_ARG, "%s: clip_eps=%g must be in [0, 1)", fn,
           hp.clip_eps);
  O5_PTR_IN(fn, h, "h");
  O5_PTR_IN(fn, Wp, "Wp");
  O5_PTR_IN(fn, bp, "bp");
  O5_PTR_IN(fn, act, "act");
  O5_PTR_IN(fn, logp_old, "logp_old");
  O5_PTR_IN(fn, adv, "adv");
  O5_PTR_IN(fn, ret, "ret");
  O5_OPT_PTR_IN(fn, head_mask, "head_mask");
  O5_OPT_PTR_IN(fn, avail, "avail");
  if (unit != nullptr) {
    st = check_unit(fn, *hm, unit, true);
    if (st != O5_OK) return st;
  }
  O5_PTR_IN(fn, stats, "stats");
  O5_PTR_IN(fn, dWp, "dWp");
  O5_PTR_IN(fn, dbp, "dbp");
  *w = unit ? ppo_ws(dt, N, H, hm->A + 1, hm->off[unit->head + 1] - hm->off[unit->head], unit->d)
            : ppo_ws(dt, N, H, hm->A + 1);
  O5_CHECK(ws != nullptr && ws_bytes >= w->total, O5_E_WORKSPACE, "%s: workspace needs %zu bytes, got %zu", fn,
           w->total, ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "%s: ws is not 16-byte aligned", fn);
  return O5_OK;
}

extern "C" int o5_ppo_loss_grad(o5_dtype dt, int N, int H, int K, const int* head_sizes, const void* h, const void* Wp,
                                const float* bp, const int32_t* act, const float* logp_old, const float* adv,
                                const float* ret, const uint8_t* head_mask, const uint8_t* avail,
                                const o5_unit_head* unit, o5_ppo_hp hp, float* stats, float* dh,
                                float* dWp, float* dbp, void* ws, size_t ws_bytes, void* stream) {
  HeadsMeta hm;
  PpoWs w;
  int st = ppo_check("o5_ppo_loss_grad", dt, N, H, K, head_sizes, h, Wp, bp, act, logp_old, adv, ret, head_mask,
                     avail, unit, hp, stats, dWp, dbp, ws, ws_bytes, &hm, &w);
  if (st != O5_OK) return st;
  O5_PTR(dh, "dh");
  char* wsp = static_cast<char*>(ws);
  hipStream_t s = as_stream(stream);
  ktimer_begin(kSitePpo, s);
  if (dt == O5_BF16)
    st = ppo_impl<uint16_t>(N, H, hm, static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(Wp), bp, act,
                            logp_old, adv, ret, head_mask, avail, unit, hp, stats, dh, dWp, dbp, wsp, w, s);
  else
    st = ppo_impl<float>(N, H, hm, static_cast<const float*>(h), static_cast<const float*>(Wp), bp, act, logp_old, adv,
                         ret, head_mask, avail, unit, hp, stats, dh, dWp, dbp, wsp, w, s);
  ktimer_end(kSitePpo, s);
  return st;
}

extern "C" int o5_ppo_head_grad_ld(int H, int K, const int* head_sizes, const o5_unit_head* unit) {
  HeadsMeta hm;
  if (check_heads("o5_ppo_head_grad_ld", O5_BF16, 1, H, K, head_sizes, &hm) != O5_OK) return 0;
  if (unit != nullptr &&
      (unit->head < 0 || unit->head >= K || unit->d < 8 || unit->d > 512 || (unit->d & (unit->d - 1)) != 0))
    return 0;
  const PpoWs w = unit ? ppo_ws(O5_BF16, 1, H, hm.A + 1, hm.off[unit->head + 1] - hm.off[unit->head], unit->d)
                       : ppo_ws(O5_BF16, 1, H, hm.A + 1);
  return 2 * w.ldh;
}

extern "C" int o5_ppo_loss_grad_factored(o5_dtype dt, int N, int H, int K, const int* head_sizes, const void* h,
                                         const void* Wp, const float* bp, const int32_t* act, const float* logp_old,
                                         const float* adv, const float* ret, const uint8_t* head_mask,
                                         const uint8_t* avail, const o5_unit_head* unit, o5_ppo_hp hp, float* stats,
                                         uint16_t* P, uint16_t* W, int ld, float* dWp, float* dbp, void* ws,
                                         size_t ws_bytes, void* stream) {
  O5_CHECK(dt == O5_BF16, O5_E_DTYPE, "o5_ppo_loss_grad_factored: the factored gradient is bf16 only (dt=%d)",
           static_cast<int>(dt));
  HeadsMeta hm;
  PpoWs w;
  int st = ppo_check("o5_ppo_loss_grad_factored", dt, N, H, K, head_sizes, h, Wp, bp, act, logp_old, adv, ret,
                     head_mask, avail, unit, hp, stats, dWp, dbp, ws, ws_bytes, &hm, &w);
  if (st != O5_OK) return st;
  O5_CHECK(ld == 2 * w.ldh, O5_E_SHAPE, "o5_ppo_loss_grad_factored: ld=%d, the heads need %d (o5_ppo_head_grad_ld)",
           ld, 2 * w.ldh);
  O5_PTR(P, "P");
  O5_PTR(W, "W");
  hipStream_t s = as_stream(stream);
  ktimer_begin(kSitePpo, s);
  st = ppo_impl<uint16_t>(N, H, hm, static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(Wp), bp, act,
                          logp_old, adv, ret, head_mask, avail, unit, hp, stats, nullptr, dWp, dbp,
                          static_cast<char*>(ws), w, s, P, W);
  ktimer_end(kSitePpo, s);
  return st;
}
