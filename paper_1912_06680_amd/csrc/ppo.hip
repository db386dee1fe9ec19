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

// One wave per row, kRowsPerWave consecutive rows per wave; lane l holds
// logit columns l + 64 i (i < CPL).  zpart: [S][N][A1] partial logits (bias
// not added).  avail [N][A] (or null = all available): an unavailable logit
// is left out of its head's softmax and gets no gradient; a head with no
// available logit adds nothing; an unavailable taken action has
// log-probability -inf.  Head kext (or none, -1) takes its logits from zext
// [N][n_kext] (the unit-selection head) and returns their gradient in dzext
// instead of dz and its sums.  Writes dz [N][A1]; on the bf16 path the (hi, lo) pair in row
// layout [N][ld_hilo] and, when dzT is set, transposed as [2 ld_hilo][ldT]
// (hi rows, then lo rows; columns n >= N zero).  Each block writes one row
// of part: the column sums of its dz (A1 values), then the sums of its rows'
// surrogate, squared value error, entropy, clip indicator, approx-KL term,
// ratio and non-finite indicator (kStatCols values); all sums in a fixed
// order.
// Read in place of an absent availability mask and unit-head logits.
__device__ const uint8_t kAllAvailable = 1;
__device__ const float kNoLogit = 0.0f;

template <int CPL, int SMAX>
__global__ void __launch_bounds__(kWavesPerBlock * 64) ppo_rows(
    int N, int A1, int S, const float* __restrict__ zpart, const float* __restrict__ bp,
    const int32_t* __restrict__ act, const float* __restrict__ logp_old, const float* __restrict__ adv,
    const float* __restrict__ ret, const uint8_t* __restrict__ mask, const uint8_t* __restrict__ avail, HeadsMeta hm,
    const float* __restrict__ zext, float* __restrict__ dzext, int kext, float clip_eps, float vf_coef,
    float ent_coef, float invN, float* __restrict__ dz, float* __restrict__ part, uint16_t* __restrict__ dz_hi,
    uint16_t* __restrict__ dz_lo, int ncol_hilo, int ld_hilo, uint16_t* __restrict__ dzT, int ldT) {
  __shared__ float red[kWavesPerBlock][CPL * 64 + kStatCols];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int K = hm.K, A = hm.A;
  int head[CPL];  // head of each column held, -1 for the value column and beyond
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int a = lane + 64 * i;
    head[i] = -1;
    for (int k = 0; k < K; ++k)
      if (a >= hm.off[k] && a < hm.off[k + 1]) head[i] = k;
  }
  float csum[CPL] = {};
  float st[kStatCols] = {};
  // the transposed pair is kept in registers (16 rows x 2 bytes per column)
  // only for up to 256 logit columns; beyond that dzT must be null
  constexpr bool kT = CPL <= 4;
  constexpr int TC = kT ? CPL : 1;
  uint32_t thi[TC][kRowsPerWave / 2] = {}, tlo[TC][kRowsPerWave / 2] = {};
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
    float z[CPL];
    bool av[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      z[i] = zr[0][i];
      av[i] = lane + 64 * i >= A || avr[0][i] != 0;
    }
    float lse[kMaxHeads], zbar[kMaxHeads];
    bool mk[kMaxHeads], some[kMaxHeads];
    int ak[kMaxHeads];
    float logpi = 0.0f, ent = 0.0f;
    // per head: the maximum over its available logits; then one exponential
    // per column; then the sums of e and e z per head (all reductions over
    // the wave in a fixed order)
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
        ak[k] = __builtin_amdgcn_readlane(actr[0], k);
        mk[k] = __builtin_amdgcn_readlane(static_cast<int>(mkr[0]), k) != 0;
        const int nk = hm.off[k + 1] - hm.off[k];
        const int a_sel = min(max(ak[k], 0), nk - 1);
        const int c_sel = hm.off[k] + a_sel;
        const float z_sel = column(z, c_sel);
        uint32_t tb = avr[0][0];
#pragma unroll
        for (int i = 1; i < CPL; ++i)
          if (c_sel >> 6 == i) tb = avr[0][i];
        const bool taken = __builtin_amdgcn_readlane(static_cast<int>(tb), c_sel & 63) != 0;
        if (mk[k] && some[k]) {
          logpi += taken ? z_sel - lse[k] : -INFINITY;
          ent += lse[k] - zbar[k];
        }
      }
    }
    const float Ad = advr[0], R = retr[0];
    const float dlog = logpi - lpor[0];
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
      float d = 0.0f;
      if (a == A) d = 2.0f * vf_coef * verr * invN;
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
        d = g_logpi * (onehot - p) + ent_scale * p * (z[i] - zb);
      }
      if (head[i] >= 0 && head[i] == kext) {
        dzext[static_cast<size_t>(n) * nke + (a - hm.off[kext])] = d;
        d = 0.0f;  // these logits do not depend on Wp, bp
      }
      if (a < A1) dz[static_cast<size_t>(n) * A1 + a] = d;
      csum[i] += d;
      if (dz_hi != nullptr && a < ncol_hilo) {
        const uint16_t hb = f32_to_bf16_bits(d);
        const uint16_t lb = f32_to_bf16_bits(d - bf16_bits_to_f32(hb));
        dz_hi[static_cast<size_t>(n) * ld_hilo + a] = hb;
        dz_lo[static_cast<size_t>(n) * ld_hilo + a] = lb;
        if constexpr (kT) {
          const int sh = (rr & 1) * 16;
#pragma unroll
          for (int q = 0; q < kRowsPerWave / 2; ++q)
            if (q == rr >> 1) {
              thi[i][q] |= static_cast<uint32_t>(hb) << sh;
              tlo[i][q] |= static_cast<uint32_t>(lb) << sh;
            }
        }
      }
    }
    const float row_loss = -surr + vf_coef * verr * verr - ent_coef * ent;
    st[0] += surr;
    st[1] += verr * verr;
    st[2] += ent;
    st[3] += fabsf(ratio - 1.0f) > clip_eps ? 1.0f : 0.0f;
    st[4] += expm1f(dlog) - dlog;  // (r - 1) - log r without the cancellation in r - 1
    st[5] += ratio;
    st[6] += isfinite(row_loss) ? 0.0f : 1.0f;
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
  if (kT && dzT != nullptr) {
    // kRowsPerWave consecutive rows of each column held: 8 bytes of a dz^T row
    static_assert(kRowsPerWave == 4, "one 8-byte store per column and half");
#pragma unroll
    for (int i = 0; i < TC; ++i) {
      const int a = lane + 64 * i;
      if (a < ncol_hilo) {
        *reinterpret_cast<uint2*>(dzT + static_cast<size_t>(a) * ldT + n0) = make_uint2(thi[i][0], thi[i][1]);
        *reinterpret_cast<uint2*>(dzT + static_cast<size_t>(ncol_hilo + a) * ldT + n0) =
            make_uint2(tlo[i][0], tlo[i][1]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < CPL; ++i) red[wave][64 * i + lane] = csum[i];
  if (lane < kStatCols) {
    float v = 0.0f;
#pragma unroll
    for (int q = 0; q < kStatCols; ++q)
      if (q == lane) v = st[q];
    red[wave][CPL * 64 + lane] = v;
  }
  __syncthreads();
  const int W = A1 + kStatCols;
  for (int t = threadIdx.x; t < W; t += blockDim.x) {
    const int c = t < A1 ? t : CPL * 64 + (t - A1);
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) v += red[w][c];
    part[static_cast<size_t>(blockIdx.x) * W + t] = v;
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
  size_t zpart, dz, part, sums, wpart, dzhi, dzlo, dzT, wpad, unit, total;
  UnitWs uw;  // the unit-selection head's scratch, at offset unit (if any)
  GemmPlan plan_z, plan_w, plan_h;
  int nblk, A1, A1p, ldh, ldT, wsplits;  // ldh: row length of the (hi, lo) pair, A1p + the unit head's dp
  bool dwp_t;  // dWp from the transposed (hi; lo) pair, h read once
};

static PpoWs ppo_ws(o5_dtype dt, int N, int H, int A1, int unit_nk = 0, int unit_d = 0) {
  PpoWs w{};
  const bool bf = dt == O5_BF16;
  w.A1 = A1;
  w.A1p = cdiv(A1, 64) * 64;  // padded logit count: a multiple of the K tile
  w.ldh = w.A1p + (unit_d > 0 ? cdiv(unit_d, 64) * 64 : 0);
  w.nblk = cdiv(N, kRowsPerBlock);
  w.ldT = w.nblk * kRowsPerBlock;
  w.dwp_t = bf && w.A1p <= 256;
  w.plan_z = plan_gemm(bf, N, A1, H);
  w.plan_w = bf ? plan_gemm(true, A1, H, 2 * N) : plan_gemm(false, A1, H, N);
  w.plan_h = bf ? plan_gemm(true, N, H, 2 * w.ldh) : GemmPlan{false, BfTile::k128x128, 1, 256};
  w.plan_h.splits = 1;
  w.wsplits = 1;
  if (w.dwp_t) {
    // M = 2 A1p (one or two 256-row tiles), N = H, K = N: split K so the
    // grid has about 256 blocks, each with at least 8 K tiles of 32
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
  o += align_up(w.dwp_t ? static_cast<size_t>(w.wsplits) * 2 * w.A1p * H * 4
                        : static_cast<size_t>(w.plan_w.splits) * A1 * H * 4);
  w.dzhi = w.dzlo = w.dzT = w.wpad = 0;
  if (bf) {
    w.dzhi = o;
    o += align_up(static_cast<size_t>(N) * w.ldh * 2);
    w.dzlo = o;
    o += align_up(static_cast<size_t>(N) * w.ldh * 2);
    w.wpad = o;
    o += align_up(static_cast<size_t>(w.ldh) * H * 2);
    if (w.dwp_t) {
      w.dzT = o;
      o += align_up(static_cast<size_t>(2) * w.A1p * w.ldT * 2);
    }
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
                        uint16_t* dzT, hipStream_t s) {
  hipLaunchKernelGGL((ppo_rows<CPL, SMAX>), dim3(w.nblk), dim3(kWavesPerBlock * 64), 0, s, N, A1, S, zpart, bp, act,
                     logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp.clip_eps, hp.vf_coef, hp.ent_coef, invN,
                     dz, part, dzhi, dzlo, w.A1p, w.ldh, dzT, w.ldT);
}

// The row kernel unrolls its reads of the logits GEMM's split partials up
// to SMAX (2 covers the usual split, 16 every plan).
template <int CPL>
static void launch_rows(const PpoWs& w, int N, int A1, int S, const float* zpart, const float* bp, const int32_t* act,
                        const float* logp_old, const float* adv, const float* ret, const uint8_t* mask,
                        const uint8_t* avail, const HeadsMeta& hm, const float* zext, float* dzext, int kext,
                        o5_ppo_hp hp, float invN, float* dz, float* part, uint16_t* dzhi, uint16_t* dzlo,
                        uint16_t* dzT, hipStream_t s) {
  if (S <= 2)
    launch_rows_s<CPL, 2>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp,
                          invN, dz, part, dzhi, dzlo, dzT, s);
  else
    launch_rows_s<CPL, 16>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp,
                           invN, dz, part, dzhi, dzlo, dzT, s);
}

template <typename E>
static int ppo_impl(int N, int H, const HeadsMeta& hm, const E* h, const E* Wp, const float* bp, const int32_t* act,
                    const float* logp_old, const float* adv, const float* ret, const uint8_t* mask,
                    const uint8_t* avail, const o5_unit_head* unit, o5_ppo_hp hp,
                    float* stats, float* dh, float* dWp, float* dbp, char* ws, const PpoWs& w, hipStream_t s) {
  const int A1 = hm.A + 1;
  float* zpart = reinterpret_cast<float*>(ws + w.zpart);
  float* dz = reinterpret_cast<float*>(ws + w.dz);
  float* part = reinterpret_cast<float*>(ws + w.part);
  float* sums = reinterpret_cast<float*>(ws + w.sums);
  float* wpart = reinterpret_cast<float*>(ws + w.wpart);
  const float invN = 1.0f / static_cast<float>(N);
  {  // z = h Wp^T
    KRows2<E> al{h, nullptr, nullptr, H, 0, H, H, N};
    KRows2<E> bl{Wp, nullptr, nullptr, H, 0, H, H, A1};
    EpiLogits epi{{zpart, A1, static_cast<size_t>(N) * A1}};
    run_gemm(w.plan_z, al, bl, epi, N, A1, H, s);
  }
  uint16_t* dzhi = nullptr;
  uint16_t* dzlo = nullptr;
  uint16_t* dzT = nullptr;
  if constexpr (sizeof(E) == 2) {
    dzhi = reinterpret_cast<uint16_t*>(ws + w.dzhi);
    dzlo = reinterpret_cast<uint16_t*>(ws + w.dzlo);
    if (w.dwp_t) dzT = reinterpret_cast<uint16_t*>(ws + w.dzT);
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
  const int S = w.plan_z.splits;
  const int cpl = cdiv(A1, 64);
  if (cpl <= 1)
    launch_rows<1>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz, part,
                   dzhi, dzlo, dzT, s);
  else if (cpl <= 2)
    launch_rows<2>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz, part,
                   dzhi, dzlo, dzT, s);
  else if (cpl <= 4)
    launch_rows<4>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz, part,
                   dzhi, dzlo, dzT, s);
  else if (cpl <= 8)
    launch_rows<8>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz, part,
                   dzhi, dzlo, dzT, s);
  else
    launch_rows<16>(w, N, A1, S, zpart, bp, act, logp_old, adv, ret, mask, avail, hm, zext, dzext, kext, hp, invN, dz, part,
                   dzhi, dzlo, dzT, s);
  if constexpr (sizeof(E) == 2) {
    const int A1p = w.A1p, ldh = w.ldh;
    uint16_t* wpad = reinterpret_cast<uint16_t*>(ws + w.wpad);
    hipLaunchKernelGGL(pad_rows_bf16, dim3(cdiv(static_cast<long long>(A1p) * H, 256)), dim3(256), 0, s, A1, A1p, H,
                       Wp, wpad);
    if (unit != nullptr) {
      // dq (hi, lo) into columns A1p .. ldh - 1 of the pair, Wq into the same rows of wpad
      unit_grad(dt, N, H, w.uw.nk, *unit, h, uws, w.uw, dzhi, dzlo, A1p, ldh, s);
      const int d = unit->d, dp = ldh - A1p;
      hipLaunchKernelGGL(pad_rows_bf16, dim3(cdiv(static_cast<long long>(dp) * H, 256)), dim3(256), 0, s, d, dp, H,
                         static_cast<const uint16_t*>(unit->Wq), wpad + static_cast<size_t>(A1p) * H);
    }
    {  // dh = [dz_hi dq_hi | dz_lo dq_lo] . [Wp Wq ; Wp Wq]  (K = 2 ldh)
      KRows2<uint16_t> al{dzhi, dzlo, nullptr, ldh, ldh, ldh, 2 * ldh, N};
      ICols2<uint16_t> bl{wpad, wpad, wpad, nullptr, H, H, 0, H, 2 * ldh, ldh};
      EpiStoreF32 epi{dh, H, 0};
      run_gemm(w.plan_h, al, bl, epi, N, H, 2 * ldh, s);
    }
    if (w.dwp_t) {
      // [dWp_hi ; dWp_lo] = [hi ; lo]^T-rows . h  (M = 2 A1p, N = H, K = N), split over K
      KRows2<uint16_t> al{dzT, nullptr, nullptr, w.ldT, 0, N, N, 2 * A1p};
      ICols2<uint16_t> bl{h, nullptr, nullptr, nullptr, H, 0, H, H, N, 0};
      EpiStoreF32 epi{wpart, H, static_cast<size_t>(2) * A1p * H};
      launch_gemm_bf16_dma(al, bl, epi, 2 * A1p, H, N, w.wsplits, s);
      hipLaunchKernelGGL(sum_hilo_splits, dim3(cdiv(static_cast<long long>(A1) * H, 256)), dim3(256), 0, s,
                         w.wsplits, A1, A1p, H, wpart, dWp);
    } else {
      // dWp = [dz_hi ; dz_lo]^T . [h ; h]  (K = 2N), split over K, fixed-order sum
      ICols2<uint16_t> al{dzhi, dzhi, dzlo, nullptr, A1p, A1p, 0, A1p, 2 * N, N};
      ICols2<uint16_t> bl{h, h, h, nullptr, H, H, 0, H, 2 * N, N};
      EpiStoreF32 epi{wpart, H, static_cast<size_t>(A1) * H};
      run_gemm(w.plan_w, al, bl, epi, A1, H, 2 * N, s);
      hipLaunchKernelGGL(colsum_rows, dim3(cdiv(static_cast<long long>(A1) * H, 256)), dim3(256), 0, s,
                         w.plan_w.splits, A1 * H, wpart, dWp);
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
  hipLaunchKernelGGL(colsum_tree, dim3(A1 + kStatCols), dim3(256), 0, s, w.nblk, A1 + kStatCols, part, sums);
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

extern "C" int o5_ppo_loss_grad(o5_dtype dt, int N, int H, int K, const int* head_sizes, const void* h, const void* Wp,
                                const float* bp, const int32_t* act, const float* logp_old, const float* adv,
                                const float* ret, const uint8_t* head_mask, const uint8_t* avail,
                                const o5_unit_head* unit, o5_ppo_hp hp, float* stats, float* dh,
                                float* dWp, float* dbp, void* ws, size_t ws_bytes, void* stream) {
  HeadsMeta hm;
  int st = check_heads("o5_ppo_loss_grad", dt, N, H, K, head_sizes, &hm);
  if (st != O5_OK) return st;
  O5_CHECK(hp.clip_eps >= 0.0f && hp.clip_eps < 1.0f, O5_E_ARG, "o5_ppo_loss_grad: clip_eps=%g must be in [0, 1)",
           hp.clip_eps);
  O5_PTR(h, "h");
  O5_PTR(Wp, "Wp");
  O5_PTR(bp, "bp");
  O5_PTR(act, "act");
  O5_PTR(logp_old, "logp_old");
  O5_PTR(adv, "adv");
  O5_PTR(ret, "ret");
  O5_OPT_PTR(head_mask, "head_mask");
  O5_OPT_PTR(avail, "avail");
  if (unit != nullptr) {
    st = check_unit("o5_ppo_loss_grad", hm, unit, true);
    if (st != O5_OK) return st;
  }
  O5_PTR(stats, "stats");
  O5_PTR(dh, "dh");
  O5_PTR(dWp, "dWp");
  O5_PTR(dbp, "dbp");
  const PpoWs w = unit ? ppo_ws(dt, N, H, hm.A + 1, hm.off[unit->head + 1] - hm.off[unit->head], unit->d)
                       : ppo_ws(dt, N, H, hm.A + 1);
  O5_CHECK(ws != nullptr && ws_bytes >= w.total, O5_E_WORKSPACE,
           "o5_ppo_loss_grad: workspace needs %zu bytes, got %zu", w.total, ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "o5_ppo_loss_grad: ws is not 16-byte aligned");
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
