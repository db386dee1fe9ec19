// Policy and value heads, PPO clipped-surrogate loss, value loss and entropy
// bonus, and their gradients (appendix "Neural Network Architecture":
// linear projections of the LSTM state for the action logits and the value,
// sharing the network and its gradients; appendix "Action Space": factorised
// action, ignored parameter heads masked out of the optimisation;
// subsection "Optimizing the Policy" and Table "Hyperparameters": clip 0.2,
// value loss weight 1.0; appendix "Exploration": entropy bonus 0.01).
//
//   z   = h Wp^T                        GEMM  (M = N rows, N = A+1, K = H)
//   row kernel: + bp, per-head log-softmax, joint log-ratio, clipped
//        surrogate, value error, entropy -> dz [N, A+1] and per-row stats
//   dh  = dz Wp                         GEMM  (M = N, N = H, K = A+1)
//   dWp = dz^T h                        GEMM  (M = A+1, N = H, K = N), split-K
//   dbp, stats: fixed-order column sums.
// On the bf16 path the two gradient products run on the MFMA engine: dz is
// written as a pair of bf16 terms hi = bf16(dz), lo = bf16(dz - hi) (relative
// error ~2^-16) laid side by side along K, against the bf16 operand repeated
// twice, so the product keeps nearly fp32 accuracy.
// Every reduction has a fixed order, so results are bitwise reproducible.
#include "gemm_plan.h"
#include "heads.h"
#include "reduce.h"

namespace o5 {

constexpr int kStatCols = 8;

// The logits store: an EpiStoreF32 under its own type name, so the heads
// GEMM is a kernel symbol of its own in profiles.
struct EpiLogits : EpiStoreF32 {};
constexpr int kRowsPerChunk = 256;

// One thread per row.  zpart: [S][N][A1] partial logits (bias not added).
// dz doubles as the row's logit scratch: it first receives z, then dL/dz.
__global__ void __launch_bounds__(256) ppo_rows(int N, int A1, int S, const float* __restrict__ zpart,
                                                const float* __restrict__ bp, const int32_t* __restrict__ act,
                                                const float* __restrict__ logp_old, const float* __restrict__ adv,
                                                const float* __restrict__ ret, const uint8_t* __restrict__ mask,
                                                HeadsMeta hm, float clip_eps, float vf_coef, float ent_coef,
                                                float invN, float* __restrict__ dz, float* __restrict__ rowstats,
                                                uint16_t* __restrict__ dz_hi, uint16_t* __restrict__ dz_lo,
                                                int ld_hilo) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  float* zr = dz + static_cast<size_t>(n) * A1;
  const size_t sstride = static_cast<size_t>(N) * A1;
  for (int a = 0; a < A1; ++a) {
    float v = bp[a];
    for (int s = 0; s < S; ++s) v += zpart[s * sstride + static_cast<size_t>(n) * A1 + a];
    zr[a] = v;
  }
  float lse[kMaxHeads], zbar[kMaxHeads], mk[kMaxHeads];
  int ak[kMaxHeads];
  float logpi = 0.0f, ent = 0.0f;
  for (int k = 0; k < hm.K; ++k) {
    const int o = hm.off[k], nk = hm.off[k + 1] - o;
    float zmax = -INFINITY;
    for (int a = 0; a < nk; ++a) zmax = fmaxf(zmax, zr[o + a]);
    float se = 0.0f, sez = 0.0f;
    for (int a = 0; a < nk; ++a) {
      const float e = expf(zr[o + a] - zmax);
      se += e;
      sez += e * zr[o + a];
    }
    lse[k] = zmax + logf(se);
    zbar[k] = sez / se;
    ak[k] = act[static_cast<size_t>(n) * hm.K + k];
    mk[k] = mask ? (mask[static_cast<size_t>(n) * hm.K + k] ? 1.0f : 0.0f) : 1.0f;
    const int a_sel = min(max(ak[k], 0), nk - 1);
    logpi += mk[k] * (zr[o + a_sel] - lse[k]);
    ent += mk[k] * (lse[k] - zbar[k]);
  }
  const float A = adv[n], R = ret[n];
  const float dlog = logpi - logp_old[n];
  const float ratio = expf(dlog);
  const float rc = fminf(fmaxf(ratio, 1.0f - clip_eps), 1.0f + clip_eps);
  const float surr = fminf(ratio * A, rc * A);
  const float V = zr[hm.A];
  const float verr = V - R;
  const bool flow = (A >= 0.0f && ratio <= 1.0f + clip_eps) || (A < 0.0f && ratio >= 1.0f - clip_eps);
  const float g_logpi = flow ? -ratio * A * invN : 0.0f;
  const float ent_scale = ent_coef * invN;
  for (int k = 0; k < hm.K; ++k) {
    const int o = hm.off[k], nk = hm.off[k + 1] - o;
    for (int a = 0; a < nk; ++a) {
      const float z = zr[o + a];
      const float p = expf(z - lse[k]);
      const float onehot = (a == ak[k]) ? 1.0f : 0.0f;
      zr[o + a] = mk[k] * (g_logpi * (onehot - p) + ent_scale * p * (z - zbar[k]));
    }
  }
  zr[hm.A] = 2.0f * vf_coef * verr * invN;
  if (dz_hi != nullptr) {  // bf16 pair (hi, lo) of the row, zero-padded to ld_hilo
    uint16_t* hr = dz_hi + static_cast<size_t>(n) * ld_hilo;
    uint16_t* lr = dz_lo + static_cast<size_t>(n) * ld_hilo;
    for (int a = 0; a < ld_hilo; ++a) {
      const float v = a < A1 ? zr[a] : 0.0f;
      const uint16_t hb = f32_to_bf16_bits(v);
      hr[a] = hb;
      lr[a] = f32_to_bf16_bits(v - bf16_bits_to_f32(hb));
    }
  }
  const float row_loss = -surr + vf_coef * verr * verr - ent_coef * ent;
  float* st = rowstats + static_cast<size_t>(n) * kStatCols;
  st[0] = surr;
  st[1] = verr * verr;
  st[2] = ent;
  st[3] = fabsf(ratio - 1.0f) > clip_eps ? 1.0f : 0.0f;
  st[4] = (ratio - 1.0f) - dlog;
  st[5] = ratio;
  st[6] = isfinite(row_loss) ? 0.0f : 1.0f;
  st[7] = 0.0f;
}

// dst [R, H] bf16 = src [A1, H] with rows A1..R-1 zero.
__global__ void __launch_bounds__(256) pad_rows_bf16(int A1, int R, int H, const uint16_t* __restrict__ src,
                                                     uint16_t* __restrict__ dst) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const size_t total = static_cast<size_t>(R) * H;
  if (i >= total) return;
  const int r = static_cast<int>(i / H);
  dst[i] = r < A1 ? src[i] : static_cast<uint16_t>(0);
}

__global__ void ppo_finalize(const float* __restrict__ sums, float invN, float vf_coef, float ent_coef,
                             float* __restrict__ stats) {
  if (threadIdx.x != 0) return;
  const float pg = -sums[0] * invN, vf = sums[1] * invN, ent = sums[2] * invN;
  stats[0] = pg + vf_coef * vf - ent_coef * ent;
  stats[1] = pg;
  stats[2] = vf;
  stats[3] = ent;
  stats[4] = sums[3] * invN;
  stats[5] = sums[4] * invN;
  stats[6] = sums[5] * invN;
  stats[7] = sums[6];
}

struct PpoWs {
  size_t zpart, dz, rowstats, wpart, dbpart, spart, ssum, dzhi, dzlo, wpad, total;
  GemmPlan plan_z, plan_w, plan_h;
  int nchunk, A1, A1p;
};

static PpoWs ppo_ws(o5_dtype dt, int N, int H, int A1) {
  PpoWs w;
  const bool bf = dt == O5_BF16;
  w.A1 = A1;
  w.A1p = cdiv(A1, 64) * 64;  // padded logit count: a multiple of the K tile
  w.plan_z = plan_gemm(bf, N, A1, H);
  w.plan_w = bf ? plan_gemm(true, A1, H, 2 * N) : plan_gemm(false, A1, H, N);
  w.plan_h = bf ? plan_gemm(true, N, H, 2 * w.A1p) : GemmPlan{false, BfTile::k128x128, 1};
  w.plan_h.splits = 1;
  w.nchunk = cdiv(N, kRowsPerChunk);
  size_t o = 0;
  w.zpart = o;
  o += align_up(static_cast<size_t>(w.plan_z.splits) * N * A1 * 4);
  w.dz = o;
  o += align_up(static_cast<size_t>(N) * A1 * 4);
  w.rowstats = o;
  o += align_up(static_cast<size_t>(N) * kStatCols * 4);
  w.wpart = o;
  o += align_up(static_cast<size_t>(w.plan_w.splits) * A1 * H * 4);
  w.dbpart = o;
  o += align_up(static_cast<size_t>(w.nchunk) * A1 * 4);
  w.spart = o;
  o += align_up(static_cast<size_t>(w.nchunk) * kStatCols * 4);
  w.ssum = o;
  o += align_up(kStatCols * 4);
  w.dzhi = w.dzlo = w.wpad = 0;
  if (bf) {
    w.dzhi = o;
    o += align_up(static_cast<size_t>(N) * w.A1p * 2);
    w.dzlo = o;
    o += align_up(static_cast<size_t>(N) * w.A1p * 2);
    w.wpad = o;
    o += align_up(static_cast<size_t>(w.A1p) * H * 2);
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

template <typename E>
static int ppo_impl(int N, int H, const HeadsMeta& hm, const E* h, const E* Wp, const float* bp, const int32_t* act,
                    const float* logp_old, const float* adv, const float* ret, const uint8_t* mask, o5_ppo_hp hp,
                    float* stats, float* dh, float* dWp, float* dbp, char* ws, const PpoWs& w, hipStream_t s) {
  const int A1 = hm.A + 1;
  float* zpart = reinterpret_cast<float*>(ws + w.zpart);
  float* dz = reinterpret_cast<float*>(ws + w.dz);
  float* rowstats = reinterpret_cast<float*>(ws + w.rowstats);
  float* wpart = reinterpret_cast<float*>(ws + w.wpart);
  float* dbpart = reinterpret_cast<float*>(ws + w.dbpart);
  float* spart = reinterpret_cast<float*>(ws + w.spart);
  float* ssum = reinterpret_cast<float*>(ws + w.ssum);
  const float invN = 1.0f / static_cast<float>(N);
  {  // z = h Wp^T
    KRows2<E> al{h, nullptr, nullptr, H, 0, H, H, N};
    KRows2<E> bl{Wp, nullptr, nullptr, H, 0, H, H, A1};
    EpiLogits epi{{zpart, A1, static_cast<size_t>(N) * A1}};
    run_gemm(w.plan_z, al, bl, epi, N, A1, H, s);
  }
  uint16_t* dzhi = nullptr;
  uint16_t* dzlo = nullptr;
  if constexpr (sizeof(E) == 2) {
    dzhi = reinterpret_cast<uint16_t*>(ws + w.dzhi);
    dzlo = reinterpret_cast<uint16_t*>(ws + w.dzlo);
  }
  hipLaunchKernelGGL(ppo_rows, dim3(cdiv(N, 256)), dim3(256), 0, s, N, A1, w.plan_z.splits, zpart, bp, act, logp_old,
                     adv, ret, mask, hm, hp.clip_eps, hp.vf_coef, hp.ent_coef, invN, dz, rowstats, dzhi, dzlo, w.A1p);
  if constexpr (sizeof(E) == 2) {
    const int A1p = w.A1p;
    uint16_t* wpad = reinterpret_cast<uint16_t*>(ws + w.wpad);
    hipLaunchKernelGGL(pad_rows_bf16, dim3(cdiv(static_cast<long long>(A1p) * H, 256)), dim3(256), 0, s, A1, A1p, H,
                       Wp, wpad);
    {  // dh = [dz_hi | dz_lo] . [Wp ; Wp]  (K = 2 A1p)
      KRows2<uint16_t> al{dzhi, dzlo, nullptr, A1p, A1p, A1p, 2 * A1p, N};
      ICols2<uint16_t> bl{wpad, wpad, wpad, nullptr, H, H, 0, H, 2 * A1p, A1p};
      EpiStoreF32 epi{dh, H, 0};
      run_gemm(w.plan_h, al, bl, epi, N, H, 2 * A1p, s);
    }
    {  // dWp = [dz_hi ; dz_lo]^T . [h ; h]  (K = 2N), split over K, fixed-order sum
      ICols2<uint16_t> al{dzhi, dzhi, dzlo, nullptr, A1p, A1p, 0, A1p, 2 * N, N};
      ICols2<uint16_t> bl{h, h, h, nullptr, H, H, 0, H, 2 * N, N};
      EpiStoreF32 epi{wpart, H, static_cast<size_t>(A1) * H};
      run_gemm(w.plan_w, al, bl, epi, A1, H, 2 * N, s);
    }
  } else {
    {  // dh = dz Wp  (fp32 FMA engine)
      KRows2<float> al{dz, nullptr, nullptr, A1, 0, A1, A1, N};
      ICols2<E> bl{Wp, nullptr, nullptr, nullptr, H, 0, H, H, A1, 0};
      EpiStoreF32 epi{dh, H, 0};
      launch_gemm_f32(al, bl, epi, N, H, A1, 1, s);
    }
    {  // dWp = dz^T h, split over rows
      ICols2<float> al{dz, nullptr, nullptr, nullptr, A1, 0, A1, A1, N, 0};
      ICols2<E> bl{h, nullptr, nullptr, nullptr, H, 0, H, H, N, 0};
      EpiStoreF32 epi{wpart, H, static_cast<size_t>(A1) * H};
      launch_gemm_f32(al, bl, epi, A1, H, N, w.plan_w.splits, s);
    }
  }
  hipLaunchKernelGGL(colsum_rows, dim3(cdiv(static_cast<long long>(A1) * H, 256)), dim3(256), 0, s, w.plan_w.splits,
                     A1 * H, wpart, dWp);
  hipLaunchKernelGGL(colsum_chunks, dim3(cdiv(A1, 256), w.nchunk), dim3(256), 0, s, N, A1, kRowsPerChunk, dz, dbpart);
  hipLaunchKernelGGL(colsum_rows, dim3(cdiv(A1, 256)), dim3(256), 0, s, w.nchunk, A1, dbpart, dbp);
  hipLaunchKernelGGL(colsum_chunks, dim3(1, w.nchunk), dim3(256), 0, s, N, kStatCols, kRowsPerChunk, rowstats, spart);
  hipLaunchKernelGGL(colsum_rows, dim3(1), dim3(256), 0, s, w.nchunk, kStatCols, spart, ssum);
  hipLaunchKernelGGL(ppo_finalize, dim3(1), dim3(64), 0, s, ssum, invN, hp.vf_coef, hp.ent_coef, stats);
  return check_launch("o5_ppo_loss_grad");
}

}  // namespace o5

using namespace o5;

extern "C" size_t o5_ppo_loss_grad_workspace_bytes(o5_dtype dt, int N, int H, int K, const int* head_sizes) {
  HeadsMeta hm;
  if (check_heads("o5_ppo_loss_grad_workspace_bytes", dt, N, H, K, head_sizes, &hm) != O5_OK) return 0;
  return ppo_ws(dt, N, H, hm.A + 1).total;
}

extern "C" int o5_ppo_loss_grad(o5_dtype dt, int N, int H, int K, const int* head_sizes, const void* h, const void* Wp,
                                const float* bp, const int32_t* act, const float* logp_old, const float* adv,
                                const float* ret, const uint8_t* head_mask, o5_ppo_hp hp, float* stats, float* dh,
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
  O5_PTR(stats, "stats");
  O5_PTR(dh, "dh");
  O5_PTR(dWp, "dWp");
  O5_PTR(dbp, "dbp");
  const PpoWs w = ppo_ws(dt, N, H, hm.A + 1);
  O5_CHECK(ws != nullptr && ws_bytes >= w.total, O5_E_WORKSPACE,
           "o5_ppo_loss_grad: workspace needs %zu bytes, got %zu", w.total, ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "o5_ppo_loss_grad: ws is not 16-byte aligned");
  char* wsp = static_cast<char*>(ws);
  hipStream_t s = as_stream(stream);
  ktimer_begin(kSitePpo, s);
  if (dt == O5_BF16)
    st = ppo_impl<uint16_t>(N, H, hm, static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(Wp), bp, act,
                              logp_old, adv, ret, head_mask, hp, stats, dh, dWp, dbp, wsp, w, s);
  else
    st = ppo_impl<float>(N, H, hm, static_cast<const float*>(h), static_cast<const float*>(Wp), bp, act, logp_old, adv,
                         ret, head_mask, hp, stats, dh, dWp, dbp, wsp, w, s);
  ktimer_end(kSitePpo, s);
  return st;
}
