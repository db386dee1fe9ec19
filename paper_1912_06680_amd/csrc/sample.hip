// Rollout-inference heads and action sampling (section "Training System",
// subsection "Playing Dota using AI": each timestep the current observation
// goes through the policy and an action is sampled from its output
// distribution).
//
//   z = h Wp^T + bp                                GEMM, as in the loss
//   a_k = argmax_a (z_{k,a} + G),  G = -ln(-ln U)  Gumbel-max, per head
//   logp = sum_k log softmax(z_k)[a_k],  value = z[A]
//
// U comes from Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
// numbers: as easy as 1, 2, 3", SC'11): a counter-based generator, so each
// logit's noise is a pure function of (seed, counter, row, head, logit) and
// needs no generator state on the device.  One Philox block yields the noise
// for 4 consecutive logits of one head.
#include "gemm_plan.h"
#include "heads.h"
#include "philox.h"
#include "reduce.h"

namespace o5 {

// One wave per row b, kSampleWaves rows per block; lane l holds logit
// columns a = l + 64 i (i < CPL).  zpart: [S][B][A1] partial logits without
// bias.  avail [B][A] or null: unavailable logits are never drawn and leave
// the log-sum-exp; a head with no available logit gets action -1 and adds
// nothing to logp.  The noise of a logit does not depend on the mask.  Head
// kext (or none, -1) takes its logits from zext [B][n_kext] (the
// unit-selection head).
//
// Each lane draws the Philox block of its own columns (the four lanes of one
// block compute the same block), so a row's noise is one block time; per
// head the draw is a wave maximum of z + G followed by a wave minimum of the
// index among the lanes that attain it (ties to the lowest index), and the
// log-sum-exp a wave maximum and sum over the available logits.  All
// reductions have a fixed order.
constexpr int kSampleWaves = 4;

__device__ const uint8_t kSampleAllAvailable = 1;
__device__ const float kSampleNoLogit = 0.0f;

template <int CPL>
__global__ void __launch_bounds__(kSampleWaves * 64) gumbel_sample_rows(
    int B, int A1, int S, const float* __restrict__ zpart, const float* __restrict__ bp,
    const uint8_t* __restrict__ avail, HeadsMeta hm, const float* __restrict__ zext, int kext, uint64_t seed,
    uint64_t counter, int32_t* __restrict__ act, float* __restrict__ logp, float* __restrict__ value) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * kSampleWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (b >= B) return;  // the whole wave
  const int K = hm.K, A = hm.A;
  const size_t sstride = static_cast<size_t>(B) * A1;
  const int nke = kext >= 0 ? hm.off[kext + 1] - hm.off[kext] : 0;
  const uint8_t* avp = avail ? avail : &kSampleAllAvailable;
  const size_t avs = avail ? 1 : 0;
  const float* zep = zext ? zext : &kSampleNoLogit;
  const size_t zes = zext ? 1 : 0;
  int head[CPL], idx[CPL];  // head of each column held (-1: value column or beyond) and index within it
  float z[CPL], score[CPL];
  bool av[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int a = lane + 64 * i;
    head[i] = -1;
    idx[i] = 0;
    for (int k = 0; k < K; ++k)
      if (a >= hm.off[k] && a < hm.off[k + 1]) {
        head[i] = k;
        idx[i] = a - hm.off[k];
      }
    // every load reads a valid address; selects drop the ones not wanted
    const int ac = min(a, A1 - 1);
    float v = bp[ac];
    for (int s2 = 0; s2 < S; ++s2) v += zpart[s2 * sstride + static_cast<size_t>(b) * A1 + ac];
    const bool ext = head[i] >= 0 && head[i] == kext;
    const float ze = zep[(static_cast<size_t>(b) * nke + (ext ? idx[i] : 0)) * zes];
    z[i] = ext ? ze : a < A1 ? v : 0.0f;
    av[i] = head[i] >= 0 && avp[(static_cast<size_t>(b) * A + min(a, A - 1)) * avs] != 0;
    score[i] = -INFINITY;
    if (head[i] >= 0) {
      uint64_t c0 = static_cast<uint64_t>(idx[i] >> 2), c1 = static_cast<uint64_t>(head[i]),
               c2 = static_cast<uint64_t>(b), c3 = counter;
      philox4x64_10(c0, c1, c2, c3, seed, 0ull);
      const int w = idx[i] & 3;
      const uint64_t word = w == 0 ? c0 : w == 1 ? c1 : w == 2 ? c2 : c3;
      score[i] = z[i] - logf(-logf(philox_uniform24(word)));
    }
  }
  const auto wave_min = [](float v) { return wave_reduce(v, INFINITY, [](float x, float y) { return fminf(x, y); }); };
  float lp = 0.0f;
  for (int k = 0; k < K; ++k) {
    float best = -INFINITY, zm = -INFINITY, first = INFINITY;
#pragma unroll
    for (int i = 0; i < CPL; ++i)
      if (head[i] == k && av[i]) {
        best = fmaxf(best, score[i]);
        zm = fmaxf(zm, z[i]);
        first = fminf(first, static_cast<float>(idx[i]));
      }
    best = wave_max(best);
    zm = wave_max(zm);
    first = wave_min(first);  // the lowest available index (+inf: none)
    float cand = INFINITY, e = 0.0f;
#pragma unroll
    for (int i = 0; i < CPL; ++i)
      if (head[i] == k && av[i]) {
        if (score[i] == best) cand = fminf(cand, static_cast<float>(idx[i]));
        e += expf(z[i] - zm);
      }
    cand = wave_min(cand);
    e = wave_sum(e);
    int a_k = -1;
    if (first < INFINITY) {
      a_k = cand < INFINITY ? static_cast<int>(cand) : static_cast<int>(first);  // (no finite score: first available)
      lp += column(z, hm.off[k] + a_k) - (zm + logf(e));
    }
    if (lane == 0) act[static_cast<size_t>(b) * K + k] = a_k;
  }
  const float v = column(z, A);
  if (lane == 0) {
    logp[b] = lp;
    value[b] = v;
  }
}

// zpart, then the unit-selection head's scratch (if any) at *unit_off.
static size_t sample_ws_bytes(o5_dtype dt, int B, int H, int A1, GemmPlan* plan, int unit_nk, int unit_d,
                              UnitWs* uw, size_t* unit_off) {
  *plan = plan_gemm(dt == O5_BF16, B, A1, H);
  size_t o = align_up(static_cast<size_t>(plan->splits) * B * A1 * 4);
  *unit_off = o;
  if (unit_d > 0) {
    *uw = unit_ws(dt, B, H, unit_nk, unit_d, false);
    o += align_up(uw->total);
  }
  return o;
}

}  // namespace o5

using namespace o5;

extern "C" size_t o5_policy_sample_workspace_bytes(o5_dtype dt, int B, int H, int K, const int* head_sizes,
                                                   const o5_unit_head* unit) {
  HeadsMeta hm;
  if (check_heads("o5_policy_sample_workspace_bytes", dt, B, H, K, head_sizes, &hm) != O5_OK) return 0;
  if (unit != nullptr && (unit->head < 0 || unit->head >= K || unit->d < 8 || unit->d > 512 || (unit->d & (unit->d - 1)) != 0)) return 0;
  GemmPlan p;
  UnitWs uw;
  size_t uo;
  return sample_ws_bytes(dt, B, H, hm.A + 1, &p, unit ? hm.off[unit->head + 1] - hm.off[unit->head] : 0,
                         unit ? unit->d : 0, &uw, &uo);
}

namespace o5 {

int policy_sample_check(const char* fn, o5_dtype dt, int B, int H, int K, const int* head_sizes, const void* h,
                        const void* Wp, const float* bp, const uint8_t* avail, const o5_unit_head* unit,
                        const int32_t* act, const float* logp, const float* value, HeadsMeta* hm, size_t* need) {
  int st = check_heads(fn, dt, B, H, K, head_sizes, hm);
  if (st != O5_OK) return st;
  O5_CHECK(h != nullptr && Wp != nullptr && bp != nullptr, O5_E_NULL, "%s: h, Wp and bp must not be NULL", fn);
  O5_CHECK(aligned16(h) && aligned16(Wp) && aligned16(bp), O5_E_ALIGN, "%s: h, Wp or bp is not 16-byte aligned", fn);
  O5_CHECK(avail == nullptr || aligned16(avail), O5_E_ALIGN, "%s: avail is not 16-byte aligned", fn);
  if (unit != nullptr) {
    st = check_unit(fn, *hm, unit, false);
    if (st != O5_OK) return st;
  }
  O5_CHECK(act != nullptr && logp != nullptr && value != nullptr, O5_E_NULL, "%s: act, logp and value must not be NULL",
           fn);
  O5_CHECK(aligned16(act) && aligned16(logp) && aligned16(value), O5_E_ALIGN,
           "%s: act, logp or value is not 16-byte aligned", fn);
  GemmPlan plan;
  UnitWs uw;
  size_t unit_off;
  *need = sample_ws_bytes(dt, B, H, hm->A + 1, &plan, unit ? hm->off[unit->head + 1] - hm->off[unit->head] : 0,
                          unit ? unit->d : 0, &uw, &unit_off);
  return O5_OK;
}

int policy_sample_run(o5_dtype dt, int B, int H, const HeadsMeta& hm, const void* h, const void* Wp, const float* bp,
                      const uint8_t* avail, const o5_unit_head* unit, uint64_t seed, uint64_t counter, int32_t* act,
                      float* logp, float* value, char* ws, hipStream_t s) {
  GemmPlan plan;
  UnitWs uw;
  size_t unit_off;
  const int unit_nk = unit ? hm.off[unit->head + 1] - hm.off[unit->head] : 0;
  sample_ws_bytes(dt, B, H, hm.A + 1, &plan, unit_nk, unit ? unit->d : 0, &uw, &unit_off);
  const int A1 = hm.A + 1;
  float* zpart = reinterpret_cast<float*>(ws);
  ktimer_begin(kSiteSample, s);
  if (dt == O5_BF16) {
    KRows2<uint16_t> al{static_cast<const uint16_t*>(h), nullptr, nullptr, H, 0, H, H, B};
    KRows2<uint16_t> bl{static_cast<const uint16_t*>(Wp), nullptr, nullptr, H, 0, H, H, A1};
    run_gemm(plan, al, bl, EpiStoreF32{zpart, A1, static_cast<size_t>(B) * A1}, B, A1, H, s);
  } else {
    KRows2<float> al{static_cast<const float*>(h), nullptr, nullptr, H, 0, H, H, B};
    KRows2<float> bl{static_cast<const float*>(Wp), nullptr, nullptr, H, 0, H, H, A1};
    run_gemm(plan, al, bl, EpiStoreF32{zpart, A1, static_cast<size_t>(B) * A1}, B, A1, H, s);
  }
  const float* zext = nullptr;
  if (unit != nullptr) {
    char* uws = ws + unit_off;
    unit_forward(dt, B, H, unit_nk, *unit, h, uws, uw, s);
    zext = reinterpret_cast<const float*>(uws + uw.zext);
  }
  const int cpl = cdiv(A1, 64);
  const dim3 grid(cdiv(B, kSampleWaves)), block(kSampleWaves * 64);
  const int kext = unit ? unit->head : -1;
  if (cpl <= 1)
    hipLaunchKernelGGL(gumbel_sample_rows<1>, grid, block, 0, s, B, A1, plan.splits, zpart, bp, avail, hm, zext, kext,
                       seed, counter, act, logp, value);
  else if (cpl <= 2)
    hipLaunchKernelGGL(gumbel_sample_rows<2>, grid, block, 0, s, B, A1, plan.splits, zpart, bp, avail, hm, zext, kext,
                       seed, counter, act, logp, value);
  else if (cpl <= 4)
    hipLaunchKernelGGL(gumbel_sample_rows<4>, grid, block, 0, s, B, A1, plan.splits, zpart, bp, avail, hm, zext, kext,
                       seed, counter, act, logp, value);
  else if (cpl <= 8)
    hipLaunchKernelGGL(gumbel_sample_rows<8>, grid, block, 0, s, B, A1, plan.splits, zpart, bp, avail, hm, zext, kext,
                       seed, counter, act, logp, value);
  else
    hipLaunchKernelGGL(gumbel_sample_rows<16>, grid, block, 0, s, B, A1, plan.splits, zpart, bp, avail, hm, zext, kext,
                       seed, counter, act, logp, value);
  ktimer_end(kSiteSample, s);
  return check_launch("o5_policy_sample");
}

}  // namespace o5

extern "C" int o5_policy_sample(o5_dtype dt, int B, int H, int K, const int* head_sizes, const void* h, const void* Wp,
                                const float* bp, const uint8_t* avail, const o5_unit_head* unit, uint64_t seed,
                                uint64_t counter, int32_t* act, float* logp, float* value, void* ws, size_t ws_bytes,
                                void* stream) {
  HeadsMeta hm;
  size_t need = 0;
  const int st = policy_sample_check("o5_policy_sample", dt, B, H, K, head_sizes, h, Wp, bp, avail, unit, act, logp,
                                     value, &hm, &need);
  if (st != O5_OK) return st;
  O5_CHECK(ws != nullptr && ws_bytes >= need, O5_E_WORKSPACE, "o5_policy_sample: workspace needs %zu bytes, got %zu",
           need, ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "o5_policy_sample: ws is not 16-byte aligned");
  return policy_sample_run(dt, B, H, hm, h, Wp, bp, avail, unit, seed, counter, act, logp, value,
                           static_cast<char*>(ws), as_stream(stream));
}
