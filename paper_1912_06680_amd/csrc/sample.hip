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

namespace o5 {

// One thread per row b.  zpart: [S][B][A1] partial logits without bias.
// avail [B][A] or null: unavailable logits are never drawn and leave the
// log-sum-exp; a head with no available logit gets action -1 and adds
// nothing to logp.  The noise of a logit does not depend on the mask.  Head
// kext (or none, -1) takes its logits from zext [B][n_kext] (the
// unit-selection head).
__global__ void __launch_bounds__(256) gumbel_sample_rows(int B, int A1, int S, const float* __restrict__ zpart,
                                                          const float* __restrict__ bp,
                                                          const uint8_t* __restrict__ avail, HeadsMeta hm,
                                                          const float* __restrict__ zext, int kext, uint64_t seed,
                                                          uint64_t counter, int32_t* __restrict__ act,
                                                          float* __restrict__ logp, float* __restrict__ value) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const size_t sstride = static_cast<size_t>(B) * A1;
  const float* zrow = zpart + static_cast<size_t>(b) * A1;
  float lp = 0.0f;
  for (int k = 0; k < hm.K; ++k) {
    const int o = hm.off[k], nk = hm.off[k + 1] - o;
    float best = -INFINITY, zbest = 0.0f, zmax = -INFINITY, se = 0.0f;
    int besta = -1;
    uint64_t w[4] = {0, 0, 0, 0};
    for (int a = 0; a < nk; ++a) {
      if ((a & 3) == 0) {
        uint64_t c0 = static_cast<uint64_t>(a >> 2), c1 = static_cast<uint64_t>(k), c2 = static_cast<uint64_t>(b),
                 c3 = counter;
        philox4x64_10(c0, c1, c2, c3, seed, 0ull);
        w[0] = c0;
        w[1] = c1;
        w[2] = c2;
        w[3] = c3;
      }
      if (avail != nullptr && avail[static_cast<size_t>(b) * hm.A + o + a] == 0) continue;
      float z;
      if (k == kext) {
        z = zext[static_cast<size_t>(b) * nk + a];
      } else {
        z = bp[o + a];
        for (int s = 0; s < S; ++s) z += zrow[s * sstride + o + a];
      }
      const uint64_t word = (a & 3) == 0 ? w[0] : (a & 3) == 1 ? w[1] : (a & 3) == 2 ? w[2] : w[3];
      const float u = philox_uniform24(word);
      const float score = z - logf(-logf(u));
      if (besta < 0 || score > best) {
        best = score;
        besta = a;
        zbest = z;
      }
      // running log-sum-exp
      if (z > zmax) {
        se = se * expf(zmax - z) + 1.0f;
        zmax = z;
      } else {
        se += expf(z - zmax);
      }
    }
    act[static_cast<size_t>(b) * hm.K + k] = besta;
    if (besta >= 0) lp += zbest - (zmax + logf(se));
  }
  float v = bp[hm.A];
  for (int s = 0; s < S; ++s) v += zrow[s * sstride + hm.A];
  logp[b] = lp;
  value[b] = v;
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

extern "C" int o5_policy_sample(o5_dtype dt, int B, int H, int K, const int* head_sizes, const void* h, const void* Wp,
                                const float* bp, const uint8_t* avail, const o5_unit_head* unit, uint64_t seed,
                                uint64_t counter, int32_t* act,
                                float* logp,
                                float* value, void* ws, size_t ws_bytes, void* stream) {
  HeadsMeta hm;
  int st = check_heads("o5_policy_sample", dt, B, H, K, head_sizes, &hm);
  if (st != O5_OK) return st;
  O5_PTR(h, "h");
  O5_PTR(Wp, "Wp");
  O5_PTR(bp, "bp");
  O5_OPT_PTR(avail, "avail");
  if (unit != nullptr) {
    st = check_unit("o5_policy_sample", hm, unit, false);
    if (st != O5_OK) return st;
  }
  O5_PTR(act, "act");
  O5_PTR(logp, "logp");
  O5_PTR(value, "value");
  GemmPlan plan;
  UnitWs uw;
  size_t unit_off;
  const int unit_nk = unit ? hm.off[unit->head + 1] - hm.off[unit->head] : 0;
  const size_t need = sample_ws_bytes(dt, B, H, hm.A + 1, &plan, unit_nk, unit ? unit->d : 0, &uw, &unit_off);
  O5_CHECK(ws != nullptr && ws_bytes >= need, O5_E_WORKSPACE, "o5_policy_sample: workspace needs %zu bytes, got %zu",
           need, ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "o5_policy_sample: ws is not 16-byte aligned");
  hipStream_t s = as_stream(stream);
  const int A1 = hm.A + 1;
  float* zpart = static_cast<float*>(ws);
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
    char* uws = static_cast<char*>(ws) + unit_off;
    unit_forward(dt, B, H, unit_nk, *unit, h, uws, uw, s);
    zext = reinterpret_cast<const float*>(uws + uw.zext);
  }
  hipLaunchKernelGGL(gumbel_sample_rows, dim3(cdiv(B, 256)), dim3(256), 0, s, B, A1, plan.splits, zpart, bp, avail, hm,
                     zext, unit ? unit->head : -1, seed, counter, act, logp, value);
  ktimer_end(kSiteSample, s);
  return check_launch("o5_policy_sample");
}
