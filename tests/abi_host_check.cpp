// Host-side checks of the C ABI, built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code of every source file (device
// code is not built: nothing here reaches a launch).  Every call below fails
// validation, or is a size query, so no GPU is needed.  Exit status 0 and the
// last line "abi_host_check: all N checks passed" mean that every check held
// and the sanitizers reported nothing (they abort the process on a report).
#include <climits>
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "o5.h"

static int g_checks = 0, g_fail = 0;

#define EXPECT(cond)                                                          \
  do {                                                                        \
    ++g_checks;                                                               \
    if (!(cond)) {                                                            \
      ++g_fail;                                                               \
      std::fprintf(stderr, "FAILED %s:%d: %s (last error: %s)\n", __FILE__,    \
                   __LINE__, #cond, o5_last_error());                         \
    }                                                                         \
  } while (0)

// A fake, 16-byte aligned device address: never dereferenced, since every
// call that receives it is rejected before any launch.
static void* P(uintptr_t a = 16) { return reinterpret_cast<void*>(a); }
static float* F(uintptr_t a = 16) { return static_cast<float*>(P(a)); }
static uint8_t* U8(uintptr_t a = 16) { return static_cast<uint8_t*>(P(a)); }

static void check_strings() {
  EXPECT(o5_version() == 100);
  for (int c = -3; c < 12; ++c) EXPECT(o5_status_str(c) != nullptr && std::strlen(o5_status_str(c)) > 0);
  EXPECT(std::strncmp(o5_status_str(0), "O5_OK", 5) == 0);
  EXPECT(o5_last_error() != nullptr);
  for (int s = -2; s < 40; ++s) EXPECT(o5_ktimer_site_name(s) != nullptr);
  double ms = 0.0;
  int n = 0;
  EXPECT(o5_ktimer_read(-1, &ms, &n) != O5_OK);
  EXPECT(o5_ktimer_read(1 << 20, &ms, &n) != O5_OK);
  EXPECT(o5_ktimer_enable(0) == O5_OK);
}

static void check_gae() {
  EXPECT(o5_gae(16, 8, nullptr, nullptr, nullptr, 0.99f, 0.95f, nullptr, nullptr, nullptr) == O5_E_NULL);
  EXPECT(o5_gae(0, 8, F(), F(), U8(), 0.99f, 0.95f, F(), F(), nullptr) == O5_E_SHAPE);
  EXPECT(o5_gae(-5, 8, F(), F(), U8(), 0.99f, 0.95f, F(), F(), nullptr) == O5_E_SHAPE);
  EXPECT(o5_gae(INT_MAX, INT_MAX, F(), F(), U8(), 0.99f, 0.95f, F(), F(), nullptr) == O5_E_SHAPE);
  EXPECT(o5_gae(16, 8, F(0x1001), F(), U8(), 0.99f, 0.95f, F(), F(), nullptr) == O5_E_ALIGN);
  EXPECT(o5_gae(16, 8, F(), F(), U8(), 1.5f, 0.95f, F(), F(), nullptr) == O5_E_ARG);
  EXPECT(o5_gae(16, 8, F(), F(), U8(), 0.99f, -0.1f, F(), F(), nullptr) == O5_E_ARG);
  EXPECT(o5_segments_to_samples(10, 2, 3, F(), F(), U8(), F(), F(), U8(), nullptr) == O5_E_SHAPE);
  EXPECT(o5_segments_to_samples(INT_MAX, INT_MAX, 16, F(), F(), U8(), F(), F(), U8(), nullptr) == O5_E_SHAPE);
  EXPECT(o5_segments_to_samples(16, 8, 16, nullptr, F(), U8(), F(), F(), U8(), nullptr) == O5_E_NULL);
}

static void check_lstm() {
  for (int dt = 0; dt < 2; ++dt) {
    const o5_dtype d = static_cast<o5_dtype>(dt);
    const size_t need = o5_lstm_fwd_workspace_bytes(d, 16, 8, 64, 128);
    EXPECT(need > 0);
    EXPECT(o5_lstm_fwd(d, 16, 8, 64, 128, P(), P(), P(), F(), F(), F(), U8(), P(), F(), P(), P(), need - 1,
                       nullptr) == O5_E_WORKSPACE);
    EXPECT(o5_lstm_fwd(d, 16, 8, 64, 128, P(), P(), P(), F(), F(), F(), U8(), P(), F(), P(), nullptr, need,
                       nullptr) == O5_E_WORKSPACE);
    EXPECT(o5_lstm_fwd(d, 1, 1, 60, 64, P(), P(), P(), F(), F(), F(), U8(), P(), F(), P(), P(), 1 << 20,
                       nullptr) == O5_E_SHAPE);
    EXPECT(o5_lstm_fwd(d, 16, 8, 64, 128, nullptr, P(), P(), F(), F(), F(), U8(), P(), F(), P(), P(), need,
                       nullptr) == O5_E_NULL);
    EXPECT(o5_lstm_fwd(d, 16, 8, 64, 128, P(0x1002), P(), P(), F(), F(), F(), U8(), P(), F(), P(), P(), need,
                       nullptr) == O5_E_ALIGN);
    const size_t bneed = o5_lstm_bptt_workspace_bytes(d, 16, 8, 64, 128);
    EXPECT(bneed > 0);
    EXPECT(o5_lstm_bptt(d, 16, 8, 64, 128, P(), P(), P(), F(), F(), U8(), P(), F(), nullptr, F(), F(), F(), F(), F(),
                        F(), nullptr, P(), bneed, nullptr) == O5_E_NULL);
    EXPECT(o5_lstm_bptt(d, 16, 8, 64, 128, P(), P(), P(), F(), F(), U8(), P(), F(), P(), F(), F(), F(), F(), F(), F(),
                        nullptr, P(), bneed - 1, nullptr) == O5_E_WORKSPACE);
    // extreme sizes: the queries reject them (0) without overflowing
    const int big[] = {0, -1, 1, 63, 64, 65536, 1 << 20, INT_MAX};
    for (int T : {1, 16, INT_MAX})
      for (int B : big)
        for (int H : big) {
          (void)o5_lstm_fwd_workspace_bytes(d, T, B, H, H);
          (void)o5_lstm_bptt_workspace_bytes(d, T, B, H, H);
          (void)o5_prelstm_bwd_workspace_bytes(d, T, B, H, H);
          ++g_checks;
        }
  }
  EXPECT(o5_lstm_fwd(static_cast<o5_dtype>(9), 1, 1, 64, 64, P(), P(), P(), F(), F(), F(), U8(), P(), F(), P(), P(),
                     1 << 20, nullptr) == O5_E_DTYPE);
  EXPECT(o5_lstm_fwd_workspace_bytes(static_cast<o5_dtype>(9), 16, 8, 64, 128) == 0);
}

static void check_heads_and_sampler() {
  const int heads[4] = {30, 8, 32, 4};
  const int bad[2] = {3, 0};
  const o5_ppo_hp hp{0.2f, 1.0f, 0.01f};
  for (int dt = 0; dt < 2; ++dt) {
    const o5_dtype d = static_cast<o5_dtype>(dt);
    EXPECT(o5_ppo_loss_grad_workspace_bytes(d, 8, 64, 2, bad, nullptr) == 0);
    EXPECT(std::strstr(o5_last_error(), "head_sizes[1]") != nullptr);
    EXPECT(o5_ppo_loss_grad_workspace_bytes(d, 8, 64, 4, nullptr, nullptr) == 0);
    EXPECT(o5_ppo_loss_grad_workspace_bytes(d, 8, 64, 0, heads, nullptr) == 0);
    EXPECT(o5_ppo_loss_grad_workspace_bytes(d, 8, 64, 99, heads, nullptr) == 0);
    const size_t need = o5_ppo_loss_grad_workspace_bytes(d, 2048, 4096, 4, heads, nullptr);
    EXPECT(need > 0);
    EXPECT(o5_ppo_loss_grad(d, 2048, 4096, 4, heads, P(), P(), F(), static_cast<int32_t*>(P()), F(), F(), F(), U8(),
                            nullptr, nullptr, hp, F(), F(), F(), F(), P(), need - 1, nullptr) == O5_E_WORKSPACE);
    EXPECT(o5_ppo_loss_grad(d, 2048, 4096, 4, heads, P(), P(), F(), static_cast<int32_t*>(P()), F(), F(), F(), U8(),
                            nullptr, nullptr, o5_ppo_hp{1.0f, 1.0f, 0.01f}, F(), F(), F(), F(), P(), need,
                            nullptr) == O5_E_ARG);
    EXPECT(o5_ppo_loss_grad(d, 2048, 4096, 4, heads, nullptr, P(), F(), static_cast<int32_t*>(P()), F(), F(), F(),
                            U8(), nullptr, nullptr, hp, F(), F(), F(), F(), P(), need, nullptr) == O5_E_NULL);
    // a unit head with d not a power of two, or pointing at a missing head
    o5_unit_head u{1, 100, P(), F(), P(), F(), F()};
    EXPECT(o5_ppo_loss_grad_workspace_bytes(d, 64, 64, 4, heads, &u) == 0);
    u.d = 128;
    u.head = 7;
    EXPECT(o5_ppo_loss_grad_workspace_bytes(d, 64, 64, 4, heads, &u) == 0);
    u.head = 1;
    EXPECT(o5_ppo_loss_grad_workspace_bytes(d, 32768, 4096, 4, heads, &u) > need);
    const size_t sneed = o5_policy_sample_workspace_bytes(d, 4096, 4096, 4, heads, nullptr);
    EXPECT(sneed > 0);
    EXPECT(o5_policy_sample(d, 4096, 4096, 4, heads, P(), P(), F(), U8(), nullptr, 1, 0, static_cast<int32_t*>(P()),
                            F(), F(), P(), sneed - 1, nullptr) == O5_E_WORKSPACE);
    EXPECT(o5_policy_sample(d, 4096, 4096, 4, heads, nullptr, P(), F(), U8(), nullptr, 1, 0,
                            static_cast<int32_t*>(P()), F(), F(), P(), sneed, nullptr) == O5_E_NULL);
    // the static-scratch sampler rejects before it touches a device
    EXPECT(o5_policy_sample_static(d, 1 << 20, 4096, 4, heads, P(), P(), F(), U8(), nullptr, 1, 0,
                                   static_cast<int32_t*>(P()), F(), F(), nullptr) == O5_E_SHAPE);
    EXPECT(o5_policy_sample_static(d, 64, 4096, 4, heads, nullptr, P(), F(), U8(), nullptr, 1, 0,
                                   static_cast<int32_t*>(P()), F(), F(), nullptr) == O5_E_NULL);
    const int big[] = {0, -1, 1, 64, 65536, 1 << 24, INT_MAX};
    for (int N : big)
      for (int H : big) {
        (void)o5_ppo_loss_grad_workspace_bytes(d, N, H, 4, heads, nullptr);
        (void)o5_ppo_loss_grad_workspace_bytes(d, N, H, 4, heads, &u);
        (void)o5_policy_sample_workspace_bytes(d, N, H, 4, heads, nullptr);
        (void)o5_policy_sample_workspace_bytes(d, N, H, 4, heads, &u);
        ++g_checks;
      }
  }
  // the factored loss and backward calls: bf16 only, ld as the heads need
  {
    const o5_ppo_hp hp{0.2f, 1.0f, 0.01f};
    const int ld = o5_ppo_head_grad_ld(4096, 4, heads, nullptr);
    EXPECT(ld == 256);
    o5_unit_head u{1, 128, P(), F(), P(), F(), F()};
    EXPECT(o5_ppo_head_grad_ld(4096, 4, heads, &u) == 512);
    EXPECT(o5_ppo_head_grad_ld(4096, 4, nullptr, nullptr) == 0);
    EXPECT(o5_ppo_head_grad_ld(-1, 4, heads, nullptr) == 0);
    const size_t need = o5_ppo_loss_grad_workspace_bytes(O5_BF16, 2048, 4096, 4, heads, nullptr);
    uint16_t* p16 = static_cast<uint16_t*>(P());
    EXPECT(o5_ppo_loss_grad_factored(O5_F32, 2048, 4096, 4, heads, P(), P(), F(), static_cast<int32_t*>(P()), F(),
                                     F(), F(), U8(), nullptr, nullptr, hp, F(), p16, p16, ld, F(), F(), P(), need,
                                     nullptr) == O5_E_DTYPE);
    EXPECT(o5_ppo_loss_grad_factored(O5_BF16, 2048, 4096, 4, heads, P(), P(), F(), static_cast<int32_t*>(P()), F(),
                                     F(), F(), U8(), nullptr, nullptr, hp, F(), p16, p16, ld + 64, F(), F(), P(), need,
                                     nullptr) == O5_E_SHAPE);
    EXPECT(o5_ppo_loss_grad_factored(O5_BF16, 2048, 4096, 4, heads, P(), P(), F(), static_cast<int32_t*>(P()), F(),
                                     F(), F(), U8(), nullptr, nullptr, hp, F(), nullptr, p16, ld, F(), F(), P(), need,
                                     nullptr) == O5_E_NULL);
    const size_t bneed = o5_lstm_bptt_workspace_bytes(O5_BF16, 16, 8, 64, 128);
    EXPECT(o5_lstm_bptt_factored(O5_F32, 16, 8, 64, 128, P(), P(), P(), F(), F(), U8(), P(), F(), P(), p16, p16, 256,
                                 nullptr, nullptr, F(), F(), F(), nullptr, P(), bneed, nullptr) == O5_E_DTYPE);
    EXPECT(o5_lstm_bptt_factored(O5_BF16, 16, 8, 64, 128, P(), P(), P(), F(), F(), U8(), P(), F(), P(), p16, p16, 100,
                                 nullptr, nullptr, F(), F(), F(), nullptr, P(), bneed, nullptr) == O5_E_SHAPE);
    EXPECT(o5_lstm_bptt_factored(O5_BF16, 16, 8, 64, 128, P(), P(), P(), F(), F(), U8(), P(), F(), P(), p16, p16, 256,
                                 nullptr, nullptr, F(), F(), F(), nullptr, P(), bneed - 1, nullptr) == O5_E_WORKSPACE);
    EXPECT(o5_lstm_bptt_factored(O5_BF16, 16, 8, 64, 128, P(), P(), P(), F(), F(), U8(), P(), F(), P(), nullptr, p16,
                                 256, nullptr, nullptr, F(), F(), F(), nullptr, P(), bneed, nullptr) == O5_E_NULL);
  }
  // many large heads: the total is capped
  int wide[8];
  for (int& w : wide) w = INT_MAX / 4;
  EXPECT(o5_ppo_loss_grad_workspace_bytes(O5_BF16, 64, 64, 8, wide, nullptr) == 0);
}

static void check_adam_surgery_misc() {
  const o5_adam_hp hp{1e-3f, 0.9f, 0.999f, 1e-8f, 5.0f};
  EXPECT(o5_adam_step(10, F(), F(), F(), F(), nullptr, hp, 0, nullptr) == O5_E_ARG);
  EXPECT(o5_adam_step(10, nullptr, F(), F(), F(), nullptr, hp, 1, nullptr) == O5_E_NULL);
  EXPECT(o5_adam_step(10, F(0x1004), F(), F(), F(), nullptr, hp, 1, nullptr) == O5_E_ALIGN);
  EXPECT(o5_adam_step(10, F(), F(), F(), F(), nullptr, o5_adam_hp{1e-3f, 1.0f, 0.999f, 1e-8f, 5.0f}, 1, nullptr) ==
         O5_E_ARG);
  EXPECT(o5_f32_to_bf16(10, nullptr, static_cast<uint16_t*>(P()), nullptr) == O5_E_NULL);
  EXPECT(o5_param_count(4096, 4096, 75) == 134541387u);
  (void)o5_param_count(INT_MAX, INT_MAX, INT_MAX);
  (void)o5_param_count(-1, -1, -1);
  EXPECT(o5_surgery_widen(64, 64, 9, 32, 64, F(), nullptr, nullptr, F(), F(), F(), 0.01f, 1, nullptr) ==
         O5_E_SHAPE);
  EXPECT(o5_surgery_widen(64, 64, 9, 64, 128, F(), nullptr, nullptr, F(), F(), F(), -1.0f, 1, nullptr) == O5_E_ARG);
  EXPECT(o5_surgery_widen(64, 64, 9, 64, 128, nullptr, nullptr, nullptr, F(), F(), F(), 0.01f, 1, nullptr) ==
         O5_E_NULL);
  EXPECT(o5_surgery_widen(INT_MAX, INT_MAX, INT_MAX, INT_MAX, INT_MAX, F(), nullptr, nullptr, F(), F(), F(), 0.01f, 1,
                          nullptr) != O5_OK);
  EXPECT(o5_surgery_fold_input(64, 64, 9, 64, F(), F(), nullptr, nullptr, F(), F(), F(), nullptr) == O5_E_SHAPE);
  const o5_reward_hp rhp{0.3f, 0.6f, 10.0f, 1e-8f};
  EXPECT(o5_reward_process(0, 4, F(), nullptr, F(), rhp, static_cast<double*>(P()), F(), P(), 1 << 20, nullptr) ==
         O5_E_SHAPE);
  EXPECT(o5_reward_process(4, 4, F(), nullptr, nullptr, rhp, static_cast<double*>(P()), F(), P(), 1 << 20,
                           nullptr) == O5_E_NULL);
  EXPECT(o5_reward_process(4, 4, F(), nullptr, F(), o5_reward_hp{1.5f, 0.6f, 10.0f, 1e-8f}, static_cast<double*>(P()),
                           F(), P(), 1 << 20, nullptr) == O5_E_ARG);
  const size_t rneed = o5_reward_process_workspace_bytes(4, 4);
  EXPECT(rneed > 0);
  EXPECT(o5_reward_process(4, 4, F(), nullptr, F(), rhp, static_cast<double*>(P()), F(), P(), rneed - 1, nullptr) ==
         O5_E_WORKSPACE);
  EXPECT(o5_reward_process_workspace_bytes(0, 1) == 0);
  (void)o5_reward_process_workspace_bytes(INT_MAX, INT_MAX);
  EXPECT(o5_obs_normalize(O5_BF16, 0, 64, F(), static_cast<double*>(P()), 5.0f, 1e-8f, P(), P(), 1 << 20, nullptr) ==
         O5_E_SHAPE);
  EXPECT(o5_obs_normalize(O5_BF16, 10, 64, F(), static_cast<double*>(P()), 0.0f, 1e-8f, P(), P(), 1 << 20, nullptr) ==
         O5_E_ARG);
  (void)o5_obs_normalize_workspace_bytes(INT_MAX, INT_MAX);
  EXPECT(o5_prelstm_fwd(O5_BF16, 2, 7, 64, 64, P(), P(), F(), F(), P(), nullptr) == O5_E_SHAPE);
  EXPECT(o5_prelstm_fwd(O5_BF16, 2, 10, 64, 96, P(), P(), F(), F(), P(), nullptr) == O5_E_SHAPE);
  EXPECT(o5_prelstm_fwd(static_cast<o5_dtype>(5), 2, 10, 64, 64, P(), P(), F(), F(), P(), nullptr) == O5_E_DTYPE);
  EXPECT(o5_prelstm_bwd(O5_BF16, 2, 10, 64, 64, P(), F(), P(), F(), F(), nullptr, 0, nullptr) == O5_E_WORKSPACE);
}

int main() {
  check_strings();
  check_gae();
  check_lstm();
  check_heads_and_sampler();
  check_adam_surgery_misc();
  if (g_fail) {
    std::printf("abi_host_check: %d of %d checks failed\n", g_fail, g_checks);
    return 1;
  }
  std::printf("abi_host_check: all %d checks passed\n", g_checks);
  return 0;
}
