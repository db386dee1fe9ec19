// Status strings, per-thread error messages, fp32 -> bf16 conversion.
#include "common.h"

#include <atomic>
#include <mutex>
#include <utility>
#include <vector>

namespace o5 {

static thread_local char g_last_error[512] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
}

void clear_error() { g_last_error[0] = '\0'; }

int check_launch(const char* where) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("%s: kernel launch failed: %s", where, hipGetErrorString(e));
    return O5_E_HIP;
  }
  return O5_OK;
}

// ----------------------------------------------------------- kernel timer
// Events are recorded on the caller's stream around each timed launch site;
// elapsed times are read (and the events returned to the pool) by
// o5_ktimer_read.  Process-wide host state, outside the stateless contract
// of the compute calls: `active` (the recorded sites, 0 = off) is read
// atomically at every launch site, and everything else is touched under
// `lock`, so concurrent callers never race on it; a begin/end pair of one
// site is only meaningful when that site is not timed from two streams at
// once.
namespace {
struct KTimer {
  std::atomic<unsigned> active{0};
  std::mutex lock;
  std::vector<hipEvent_t> pool;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> done[kSiteCount];
  hipEvent_t open[kSiteCount] = {};
  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
KTimer g_kt;
const char* kSiteNames[kSiteCount] = {"lstm_fwd_gemm", "lstm_fwd_cell", "lstm_dh_gemm", "lstm_bwd_cell",
                                      "lstm_dw_gemm",  "lstm_dx_gemm",  "ppo_loss_grad", "adam_step",
                                      "gae",           "policy_sample", "reward_process",
                                      "obs_normalize", "prelstm_fwd",   "prelstm_bwd",   "lstm_fwd_call"};
}  // namespace

void ktimer_begin(int site, hipStream_t s) {
  if (!((g_kt.active.load(std::memory_order_acquire) >> site) & 1u)) return;
  std::lock_guard<std::mutex> g(g_kt.lock);
  hipEvent_t e = g_kt.get();
  if (e && hipEventRecord(e, s) == hipSuccess) g_kt.open[site] = e;
}

void ktimer_end(int site, hipStream_t s) {
  if (!((g_kt.active.load(std::memory_order_acquire) >> site) & 1u)) return;
  std::lock_guard<std::mutex> g(g_kt.lock);
  if (!g_kt.open[site]) return;
  hipEvent_t e = g_kt.get();
  if (e && hipEventRecord(e, s) == hipSuccess) g_kt.done[site].emplace_back(g_kt.open[site], e);
  g_kt.open[site] = nullptr;
}

// 8 elements per thread: two float4 loads, one 16-byte store.
__global__ void __launch_bounds__(256) f32_to_bf16_kernel(size_t n, const float* __restrict__ src,
                                                          uint16_t* __restrict__ dst) {
  const size_t n8 = n / 8;
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n8; i += stride) {
    const float4 a = reinterpret_cast<const float4*>(src)[2 * i];
    const float4 b = reinterpret_cast<const float4*>(src)[2 * i + 1];
    uint4 o;
    o.x = f32x2_to_bf16x2(a.x, a.y);
    o.y = f32x2_to_bf16x2(a.z, a.w);
    o.z = f32x2_to_bf16x2(b.x, b.y);
    o.w = f32x2_to_bf16x2(b.z, b.w);
    reinterpret_cast<uint4*>(dst)[i] = o;
  }
  // tail (fewer than 8 elements), handled by the first block
  if (blockIdx.x == 0) {
    const size_t t = n8 * 8 + threadIdx.x;
    if (t < n) dst[t] = f32_to_bf16_bits(src[t]);
  }
}

}  // namespace o5

using namespace o5;

extern "C" int o5_version(void) { return O5_VERSION; }

extern "C" const char* o5_status_str(int status) {
  switch (status) {
    case O5_OK: return "O5_OK: success";
    case O5_E_NULL: return "O5_E_NULL: a required pointer is NULL";
    case O5_E_SHAPE: return "O5_E_SHAPE: a size is out of range or inconsistent";
    case O5_E_DTYPE: return "O5_E_DTYPE: unknown dtype";
    case O5_E_ALIGN: return "O5_E_ALIGN: a device pointer is not 16-byte aligned";
    case O5_E_WORKSPACE: return "O5_E_WORKSPACE: workspace missing or too small";
    case O5_E_HIP: return "O5_E_HIP: the HIP runtime refused a launch";
    case O5_E_ARG: return "O5_E_ARG: an argument is out of range";
    default: return "unknown o5 status";
  }
}

extern "C" const char* o5_last_error(void) { return o5::g_last_error; }

extern "C" int o5_ktimer_enable_sites(unsigned mask) {
  if (mask == 0) {  // stop recording; keep what was recorded
    g_kt.active.store(0, std::memory_order_release);
    return O5_OK;
  }
  std::lock_guard<std::mutex> g(g_kt.lock);
  for (int i = 0; i < kSiteCount; ++i) {
    for (auto& pr : g_kt.done[i]) {
      g_kt.pool.push_back(pr.first);
      g_kt.pool.push_back(pr.second);
    }
    g_kt.done[i].clear();
    g_kt.open[i] = nullptr;
  }
  g_kt.active.store(mask & ((1u << kSiteCount) - 1u), std::memory_order_release);
  return O5_OK;
}

extern "C" int o5_ktimer_enable(int on) { return o5_ktimer_enable_sites(on ? ~0u : 0u); }

extern "C" int o5_ktimer_read(int site, double* total_ms, int* launches) {
  O5_CHECK(site >= 0 && site < kSiteCount, O5_E_ARG, "o5_ktimer_read: site %d out of range", site);
  O5_CHECK(total_ms != nullptr && launches != nullptr, O5_E_NULL, "o5_ktimer_read: NULL output");
  std::lock_guard<std::mutex> g(g_kt.lock);
  double t = 0.0;
  for (auto& pr : g_kt.done[site]) {
    float ms = 0.0f;
    if (hipEventSynchronize(pr.second) != hipSuccess || hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess) {
      set_error("o5_ktimer_read: event query failed");
      return O5_E_HIP;
    }
    t += ms;
  }
  *total_ms = t;
  *launches = static_cast<int>(g_kt.done[site].size());
  return O5_OK;
}

extern "C" const char* o5_ktimer_site_name(int site) {
  return (site >= 0 && site < kSiteCount) ? kSiteNames[site] : "";
}

extern "C" int o5_f32_to_bf16(size_t n, const float* src, uint16_t* dst, void* stream) {
  O5_CHECK(n >= 1, O5_E_SHAPE, "o5_f32_to_bf16: n must be >= 1");
  O5_PTR(src, "src");
  O5_PTR(dst, "dst");
  size_t n8 = n / 8;
  size_t blocks = (n8 + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(f32_to_bf16_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     as_stream(stream), n, src, dst);
  return check_launch("o5_f32_to_bf16");
}
