// o5_policy_sample_static: the rollout sampler for callers that cannot
// allocate (code under HIP graph capture, tight serving loops, harnesses
// that forbid allocation).  Same kernels as o5_policy_sample; its scratch
// (the logits GEMM's partial sums and the unit-selection head's query and
// logits) lives in a file-scope device array instead of a caller workspace.
#include <mutex>

#include "heads.h"

namespace o5 {

namespace {

// The static scratch: one copy per GPU, held until the process ends.  In
// host code `scratch` only names the symbol; its device address on the
// current GPU comes from hipGetSymbolAddress (scratch_on_device below) and
// is the only form ever passed to a kernel or a copy.
__device__ __align__(256) char scratch[O5_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_lock;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch array's address on the current device, looked up on the first
// call on that device (with the device current) and kept.
int scratch_on_device(const char* fn, char** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  O5_CHECK(e == hipSuccess && dev >= 0 && dev < kMaxDevices, O5_E_HIP, "%s: no current device (%s)", fn,
           hipGetErrorString(e));
  std::lock_guard<std::mutex> g(g_scratch_lock);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    O5_CHECK(e == hipSuccess && p != nullptr, O5_E_HIP, "%s: hipGetSymbolAddress(scratch) on device %d failed: %s", fn,
             dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = static_cast<char*>(g_scratch_ptr[dev]);
  return O5_OK;
}

}  // namespace

}  // namespace o5

using namespace o5;

extern "C" int o5_policy_sample_static(o5_dtype dt, int B, int H, int K, const int* head_sizes, const void* h,
                                       const void* Wp, const float* bp, const uint8_t* avail,
                                       const o5_unit_head* unit, uint64_t seed, uint64_t counter, int32_t* act,
                                       float* logp, float* value, void* stream) {
  static const char* fn = "o5_policy_sample_static";
  HeadsMeta hm;
  size_t need = 0;
  int st = policy_sample_check(fn, dt, B, H, K, head_sizes, h, Wp, bp, avail, unit, act, logp, value, &hm, &need);
  if (st != O5_OK) return st;
  O5_CHECK(need <= static_cast<size_t>(O5_STATIC_SCRATCH_BYTES), O5_E_SHAPE,
           "%s: this shape needs %zu bytes of scratch, the static buffer holds %d (B=%d, %d logits, H=%d)", fn, need,
           O5_STATIC_SCRATCH_BYTES, B, hm.A + 1, H);
  char* ws = nullptr;
  st = scratch_on_device(fn, &ws);
  if (st != O5_OK) return st;
  return policy_sample_run(dt, B, H, hm, h, Wp, bp, avail, unit, seed, counter, act, logp, value, ws,
                           as_stream(stream));
}
