// Shared host/device helpers of libo5: error reporting, argument checks,
// bf16 conversion, launch helpers.  gfx950 (CDNA4) only.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstddef>
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "../../include/o5.h"

namespace o5 {

// ---------------------------------------------------------------- errors
void set_error(const char* fmt, ...);
void clear_error();

#define O5_CHECK(cond, code, ...)          \
  do {                                     \
    if (!(cond)) {                         \
      ::o5::set_error(__VA_ARGS__);        \
      return (code);                       \
    }                                      \
  } while (0)

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Pointer checks; the _IN forms name the entry point fn in the message (for
// validation helpers shared by several entry points).
#define O5_PTR_IN(fn, p, name)                                                 \
  do {                                                                         \
    O5_CHECK((p) != nullptr, O5_E_NULL, "%s: argument '%s' is NULL", fn, name); \
    O5_CHECK(::o5::aligned16(p), O5_E_ALIGN, "%s: '%s' is not 16-byte aligned", fn, name); \
  } while (0)

#define O5_OPT_PTR_IN(fn, p, name)                                             \
  do {                                                                         \
    if ((p) != nullptr)                                                        \
      O5_CHECK(::o5::aligned16(p), O5_E_ALIGN, "%s: '%s' is not 16-byte aligned", fn, name); \
  } while (0)

#define O5_PTR(p, name) O5_PTR_IN(__func__, p, name)
#define O5_OPT_PTR(p, name) O5_OPT_PTR_IN(__func__, p, name)

// Returns O5_OK, or O5_E_HIP with a message if the last launch failed.
int check_launch(const char* where);

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// ------------------------------------------------------- kernel timing
// Launch sites whose device time o5_ktimer_* can report (see o5.h).
enum KSite {
  kSiteLstmFwdGemm = 0,
  kSiteLstmFwdCell,
  kSiteLstmDhGemm,
  kSiteLstmBwdCell,
  kSiteLstmDwGemm,
  kSiteLstmDxGemm,
  kSitePpo,
  kSiteAdam,
  kSiteGae,
  kSiteSample,
  kSiteReward,
  kSiteObsNorm,
  kSitePreFwd,
  kSitePreBwd,
  kSiteLstmFwdCall,  // the whole o5_lstm_fwd call (all T steps)
  kSiteCount
};
// When timing is on, record an event on `s` before / after a launch site.
void ktimer_begin(int site, hipStream_t s);
void ktimer_end(int site, hipStream_t s);

inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

// ------------------------------------------------------------------ bf16
// Round-to-nearest-even fp32 -> bf16 bits; NaN keeps a quiet NaN.
// f32 -> bf16 bits, rounding to nearest even: for every non-NaN pattern u the
// bits of (u + 0x7fff + ((u >> 16) & 1)) >> 16, and for NaN (u >> 16) | 0x40
// (sign and top payload kept, quiet).  gfx950 has this conversion as one
// instruction (v_cvt_pk_bf16_f32, two values at a time); the conversion
// tests check it against that formula on all 2^32 inputs.
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// Two at once: a in the low 16 bits, b in the high.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float a, float b) {
  typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
  const bf16x2_v v = {static_cast<__bf16>(a), static_cast<__bf16>(b)};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// ------------------------------------------------------------- activations
// sigma(a) = 1 / (1 + e^-a) and tanh(a) = 1 - 2 / (1 + e^2a) with the
// hardware exp2 and reciprocal (about 1 ulp each); both saturate correctly
// when the exponential overflows or underflows.
__device__ __forceinline__ float sigmoid_f(float a) { return __builtin_amdgcn_rcpf(1.0f + __expf(-a)); }
__device__ __forceinline__ float tanh_f(float a) { return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + __expf(2.0f * a)); }

// Element type tags used by templates: float (fp32 path) or uint16_t
// holding bf16 bits (bf16 path).
template <typename E> struct elem;
template <> struct elem<float> {
  __device__ __forceinline__ static float to_f32(float v) { return v; }
  __device__ __forceinline__ static float from_f32(float v) { return v; }
};
template <> struct elem<uint16_t> {
  __device__ __forceinline__ static float to_f32(uint16_t v) { return bf16_bits_to_f32(v); }
  __device__ __forceinline__ static uint16_t from_f32(float v) { return f32_to_bf16_bits(v); }
};

inline size_t dtype_size(o5_dtype dt) { return dt == O5_BF16 ? 2 : 4; }

}  // namespace o5
