// Adam with the per-parameter gradient clip to +-clip_k sqrt(v_hat)
// (subsection "Optimizing the Policy"; Table "Hyperparameters").
//
// One pass over the flat fp32 parameter vector: read p, m, v, g (16 B),
// write p, m, v (12 B) and optionally the bf16 copy of p (2 B) that the bf16
// GEMMs read -- 30 B per parameter, an HBM-bound stream.  Each thread
// handles 4 consecutive parameters with 16-byte loads and stores; the grid
// strides over the vector.
#include "common.h"

namespace o5 {

struct AdamConsts {
  float lr, b1, b2, one_m_b1, one_m_b2, inv_bc1, inv_bc2, eps, clip_k;
};

__device__ __forceinline__ void adam_one(const AdamConsts& c, float& p, float& m, float& v, float g) {
  v = c.b2 * v + c.one_m_b2 * (g * g);
  const float sq = sqrtf(v * c.inv_bc2);
  float gc = g;
  if (c.clip_k > 0.0f) {
    const float bound = c.clip_k * sq;
    gc = fminf(fmaxf(g, -bound), bound);
  }
  m = c.b1 * m + c.one_m_b1 * gc;
  p = p - c.lr * (m * c.inv_bc1) / (sq + c.eps);
}

template <bool kBf16Out>
__global__ void __launch_bounds__(256) adam_kernel(size_t n, float* __restrict__ p, float* __restrict__ m,
                                                   float* __restrict__ v, const float* __restrict__ g,
                                                   uint16_t* __restrict__ pb, AdamConsts c) {
  const size_t n4 = n / 4;
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n4; i += stride) {
    float4 pp = reinterpret_cast<float4*>(p)[i];
    float4 mm = reinterpret_cast<float4*>(m)[i];
    float4 vv = reinterpret_cast<float4*>(v)[i];
    const float4 gg = reinterpret_cast<const float4*>(g)[i];
    adam_one(c, pp.x, mm.x, vv.x, gg.x);
    adam_one(c, pp.y, mm.y, vv.y, gg.y);
    adam_one(c, pp.z, mm.z, vv.z, gg.z);
    adam_one(c, pp.w, mm.w, vv.w, gg.w);
    reinterpret_cast<float4*>(p)[i] = pp;
    reinterpret_cast<float4*>(m)[i] = mm;
    reinterpret_cast<float4*>(v)[i] = vv;
    if (kBf16Out) {
      uint2 o;
      o.x = f32_to_bf16_bits(pp.x) | (static_cast<uint32_t>(f32_to_bf16_bits(pp.y)) << 16);
      o.y = f32_to_bf16_bits(pp.z) | (static_cast<uint32_t>(f32_to_bf16_bits(pp.w)) << 16);
      reinterpret_cast<uint2*>(pb)[i] = o;
    }
  }
  if (blockIdx.x == 0) {
    const size_t t = n4 * 4 + threadIdx.x;
    if (t < n) {
      float pp = p[t], mm = m[t], vv = v[t];
      adam_one(c, pp, mm, vv, g[t]);
      p[t] = pp;
      m[t] = mm;
      v[t] = vv;
      if (kBf16Out) pb[t] = f32_to_bf16_bits(pp);
    }
  }
}

}  // namespace o5

using namespace o5;

extern "C" int o5_adam_step(size_t n, float* p, float* m, float* v, const float* g, uint16_t* p_bf16,
                            o5_adam_hp hp, int step, void* stream) {
  O5_CHECK(n >= 1, O5_E_SHAPE, "o5_adam_step: n must be >= 1");
  O5_CHECK(step >= 1, O5_E_ARG, "o5_adam_step: step=%d must be >= 1", step);
  O5_CHECK(hp.beta1 >= 0.0f && hp.beta1 < 1.0f && hp.beta2 >= 0.0f && hp.beta2 < 1.0f, O5_E_ARG,
           "o5_adam_step: betas must lie in [0, 1)");
  O5_CHECK(hp.eps > 0.0f && hp.lr >= 0.0f, O5_E_ARG, "o5_adam_step: need eps > 0 and lr >= 0");
  O5_PTR(p, "p");
  O5_PTR(m, "m");
  O5_PTR(v, "v");
  O5_PTR(g, "g");
  O5_OPT_PTR(p_bf16, "p_bf16");
  AdamConsts c;
  c.lr = hp.lr;
  c.b1 = hp.beta1;
  c.b2 = hp.beta2;
  c.one_m_b1 = 1.0f - hp.beta1;
  c.one_m_b2 = 1.0f - hp.beta2;
  // bias corrections in double on the host, then rounded once
  c.inv_bc1 = static_cast<float>(1.0 / (1.0 - std::pow(static_cast<double>(hp.beta1), step)));
  c.inv_bc2 = static_cast<float>(1.0 / (1.0 - std::pow(static_cast<double>(hp.beta2), step)));
  c.eps = hp.eps;
  c.clip_k = hp.clip_k;
  size_t blocks = (n / 4 + 255) / 256;
  const size_t cap = 256 * 16;  // 16 blocks per CU of MI355X: enough waves in flight to saturate HBM
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  ktimer_begin(kSiteAdam, as_stream(stream));
  if (p_bf16)
    hipLaunchKernelGGL(adam_kernel<true>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, as_stream(stream), n,
                       p, m, v, g, p_bf16, c);
  else
    hipLaunchKernelGGL(adam_kernel<false>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, as_stream(stream), n,
                       p, m, v, g, p_bf16, c);
  ktimer_end(kSiteAdam, as_stream(stream));
  return check_launch("o5_adam_step");
}
