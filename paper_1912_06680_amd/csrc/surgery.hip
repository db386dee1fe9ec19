// Surgery on the flat parameter vector (appendix "Surgery"; subsection
// "Continual Transfer via Surgery"): widen the LSTM from H to H2 units and
// extend its input from D to D2 features, or fold trailing constant inputs
// into the bias, carrying Adam's moments along.
//
// Flat layout (as the optimizer step uses it): Wx [4H, D], Wh [4H, H], b
// [4H], Wp [A1, H], bp [A1], gate blocks (i, f, g, o) along 4H.
//
// widen: one thread per 4 consecutive elements of the new vector.  Each
// element is a copy of its old counterpart (parameter and both moments), a
// zero (LSTM columns reading new inputs, head columns reading new units), or
// new: parameter scale * (2U - 1), one fp32 rounding, with U from Philox4x64-10 (counter
// (e div 4, 0, 0, 0), key (seed, 1), word e mod 4 for element e), moments
// zero.  The thread's 4 words are one Philox block.  Writes are contiguous;
// reads are contiguous runs of the old rows.
//
// fold_input: the last D - Dk inputs of the LSTM are a constant vector E
// (an embedding that no longer depends on the observation): b' = b +
// Wx[:, Dk:] E and Wx' = Wx[:, :Dk]; one wave per row of Wx for the dot
// product (fixed order), a copy kernel for the rest.  The moments of the
// dropped columns are discarded; the bias keeps its moments.
#include "common.h"
#include "philox.h"

namespace o5 {

struct Shape5 {
  int D, H, A1;
  size_t wx, wh, b, wp, bp, total;  // offsets of the five blocks and the size
};

static Shape5 shape5(int D, int H, int A1) {
  Shape5 s{D, H, A1, 0, 0, 0, 0, 0, 0};
  const size_t G = 4 * static_cast<size_t>(H);
  s.wx = 0;
  s.wh = s.wx + G * D;
  s.b = s.wh + G * H;
  s.wp = s.b + G;
  s.bp = s.wp + static_cast<size_t>(A1) * H;
  s.total = s.bp + A1;
  return s;
}

constexpr int64_t kNew = -1;   // element takes a new random value
constexpr int64_t kZero = -2;  // element is zero

// Source of element e of the widened vector in the old one, or kNew / kZero.
// I is the index type: 32-bit divisions where the vectors allow them.
template <typename I>
__device__ __forceinline__ int64_t widen_source(I e, const Shape5& o, const Shape5& n) {
  const I nD = n.D, nH = n.H, oD = o.D, oH = o.H;
  if (e < static_cast<I>(n.wh)) {  // Wx': row (gate g, unit j), column k
    const I r = e / nD, k = e - r * nD;
    const I g = r / nH, j = r - g * nH;
    if (j >= oH) return kNew;
    if (k >= oD) return kZero;
    return static_cast<int64_t>(o.wx + (static_cast<size_t>(g) * oH + j) * oD + k);
  }
  if (e < static_cast<I>(n.b)) {
    const I q = e - static_cast<I>(n.wh);
    const I r = q / nH, k = q - r * nH;
    const I g = r / nH, j = r - g * nH;
    if (j >= oH || k >= oH) return kNew;
    return static_cast<int64_t>(o.wh + (static_cast<size_t>(g) * oH + j) * oH + k);
  }
  if (e < static_cast<I>(n.wp)) {
    const I r = e - static_cast<I>(n.b);
    const I g = r / nH, j = r - g * nH;
    if (j >= oH) return kNew;
    return static_cast<int64_t>(o.b + static_cast<size_t>(g) * oH + j);
  }
  if (e < static_cast<I>(n.bp)) {
    const I q = e - static_cast<I>(n.wp);
    const I a = q / nH, k = q - a * nH;
    if (k >= oH) return kZero;
    return static_cast<int64_t>(o.wp + static_cast<size_t>(a) * oH + k);
  }
  return static_cast<int64_t>(o.bp + (e - static_cast<I>(n.bp)));
}

template <typename I>
__global__ void __launch_bounds__(256) widen_kernel(Shape5 o, Shape5 n, const float* __restrict__ p_old,
                                                    const float* __restrict__ m_old, const float* __restrict__ v_old,
                                                    float* __restrict__ p_new, float* __restrict__ m_new,
                                                    float* __restrict__ v_new, float scale, uint64_t seed) {
  const size_t t = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const size_t e0 = t * 4;
  if (e0 >= n.total) return;
  uint64_t w0 = t, w1 = 0, w2 = 0, w3 = 0;
  philox4x64_10(w0, w1, w2, w3, seed, 1ull);
  const uint64_t words[4] = {w0, w1, w2, w3};
  float p[4] = {0.0f, 0.0f, 0.0f, 0.0f}, m[4] = {0.0f, 0.0f, 0.0f, 0.0f}, v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const size_t e = e0 + q;
    if (e >= n.total) break;
    const int64_t src = widen_source<I>(static_cast<I>(e), o, n);
    if (src >= 0) {
      p[q] = p_old[src];
      m[q] = m_old ? m_old[src] : 0.0f;
      v[q] = v_old ? v_old[src] : 0.0f;
    } else if (src == kNew) {
      // 2U - 1 = (2 (word >> 40) + 1 - 2^24) / 2^24: an odd integer below 2^24
      // in magnitude times a power of two, exact in fp32 (U itself is not:
      // it needs 25 bits), so the product with scale is the only rounding
      const int32_t k = static_cast<int32_t>(words[q] >> 40);
      p[q] = scale * (static_cast<float>(2 * k + 1 - (1 << 24)) * 5.9604644775390625e-08f);
    }
  }
  if (e0 + 4 <= n.total) {  // 16-byte stores (the vectors are 16-byte aligned)
    *reinterpret_cast<float4*>(p_new + e0) = make_float4(p[0], p[1], p[2], p[3]);
    *reinterpret_cast<float4*>(m_new + e0) = make_float4(m[0], m[1], m[2], m[3]);
    *reinterpret_cast<float4*>(v_new + e0) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    for (int q = 0; q < 4 && e0 + q < n.total; ++q) {
      p_new[e0 + q] = p[q];
      m_new[e0 + q] = m[q];
      v_new[e0 + q] = v[q];
    }
  }
}

// Element e of the folded vector (inputs 0..Dk-1) from the old one (inputs
// 0..D-1): same structure with the Wx columns cut.
__device__ __forceinline__ size_t fold_source(size_t e, const Shape5& o, const Shape5& n) {
  if (e < n.wh) {
    const size_t r = e / n.D, k = e % n.D;
    return o.wx + r * o.D + k;
  }
  return o.wh + (e - n.wh);  // Wh, b, Wp, bp keep their order and sizes
}

__global__ void __launch_bounds__(256) fold_copy(Shape5 o, Shape5 n, const float* __restrict__ p_old,
                                                 const float* __restrict__ m_old, const float* __restrict__ v_old,
                                                 float* __restrict__ p_new, float* __restrict__ m_new,
                                                 float* __restrict__ v_new) {
  const size_t e = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= n.total) return;
  const size_t src = fold_source(e, o, n);
  p_new[e] = p_old[src];
  m_new[e] = m_old ? m_old[src] : 0.0f;
  v_new[e] = v_old ? v_old[src] : 0.0f;
}

// b'[r] = b[r] + sum_k Wx[r, Dk + k] E[k], one wave per row, lanes over k in
// order, then a fixed butterfly.
__global__ void __launch_bounds__(256) fold_bias(Shape5 o, Shape5 n, int Dk, const float* __restrict__ p_old,
                                                 const float* __restrict__ E, float* __restrict__ p_new) {
  const int lane = threadIdx.x & 63;
  const size_t r = static_cast<size_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (r >= 4 * static_cast<size_t>(o.H)) return;
  const float* w = p_old + o.wx + r * o.D + Dk;
  float s = 0.0f;
  for (int k = lane; k < o.D - Dk; k += 64) s += w[k] * E[k];
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) s += __shfl_xor(s, d, 64);
  if (lane == 0) p_new[n.b + r] = p_old[o.b + r] + s;
}

static int check_shape(const char* fn, int D, int H, int A1) {
  O5_CHECK(D >= 1 && H >= 1 && A1 >= 1, O5_E_SHAPE, "%s: D=%d H=%d A1=%d must be >= 1", fn, D, H, A1);
  O5_CHECK(D <= (1 << 24) && H <= (1 << 24) && A1 <= (1 << 24), O5_E_SHAPE, "%s: D, H and A1 must be <= 2^24", fn);
  O5_CHECK(static_cast<long long>(4) * H * (static_cast<long long>(D) + H + 1) +
                   static_cast<long long>(A1) * (static_cast<long long>(H) + 1) <
               (1ll << 40),
           O5_E_SHAPE, "%s: parameter vector too large", fn);
  return O5_OK;
}

}  // namespace o5

using namespace o5;

extern "C" size_t o5_param_count(int D, int H, int A1) {
  if (check_shape("o5_param_count", D, H, A1) != O5_OK) return 0;
  return shape5(D, H, A1).total;
}

extern "C" int o5_surgery_widen(int D, int H, int A1, int D2, int H2, const float* p_old, const float* m_old,
                                const float* v_old, float* p_new, float* m_new, float* v_new, float scale,
                                uint64_t seed, void* stream) {
  int st = check_shape("o5_surgery_widen", D, H, A1);
  if (st != O5_OK) return st;
  st = check_shape("o5_surgery_widen", D2, H2, A1);
  if (st != O5_OK) return st;
  O5_CHECK(D2 >= D && H2 >= H, O5_E_SHAPE, "o5_surgery_widen: need D2 >= D and H2 >= H (D=%d D2=%d H=%d H2=%d)", D,
           D2, H, H2);
  O5_CHECK(scale >= 0.0f, O5_E_ARG, "o5_surgery_widen: scale=%g must be >= 0", scale);
  O5_PTR(p_old, "p_old");
  O5_OPT_PTR(m_old, "m_old");
  O5_OPT_PTR(v_old, "v_old");
  O5_PTR(p_new, "p_new");
  O5_PTR(m_new, "m_new");
  O5_PTR(v_new, "v_new");
  const Shape5 o = shape5(D, H, A1), n = shape5(D2, H2, A1);
  const size_t threads = (n.total + 3) / 4;
  const dim3 grid(static_cast<unsigned>((threads + 255) / 256));
  if (n.total < (size_t{1} << 32))
    hipLaunchKernelGGL(widen_kernel<uint32_t>, grid, dim3(256), 0, as_stream(stream), o, n, p_old, m_old, v_old,
                       p_new, m_new, v_new, scale, seed);
  else
    hipLaunchKernelGGL(widen_kernel<uint64_t>, grid, dim3(256), 0, as_stream(stream), o, n, p_old, m_old, v_old,
                       p_new, m_new, v_new, scale, seed);
  return check_launch("o5_surgery_widen");
}

extern "C" int o5_surgery_fold_input(int D, int H, int A1, int Dk, const float* E, const float* p_old,
                                     const float* m_old, const float* v_old, float* p_new, float* m_new,
                                     float* v_new, void* stream) {
  int st = check_shape("o5_surgery_fold_input", D, H, A1);
  if (st != O5_OK) return st;
  O5_CHECK(Dk >= 1 && Dk < D, O5_E_SHAPE, "o5_surgery_fold_input: need 1 <= Dk < D (Dk=%d D=%d)", Dk, D);
  O5_PTR(E, "E");
  O5_PTR(p_old, "p_old");
  O5_OPT_PTR(m_old, "m_old");
  O5_OPT_PTR(v_old, "v_old");
  O5_PTR(p_new, "p_new");
  O5_PTR(m_new, "m_new");
  O5_PTR(v_new, "v_new");
  const Shape5 o = shape5(D, H, A1), n = shape5(Dk, H, A1);
  hipStream_t s = as_stream(stream);
  hipLaunchKernelGGL(fold_copy, dim3(static_cast<unsigned>((n.total + 255) / 256)), dim3(256), 0, s, o, n, p_old,
                     m_old, v_old, p_new, m_new, v_new);
  hipLaunchKernelGGL(fold_bias, dim3(static_cast<unsigned>(H)), dim3(256), 0, s, o, n, Dk, p_old, E, p_new);
  return check_launch("o5_surgery_fold_input");
}
