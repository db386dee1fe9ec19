// Generalized advantage estimation over rollout segments, and the cut of
// segments into 16-step samples (subsection "Optimizing the Policy"; Figure
// "Timescales and Staleness").
//
// GAE is the reverse linear recurrence  A_t = delta_t + c_t A_{t+1}  with
// c_t = gamma lambda (1 - done_t) and A_L = 0.  A stretch of steps reduces
// to an affine map A_in -> alpha + beta A_in of the advantage arriving from
// its end, and maps compose, so a segment can be cut into chunks that are
// reduced in parallel, combined, and replayed from their carry-in.  Three
// kernels:
//  * wave per segment (S <= 256, or L > 256 and S <= 4096): the 64 lanes of
//    a wave take 64 chunks of one segment and combine their maps with a
//    wavefront suffix scan (shuffles): L/64 + log2(64) dependent steps;
//  * chunked lanes (256 < S < 32768, L <= 256): lane = segment, wave = one
//    of 16 chunks of at most 16 steps, kept in registers between the reduce
//    and the replay; the 16 maps of a segment combine through LDS.  A wave
//    reads 64 consecutive segments at each step (coalesced), every input is
//    read once, and a block of 16 waves covers 64 segments, so 11,520
//    segments (the paper's batch) already give 2,880 waves;
//  * otherwise (S >= 32768, or L > 256): a lane per 4 segments with 16-byte
//    accesses when S is a multiple of 4, else a lane per segment; each lane
//    walks its segments backwards, coalesced as above.
#include "common.h"

namespace o5 {

constexpr int kGaeLaneUnroll = 16;

__global__ void __launch_bounds__(256) gae_lane_per_segment(int L, int S, const float* __restrict__ r,
                                                            const float* __restrict__ v,
                                                            const uint8_t* __restrict__ done, float gamma,
                                                            float gl, float* __restrict__ adv,
                                                            float* __restrict__ ret) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  const size_t S_ = static_cast<size_t>(S);
  float carry = 0.0f;
  float vnext = v[static_cast<size_t>(L) * S_ + s];
  int t_hi = L - 1;
  // full chunks: issue all loads of a chunk first, then run the recurrence
  while (t_hi + 1 >= kGaeLaneUnroll) {
    float rr[kGaeLaneUnroll], vv[kGaeLaneUnroll];
    uint8_t dd[kGaeLaneUnroll];
#pragma unroll
    for (int u = 0; u < kGaeLaneUnroll; ++u) {
      const size_t idx = static_cast<size_t>(t_hi - u) * S_ + s;
      rr[u] = r[idx];
      vv[u] = v[idx];
      dd[u] = done[idx];
    }
    __builtin_amdgcn_sched_barrier(0);  // keep every load of the chunk ahead of the recurrence
#pragma unroll
    for (int u = 0; u < kGaeLaneUnroll; ++u) {
      const float nd = dd[u] ? 0.0f : 1.0f;
      const float delta = rr[u] + gamma * nd * vnext - vv[u];
      carry = delta + gl * nd * carry;
      const size_t idx = static_cast<size_t>(t_hi - u) * S_ + s;
      adv[idx] = carry;
      ret[idx] = carry + vv[u];
      vnext = vv[u];
    }
    t_hi -= kGaeLaneUnroll;
  }
  for (; t_hi >= 0; --t_hi) {
    const size_t idx = static_cast<size_t>(t_hi) * S_ + s;
    const float vt = v[idx];
    const float nd = done[idx] ? 0.0f : 1.0f;
    const float delta = r[idx] + gamma * nd * vnext - vt;
    carry = delta + gl * nd * carry;
    adv[idx] = carry;
    ret[idx] = carry + vt;
    vnext = vt;
  }
}

constexpr int kGaeChunks = 16;     // waves per block = chunks per segment
constexpr int kGaeChunkMax = 16;   // steps per chunk (so L <= 256)

// Lane = segment (64 per block), wave c = chunk c of ceil(L / 16) steps.
__global__ void __launch_bounds__(kGaeChunks * 64) gae_chunked(int L, int S, const float* __restrict__ r,
                                                               const float* __restrict__ v,
                                                               const uint8_t* __restrict__ done, float gamma,
                                                               float gl, float* __restrict__ adv,
                                                               float* __restrict__ ret) {
  __shared__ float map_a[kGaeChunks][64], map_b[kGaeChunks][64];
  const int lane = threadIdx.x & 63;
  const int c = threadIdx.x >> 6;
  const int s = blockIdx.x * 64 + lane;
  const bool live = s < S;
  const size_t S_ = static_cast<size_t>(S);
  const int q = (L + kGaeChunks - 1) / kGaeChunks;  // <= kGaeChunkMax (checked on the host)
  const int t0 = c * q;
  const int t1 = min(t0 + q, L);
  // the chunk's inputs, all requests in flight at once
  float rr[kGaeChunkMax], vv[kGaeChunkMax], nd[kGaeChunkMax];
#pragma unroll
  for (int u = 0; u < kGaeChunkMax; ++u) {
    rr[u] = 0.0f;
    vv[u] = 0.0f;
    nd[u] = 1.0f;
    if (live && t0 + u < t1) {
      const size_t idx = static_cast<size_t>(t0 + u) * S_ + s;
      rr[u] = r[idx];
      vv[u] = v[idx];
      nd[u] = done[idx] ? 0.0f : 1.0f;
    }
  }
  const float v_end = (live && t0 < t1) ? v[static_cast<size_t>(t1) * S_ + s] : 0.0f;  // V(t1); row L bootstraps
  // reduce: A(t0) = alpha + beta A(t1)
  float alpha = 0.0f, beta = 1.0f, vn = v_end;
#pragma unroll
  for (int u = kGaeChunkMax - 1; u >= 0; --u) {
    if (t0 + u < t1) {
      const float delta = rr[u] + gamma * nd[u] * vn - vv[u];
      const float k = gl * nd[u];
      alpha = delta + k * alpha;
      beta = k * beta;
      vn = vv[u];
    }
  }
  map_a[c][lane] = alpha;
  map_b[c][lane] = beta;
  __syncthreads();
  // carry-in A(t1): the maps of the later chunks applied to A_L = 0
  float carry = 0.0f;
  for (int k = kGaeChunks - 1; k > c; --k) carry = map_a[k][lane] + map_b[k][lane] * carry;
  // replay from the carry-in
  vn = v_end;
#pragma unroll
  for (int u = kGaeChunkMax - 1; u >= 0; --u) {
    if (t0 + u < t1) {
      const float delta = rr[u] + gamma * nd[u] * vn - vv[u];
      carry = delta + gl * nd[u] * carry;
      if (live) {
        const size_t idx = static_cast<size_t>(t0 + u) * S_ + s;
        adv[idx] = carry;
        ret[idx] = carry + vv[u];
      }
      vn = vv[u];
    }
  }
}

// V consecutive segments per lane (V = 4: 16-byte loads and stores, a wave
// moves 1 KB of a row per instruction), walking backwards in chunks of
// kGaeLaneUnroll steps whose loads are all issued before the recurrence
// runs.  S % V == 0.
template <int V> struct GaeVec;
template <> struct GaeVec<2> {
  typedef float2 F;
  typedef uchar2 U;
  __device__ static float get(const F& v, int k) { return k == 0 ? v.x : v.y; }
  __device__ static uint8_t get(const U& v, int k) { return k == 0 ? v.x : v.y; }
  __device__ static F make(const float* a) { return make_float2(a[0], a[1]); }
};
template <> struct GaeVec<4> {
  typedef float4 F;
  typedef uchar4 U;
  __device__ static float get(const F& v, int k) { return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w; }
  __device__ static uint8_t get(const U& v, int k) { return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w; }
  __device__ static F make(const float* a) { return make_float4(a[0], a[1], a[2], a[3]); }
};

template <int V>
__global__ void __launch_bounds__(64) gae_laneV(int L, int S, const float* __restrict__ r, const float* __restrict__ v,
                                                const uint8_t* __restrict__ done, float gamma, float gl,
                                                float* __restrict__ adv, float* __restrict__ ret) {
  typedef GaeVec<V> G;
  typedef typename G::F F;
  typedef typename G::U U;
  const int g = blockIdx.x * blockDim.x + threadIdx.x;  // segments V g .. V g + V - 1
  const size_t SV = static_cast<size_t>(S) / V;
  if (static_cast<size_t>(g) >= SV) return;
  const F* rv = reinterpret_cast<const F*>(r);
  const F* vv4 = reinterpret_cast<const F*>(v);
  const U* dv = reinterpret_cast<const U*>(done);
  F* av = reinterpret_cast<F*>(adv);
  F* qv = reinterpret_cast<F*>(ret);
  float cy[V], vn[V];
  const F vl = vv4[static_cast<size_t>(L) * SV + g];
#pragma unroll
  for (int k = 0; k < V; ++k) {
    cy[k] = 0.0f;
    vn[k] = G::get(vl, k);
  }
  auto step = [&](size_t idx, const F& rq, const F& vq, const U& dq) {
    float ao[V], ro[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
      const float nd = G::get(dq, k) ? 0.0f : 1.0f;
      const float vs = G::get(vq, k);
      const float delta = G::get(rq, k) + gamma * nd * vn[k] - vs;
      cy[k] = delta + gl * nd * cy[k];
      ao[k] = cy[k];
      ro[k] = cy[k] + vs;
      vn[k] = vs;
    }
    av[idx] = G::make(ao);
    qv[idx] = G::make(ro);
  };
  int t_hi = L - 1;
  while (t_hi + 1 >= kGaeLaneUnroll) {
    F rr[kGaeLaneUnroll], vq[kGaeLaneUnroll];
    U dd[kGaeLaneUnroll];
#pragma unroll
    for (int u = 0; u < kGaeLaneUnroll; ++u) {
      const size_t idx = static_cast<size_t>(t_hi - u) * SV + g;
      rr[u] = rv[idx];
      vq[u] = vv4[idx];
      dd[u] = dv[idx];
    }
    __builtin_amdgcn_sched_barrier(0);  // keep every load of the chunk ahead of the recurrence
#pragma unroll
    for (int u = 0; u < kGaeLaneUnroll; ++u) step(static_cast<size_t>(t_hi - u) * SV + g, rr[u], vq[u], dd[u]);
    t_hi -= kGaeLaneUnroll;
  }
  for (; t_hi >= 0; --t_hi) {
    const size_t idx = static_cast<size_t>(t_hi) * SV + g;
    step(idx, rv[idx], vv4[idx], dv[idx]);
  }
}

// One wave (64 lanes) per segment; blockDim = 256 holds 4 segments.
__global__ void __launch_bounds__(256) gae_wave_per_segment(int L, int S, const float* __restrict__ r,
                                                            const float* __restrict__ v,
                                                            const uint8_t* __restrict__ done, float gamma,
                                                            float gl, float* __restrict__ adv,
                                                            float* __restrict__ ret) {
  const int lane = threadIdx.x & 63;
  const int s = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (s >= S) return;  // whole wave exits together
  const size_t S_ = static_cast<size_t>(S);
  const int q = (L + 63) / 64;             // steps per lane
  const int t0 = lane * q;                 // this lane's chunk [t0, t1)
  const int t1 = min(t0 + q, L);

  // 1) reduce the chunk to A(t0) = alpha + beta * A(t1), with A(t1) unknown
  float alpha = 0.0f, beta = 1.0f;
  for (int t = t1 - 1; t >= t0; --t) {
    const size_t idx = static_cast<size_t>(t) * S_ + s;
    const float nd = done[idx] ? 0.0f : 1.0f;
    const float delta = r[idx] + gamma * nd * v[idx + S_] - v[idx];
    const float c = gl * nd;
    alpha = delta + c * alpha;
    beta = c * beta;
  }
  // 2) suffix scan of the maps: lane j ends with F_j = f_j o f_{j+1} o ... o f_63
  for (int d = 1; d < 64; d <<= 1) {
    const float a2 = __shfl_down(alpha, d, 64);
    const float b2 = __shfl_down(beta, d, 64);
    if (lane + d < 64) {
      alpha = alpha + beta * a2;
      beta = beta * b2;
    }
  }
  // carry-in of lane j is A at the start of chunk j+1, i.e. F_{j+1}(0)
  float carry = __shfl_down(alpha, 1, 64);
  if (lane == 63) carry = 0.0f;
  // 3) replay the chunk from its carry-in
  for (int t = t1 - 1; t >= t0; --t) {
    const size_t idx = static_cast<size_t>(t) * S_ + s;
    const float vt = v[idx];
    const float nd = done[idx] ? 0.0f : 1.0f;
    const float delta = r[idx] + gamma * nd * v[idx + S_] - vt;
    carry = delta + gl * nd * carry;
    adv[idx] = carry;
    ret[idx] = carry + vt;
  }
}

// One thread per (t, b) of the sample layout, grid-stride; every index is
// 64-bit, so T * B = L * S may exceed 2^31.
__global__ void __launch_bounds__(256) segments_to_samples_kernel(int L, int S, int T,
                                                                  const float* __restrict__ adv,
                                                                  const float* __restrict__ ret,
                                                                  const uint8_t* __restrict__ done,
                                                                  float* __restrict__ adv_s,
                                                                  float* __restrict__ ret_s,
                                                                  uint8_t* __restrict__ reset) {
  const size_t J = static_cast<size_t>(L / T);
  const size_t S_ = static_cast<size_t>(S);
  const size_t B = S_ * J;
  const size_t total = static_cast<size_t>(T) * B;
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total; i += stride) {
    const size_t t = i / B;
    const size_t b = i - t * B;
    const size_t s = b / J;
    const size_t j = b - s * J;
    const size_t src = (static_cast<size_t>(T) * j + t) * S_ + s;
    adv_s[i] = adv[src];
    ret_s[i] = ret[src];
    reset[i] = (t > 0 && done[src - S_] != 0) ? 1 : 0;
  }
}

}  // namespace o5

using namespace o5;

// Segments per launch up to which the wave-per-segment scan is used (for
// segments longer than the chunked kernel takes: up to kGaeWaveScanLongMaxS),
// and below which the chunked-lane kernel is (above it there are enough
// lanes for one per segment, and 16-byte accesses stream better).  At L =
// 256 the chunked kernel (16 chunks of 16 steps) beats the wave scan from a
// few hundred segments on: 16 against 57 us at S = 4096.
static constexpr int kGaeWaveScanMaxS = 256;
static constexpr int kGaeWaveScanLongMaxS = 4096;
static constexpr int kGaeChunkedMaxS = 32768;
static constexpr int kGaeLaneV = 4;  // segments per lane of the large-S kernel

extern "C" int o5_gae(int L, int S, const float* r, const float* v, const uint8_t* done, float gamma,
                      float lambda, float* adv, float* ret, void* stream) {
  O5_CHECK(L >= 1 && S >= 1, O5_E_SHAPE, "o5_gae: L=%d and S=%d must be >= 1", L, S);
  O5_CHECK((static_cast<long long>(L) + 1) * S < (1ll << 40), O5_E_SHAPE, "o5_gae: L*S too large");
  O5_CHECK(gamma >= 0.0f && gamma <= 1.0f && lambda >= 0.0f && lambda <= 1.0f, O5_E_ARG,
           "o5_gae: gamma=%g and lambda=%g must lie in [0, 1]", gamma, lambda);
  O5_PTR(r, "r");
  O5_PTR(v, "v");
  O5_PTR(done, "done");
  O5_PTR(adv, "adv");
  O5_PTR(ret, "ret");
  const float gl = gamma * lambda;
  ktimer_begin(kSiteGae, as_stream(stream));
  const bool chunkable = L <= kGaeChunks * kGaeChunkMax;
  if (S <= kGaeWaveScanMaxS || (!chunkable && S <= kGaeWaveScanLongMaxS)) {
    hipLaunchKernelGGL(gae_wave_per_segment, dim3((S + 3) / 4), dim3(256), 0, as_stream(stream), L, S,
                       r, v, done, gamma, gl, adv, ret);
  } else if (S < kGaeChunkedMaxS && chunkable) {
    hipLaunchKernelGGL(gae_chunked, dim3((S + 63) / 64), dim3(kGaeChunks * 64), 0, as_stream(stream), L, S, r, v,
                       done, gamma, gl, adv, ret);
  } else if (S % kGaeLaneV == 0 && aligned16(r) && aligned16(v) && aligned16(adv) && aligned16(ret) &&
             reinterpret_cast<uintptr_t>(done) % kGaeLaneV == 0) {
    hipLaunchKernelGGL(gae_laneV<kGaeLaneV>, dim3((S / kGaeLaneV + 63) / 64), dim3(64), 0, as_stream(stream), L, S,
                       r, v, done, gamma, gl, adv, ret);
  } else {
    hipLaunchKernelGGL(gae_lane_per_segment, dim3((S + 255) / 256), dim3(256), 0, as_stream(stream), L,
                       S, r, v, done, gamma, gl, adv, ret);
  }
  ktimer_end(kSiteGae, as_stream(stream));
  return check_launch("o5_gae");
}

extern "C" int o5_segments_to_samples(int L, int S, int T, const float* adv, const float* ret,
                                      const uint8_t* done, float* adv_s, float* ret_s, uint8_t* reset,
                                      void* stream) {
  O5_CHECK(L >= 1 && S >= 1 && T >= 1 && L % T == 0, O5_E_SHAPE,
           "o5_segments_to_samples: need L, S, T >= 1 and T | L (L=%d S=%d T=%d)", L, S, T);
  O5_CHECK(static_cast<long long>(L) * S < (1ll << 40), O5_E_SHAPE, "o5_segments_to_samples: too large");
  O5_PTR(adv, "adv");
  O5_PTR(ret, "ret");
  O5_PTR(done, "done");
  O5_PTR(adv_s, "adv_s");
  O5_PTR(ret_s, "ret_s");
  O5_PTR(reset, "reset");
  const size_t total = static_cast<size_t>(L) * S;
  const size_t blocks = std::min<size_t>((total + 255) / 256, size_t{1} << 20);
  hipLaunchKernelGGL(segments_to_samples_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     as_stream(stream), L, S, T, adv, ret, done, adv_s, ret_s, reset);
  return check_launch("o5_segments_to_samples");
}
