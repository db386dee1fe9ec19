// The LSTM's input side: running observation normalisation (appendix
// "Observation Space": subtract a running mean, divide by a running standard
// deviation of all data ever observed, clip to (-5, 5)), then the pre-LSTM
// fully-connected layer and the cross-hero pool (appendix "Neural Network
// Architecture": the first 25% of the vector max-pooled across the five
// replica networks of a team), forward and backward.
//
//   o   = clip((obs - mean) / sqrt(var + eps), -5, 5)      obs_stats/finalize/apply
//   y   = relu(o W^T + b)                                  GEMM + bias/ReLU epilogue
//   x   = y, its first D/4 features replaced by their      pool_fwd
//         maximum over the team's 5 replicas
//   dpre = pool and ReLU backward of dx                    pool_bwd (+ db partials)
//   dW  = dpre^T o,  db = column sums of dpre              GEMM, fixed-order sums
//
// Replicas are five consecutive samples b = 5 q + r; rows n = t B + b.  A
// thread of the pool kernels owns one feature j of one team-timestep (5
// rows), so the maximum, its first arg-maximum and the summed gradient stay
// in registers; a wave covers 64 consecutive features (coalesced).  Every
// reduction has a fixed order, so results are bitwise reproducible.
#include "gemm_plan.h"
#include "reduce.h"

namespace o5 {

constexpr int kReplicas = 5;
constexpr int kObsRowsPerChunk = 128;

struct ColSummary {
  double n, mean, m2;
};

__device__ __forceinline__ ColSummary merge_cols(const ColSummary& a, const ColSummary& b) {
  const double n = a.n + b.n;
  if (n == 0.0) return a;
  const double d = b.mean - a.mean;
  return {n, a.mean + d * (b.n / n), a.m2 + b.m2 + d * d * (a.n * b.n / n)};
}

// part[c][j]: count, mean and M2 of feature j over rows of chunk c, from
// sums shifted by the chunk's first value (exact enough in fp64 for fp32
// data, one division per chunk).  A thread owns 4 consecutive features
// (16-byte loads: a wave reads 1 KB of a row).
__global__ void __launch_bounds__(256) obs_stats(int N, int Do, const float* __restrict__ obs,
                                                 ColSummary* __restrict__ part) {
  const int j = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (j >= Do) return;
  const int r0 = blockIdx.y * kObsRowsPerChunk;
  const int r1 = min(N, r0 + kObsRowsPerChunk);
  const float4 f0 = *reinterpret_cast<const float4*>(obs + static_cast<size_t>(r0) * Do + j);
  const double x0[4] = {f0.x, f0.y, f0.z, f0.w};
  double s1[4] = {0.0, 0.0, 0.0, 0.0}, s2[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
  for (int r = r0; r < r1; ++r) {
    const float4 f = *reinterpret_cast<const float4*>(obs + static_cast<size_t>(r) * Do + j);
    const float v[4] = {f.x, f.y, f.z, f.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const double d = static_cast<double>(v[q]) - x0[q];
      s1[q] += d;
      s2[q] += d * d;
    }
  }
  const double n = r1 - r0;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    part[static_cast<size_t>(blockIdx.y) * Do + j + q] = {n, x0[q] + s1[q] / n, fmax(s2[q] - s1[q] * s1[q] / n, 0.0)};
}

// Merge the chunks into the running summary stats [3][Do] (counts, means,
// M2), write it back, and leave mean and 1/sqrt(var + eps) in fp32.  Block =
// 64 features x 4 chunk lanes: lane q merges chunks q, q + 4, ... in order,
// then the four lane summaries of a feature merge in order 0..3.
__global__ void __launch_bounds__(256) obs_finalize(int Do, int nchunks, const ColSummary* __restrict__ part,
                                                    double* __restrict__ stats, float eps, float* __restrict__ mean_f,
                                                    float* __restrict__ rstd_f) {
  __shared__ ColSummary lane_sum[4][64];
  const int jj = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + jj;
  ColSummary b{0.0, 0.0, 0.0};
  if (j < Do) {
#pragma unroll 8
    for (int c = q; c < nchunks; c += 4) b = merge_cols(b, part[static_cast<size_t>(c) * Do + j]);
  }
  lane_sum[q][jj] = b;
  __syncthreads();
  if (q != 0 || j >= Do) return;
  ColSummary t = lane_sum[0][jj];
  for (int k = 1; k < 4; ++k) t = merge_cols(t, lane_sum[k][jj]);
  const ColSummary run = merge_cols(ColSummary{stats[j], stats[Do + j], stats[2 * Do + j]}, t);
  stats[j] = run.n;
  stats[Do + j] = run.mean;
  stats[2 * Do + j] = run.m2;
  mean_f[j] = static_cast<float>(run.mean);
  rstd_f[j] = static_cast<float>(1.0 / sqrt(run.m2 / run.n + static_cast<double>(eps)));
}

template <typename E>
__global__ void __launch_bounds__(256) obs_apply(size_t total4, int Do, const float* __restrict__ obs,
                                                 const float* __restrict__ mean_f, const float* __restrict__ rstd_f,
                                                 float clip, E* __restrict__ o) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;  // 4 consecutive elements
  if (i >= total4) return;
  const int j = static_cast<int>((i * 4) % Do);
  const float4 x = reinterpret_cast<const float4*>(obs)[i];
  const float4 m = *reinterpret_cast<const float4*>(mean_f + j);
  const float4 s = *reinterpret_cast<const float4*>(rstd_f + j);
  float4 v;
  v.x = fminf(fmaxf((x.x - m.x) * s.x, -clip), clip);
  v.y = fminf(fmaxf((x.y - m.y) * s.y, -clip), clip);
  v.z = fminf(fmaxf((x.z - m.z) * s.z, -clip), clip);
  v.w = fminf(fmaxf((x.w - m.w) * s.w, -clip), clip);
  if constexpr (sizeof(E) == 2) {
    uint2 u;
    u.x = f32x2_to_bf16x2(v.x, v.y);
    u.y = f32x2_to_bf16x2(v.z, v.w);
    *reinterpret_cast<uint2*>(o + i * 4) = u;
  } else {
    *reinterpret_cast<float4*>(o + i * 4) = v;
  }
}

// y = relu(acc + b) in fp32.
struct EpiBiasRelu {
  static constexpr int kTileSmem = 0;
  float* y;
  const float* bias;
  int ld;
  __device__ __forceinline__ void operator()(int i, int j, float v, int) const {
    y[static_cast<size_t>(i) * ld + j] = fmaxf(v + bias[j], 0.0f);
  }
};

// Thread = feature j of team-timestep g (rows 5 g .. 5 g + 4).
template <typename E>
__global__ void __launch_bounds__(256) pool_fwd(int groups, int D, int P, const float* __restrict__ y,
                                                E* __restrict__ x) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int g = blockIdx.y;
  if (j >= D || g >= groups) return;
  const size_t base = static_cast<size_t>(g) * kReplicas * D + j;
  float v[kReplicas];
#pragma unroll
  for (int r = 0; r < kReplicas; ++r) v[r] = y[base + static_cast<size_t>(r) * D];
  if (j < P) {
    float m = v[0];
#pragma unroll
    for (int r = 1; r < kReplicas; ++r) m = fmaxf(m, v[r]);
#pragma unroll
    for (int r = 0; r < kReplicas; ++r) v[r] = m;
  }
#pragma unroll
  for (int r = 0; r < kReplicas; ++r) x[base + static_cast<size_t>(r) * D] = elem<E>::from_f32(v[r]);
}

// dpre for the 5 rows of team-timestep g, feature j; the column sums of the
// (unrounded) dpre over this block's row-groups go to dbpart[blockIdx.y][j].
template <typename E>
__global__ void __launch_bounds__(256) pool_bwd(int groups, int D, int P, int groups_per_block,
                                                const float* __restrict__ y, const E* __restrict__ dx,
                                                E* __restrict__ dpre, float* __restrict__ dbpart) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= D) return;
  const int g0 = blockIdx.y * groups_per_block;
  const int g1 = min(groups, g0 + groups_per_block);
  float dbs = 0.0f;
  for (int g = g0; g < g1; ++g) {
    const size_t base = static_cast<size_t>(g) * kReplicas * D + j;
    float yv[kReplicas], d[kReplicas];
#pragma unroll
    for (int r = 0; r < kReplicas; ++r) {
      yv[r] = y[base + static_cast<size_t>(r) * D];
      d[r] = elem<E>::to_f32(dx[base + static_cast<size_t>(r) * D]);
    }
    if (j < P) {
      // the summed gradient goes to the first replica attaining the maximum
      int win = 0;
      float tot = d[0];
#pragma unroll
      for (int r = 1; r < kReplicas; ++r) {
        if (yv[r] > yv[win]) win = r;
        tot += d[r];
      }
#pragma unroll
      for (int r = 0; r < kReplicas; ++r) d[r] = r == win ? tot : 0.0f;
    }
#pragma unroll
    for (int r = 0; r < kReplicas; ++r) {
      const float v = yv[r] > 0.0f ? d[r] : 0.0f;
      dbs += v;
      dpre[base + static_cast<size_t>(r) * D] = elem<E>::from_f32(v);
    }
  }
  dbpart[static_cast<size_t>(blockIdx.y) * D + j] = dbs;
}

// ------------------------------------------------------------ workspaces

struct ObsWs {
  size_t part, mean, rstd, total;
  int nchunks;
};

static ObsWs obs_ws(int N, int Do) {
  ObsWs w;
  w.nchunks = cdiv(N, kObsRowsPerChunk);
  w.part = 0;
  w.mean = align_up(static_cast<size_t>(w.nchunks) * Do * sizeof(ColSummary));
  w.rstd = w.mean + align_up(static_cast<size_t>(Do) * 4);
  w.total = w.rstd + align_up(static_cast<size_t>(Do) * 4);
  return w;
}

constexpr int kPoolGroupsPerBlock = 64;

struct PreBwdWs {
  size_t dpre, dbpart, total;
  int nby;
};

static PreBwdWs prelstm_bwd_ws(o5_dtype dt, int N, int D) {
  PreBwdWs w;
  const int groups = N / kReplicas;
  w.nby = cdiv(groups, kPoolGroupsPerBlock);
  w.dpre = 0;
  w.dbpart = align_up(static_cast<size_t>(N) * D * (dt == O5_BF16 ? 2 : 4));
  w.total = w.dbpart + align_up(static_cast<size_t>(w.nby) * D * 4);
  return w;
}

template <typename E>
static void prelstm_fwd_impl(int N, int Do, int D, const E* o, const E* W, const float* b, float* y, E* x,
                             hipStream_t s) {
  GemmPlan plan = plan_gemm(sizeof(E) == 2, N, D, Do);
  plan.splits = 1;  // the epilogue needs whole sums
  KRows2<E> al{o, nullptr, nullptr, Do, 0, Do, Do, N};
  KRows2<E> bl{W, nullptr, nullptr, Do, 0, Do, Do, D};
  run_gemm(plan, al, bl, EpiBiasRelu{y, b, D}, N, D, Do, s);
  const int groups = N / kReplicas;
  hipLaunchKernelGGL(pool_fwd<E>, dim3(cdiv(D, 256), groups), dim3(256), 0, s, groups, D, D / 4, y, x);
}

template <typename E>
static void prelstm_bwd_impl(int N, int Do, int D, const E* o, const float* y, const E* dx, float* dW, float* db,
                             char* ws, const PreBwdWs& w, hipStream_t s) {
  E* dpre = reinterpret_cast<E*>(ws + w.dpre);
  float* dbpart = reinterpret_cast<float*>(ws + w.dbpart);
  const int groups = N / kReplicas;
  hipLaunchKernelGGL(pool_bwd<E>, dim3(cdiv(D, 256), w.nby), dim3(256), 0, s, groups, D, D / 4, kPoolGroupsPerBlock, y,
                     dx, dpre, dbpart);
  hipLaunchKernelGGL(colsum_rows4, dim3(cdiv(D, 64)), dim3(256), 0, s, w.nby, D, dbpart, db);
  // dW[d, k] = sum_n dpre[n, d] o[n, k]: both operands I-contiguous
  GemmPlan plan = plan_gemm(sizeof(E) == 2, D, Do, N);
  plan.splits = 1;
  ICols2<E> al{dpre, nullptr, nullptr, nullptr, D, 0, D, D, N, 0};
  ICols2<E> bl{o, nullptr, nullptr, nullptr, Do, 0, Do, Do, N, 0};
  run_gemm(plan, al, bl, EpiStoreF32{dW, Do, 0}, D, Do, N, s);
}

static int check_prelstm(const char* fn, o5_dtype dt, int T, int B, int Do, int D) {
  O5_CHECK(dt == O5_F32 || dt == O5_BF16, O5_E_DTYPE, "%s: unknown dtype %d", fn, static_cast<int>(dt));
  O5_CHECK(T >= 1 && B >= kReplicas && B % kReplicas == 0, O5_E_SHAPE,
           "%s: need T >= 1 and B a positive multiple of 5 (T=%d B=%d)", fn, T, B);
  O5_CHECK(Do >= 64 && Do % 64 == 0 && D >= 64 && D % 64 == 0, O5_E_SHAPE,
           "%s: Do=%d and D=%d must be positive multiples of 64", fn, Do, D);
  O5_CHECK(static_cast<long long>(T) * B < (1ll << 31) && static_cast<long long>(T) * B * (Do > D ? Do : D) < (1ll << 31),
           O5_E_SHAPE, "%s: T*B*max(Do, D) too large", fn);
  O5_CHECK(T * B / kReplicas <= 65535, O5_E_SHAPE, "%s: T*B/5 must be <= 65535", fn);
  return O5_OK;
}

}  // namespace o5

using namespace o5;

static int check_obs_shape(const char* fn, int N, int Do) {
  O5_CHECK(N >= 1 && Do >= 4 && Do % 4 == 0, O5_E_SHAPE, "%s: need N >= 1 and Do a positive multiple of 4", fn);
  O5_CHECK(static_cast<long long>(N) * Do < (1ll << 40) && cdiv(N, kObsRowsPerChunk) <= 65535, O5_E_SHAPE,
           "%s: N*Do too large", fn);
  return O5_OK;
}

extern "C" size_t o5_obs_normalize_workspace_bytes(int N, int Do) {
  if (check_obs_shape("o5_obs_normalize_workspace_bytes", N, Do) != O5_OK) return 0;
  return obs_ws(N, Do).total;
}

extern "C" int o5_obs_normalize(o5_dtype dt, int N, int Do, const float* obs, double* stats, float clip, float eps,
                                void* o, void* ws, size_t ws_bytes, void* stream) {
  O5_CHECK(dt == O5_F32 || dt == O5_BF16, O5_E_DTYPE, "o5_obs_normalize: unknown dtype %d", static_cast<int>(dt));
  {
    const int st = check_obs_shape("o5_obs_normalize", N, Do);
    if (st != O5_OK) return st;
  }
  O5_CHECK(clip > 0.0f && eps > 0.0f, O5_E_ARG, "o5_obs_normalize: need clip > 0 and eps > 0");
  O5_PTR(obs, "obs");
  O5_PTR(stats, "stats");
  O5_PTR(o, "o");
  const ObsWs w = obs_ws(N, Do);
  O5_CHECK(ws != nullptr && ws_bytes >= w.total, O5_E_WORKSPACE,
           "o5_obs_normalize: workspace needs %zu bytes, got %zu", w.total, ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "o5_obs_normalize: 'ws' is not 16-byte aligned");
  char* wsb = static_cast<char*>(ws);
  ColSummary* part = reinterpret_cast<ColSummary*>(wsb + w.part);
  float* mean_f = reinterpret_cast<float*>(wsb + w.mean);
  float* rstd_f = reinterpret_cast<float*>(wsb + w.rstd);
  hipStream_t s = as_stream(stream);
  ktimer_begin(kSiteObsNorm, s);
  hipLaunchKernelGGL(obs_stats, dim3(cdiv(Do, 1024), w.nchunks), dim3(256), 0, s, N, Do, obs, part);
  hipLaunchKernelGGL(obs_finalize, dim3(cdiv(Do, 64)), dim3(256), 0, s, Do, w.nchunks, part, stats, eps, mean_f, rstd_f);
  const size_t total4 = static_cast<size_t>(N) * Do / 4;
  const dim3 grid(static_cast<unsigned>((total4 + 255) / 256));
  if (dt == O5_BF16)
    hipLaunchKernelGGL(obs_apply<uint16_t>, grid, dim3(256), 0, s, total4, Do, obs, mean_f, rstd_f, clip,
                       static_cast<uint16_t*>(o));
  else
    hipLaunchKernelGGL(obs_apply<float>, grid, dim3(256), 0, s, total4, Do, obs, mean_f, rstd_f, clip,
                       static_cast<float*>(o));
  ktimer_end(kSiteObsNorm, s);
  return check_launch("o5_obs_normalize");
}

extern "C" int o5_prelstm_fwd(o5_dtype dt, int T, int B, int Do, int D, const void* o, const void* W, const float* b,
                              float* y, void* x, void* stream) {
  int st = check_prelstm("o5_prelstm_fwd", dt, T, B, Do, D);
  if (st != O5_OK) return st;
  O5_PTR(o, "o");
  O5_PTR(W, "W");
  O5_PTR(b, "b");
  O5_PTR(y, "y");
  O5_PTR(x, "x");
  hipStream_t s = as_stream(stream);
  const int N = T * B;
  ktimer_begin(kSitePreFwd, s);
  if (dt == O5_BF16)
    prelstm_fwd_impl<uint16_t>(N, Do, D, static_cast<const uint16_t*>(o), static_cast<const uint16_t*>(W), b, y,
                               static_cast<uint16_t*>(x), s);
  else
    prelstm_fwd_impl<float>(N, Do, D, static_cast<const float*>(o), static_cast<const float*>(W), b, y,
                            static_cast<float*>(x), s);
  ktimer_end(kSitePreFwd, s);
  return check_launch("o5_prelstm_fwd");
}

extern "C" size_t o5_prelstm_bwd_workspace_bytes(o5_dtype dt, int T, int B, int Do, int D) {
  if (check_prelstm("o5_prelstm_bwd_workspace_bytes", dt, T, B, Do, D) != O5_OK) return 0;
  return prelstm_bwd_ws(dt, T * B, D).total;
}

extern "C" int o5_prelstm_bwd(o5_dtype dt, int T, int B, int Do, int D, const void* o, const float* y, const void* dx,
                              float* dW, float* db, void* ws, size_t ws_bytes, void* stream) {
  int st = check_prelstm("o5_prelstm_bwd", dt, T, B, Do, D);
  if (st != O5_OK) return st;
  O5_PTR(o, "o");
  O5_PTR(y, "y");
  O5_PTR(dx, "dx");
  O5_PTR(dW, "dW");
  O5_PTR(db, "db");
  const PreBwdWs w = prelstm_bwd_ws(dt, T * B, D);
  O5_CHECK(ws != nullptr && ws_bytes >= w.total, O5_E_WORKSPACE,
           "o5_prelstm_bwd: workspace needs %zu bytes, got %zu", w.total, ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "o5_prelstm_bwd: 'ws' is not 16-byte aligned");
  hipStream_t s = as_stream(stream);
  const int N = T * B;
  ktimer_begin(kSitePreBwd, s);
  if (dt == O5_BF16)
    prelstm_bwd_impl<uint16_t>(N, Do, D, static_cast<const uint16_t*>(o), y, static_cast<const uint16_t*>(dx), dW, db,
                               static_cast<char*>(ws), w, s);
  else
    prelstm_bwd_impl<float>(N, Do, D, static_cast<const float*>(o), y, static_cast<const float*>(dx), dW, db,
                            static_cast<char*>(ws), w, s);
  ktimer_end(kSitePreBwd, s);
  return check_launch("o5_prelstm_bwd");
}
