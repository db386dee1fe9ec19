// Reward post-processing ahead of GAE (appendix "Reward Weights": game time
// weighting, team spirit, zero sum; Table "Hyperparameters": rewards are
// normalised by a running estimate of their standard deviation).
//
// The ten heroes of a game are ten adjacent segments of the [L, S] layout,
// so one thread owns one (step, game): it reads 10 shaped rewards, 10
// outcomes and the game time (84 bytes, 8-byte loads; a wave reads 64
// consecutive games) and forms the ten processed rewards z in registers.
// (Staging the 10-wide rows through LDS for 16-byte coalesced loads measured
// slower: the block-wide barriers serialise the tiles.)
// The normalisation needs the variance of every z before any output can be
// written, hence three launches:
//  1. reward_stats: z per (step, game); per-block (count, mean, M2) in fp64,
//     merged in a fixed tree order;
//  2. reward_finalize (one block): merges the block summaries in a fixed
//     order, merges the result into the running summary, writes it back,
//     and stores 1 / sqrt(var + eps);
//  3. reward_apply: recomputes z (cheaper than a round trip of z through
//     HBM: the same 84 bytes are read either way) and writes r = z * scale.
// 20.8 bytes move per (step, segment) against 12.4 that the operation needs
// at least (inputs once, output once): the inputs are read twice.
#include "common.h"

namespace o5 {

constexpr int kHeroes = 10;       // two teams of five
constexpr int kRwThreads = 256;
constexpr int kRwMaxBlocks = 1024;

struct Summary {
  double n, mean, m2;  // count, mean, sum of squared deviations
};

// Pairwise merge of two summaries of disjoint sets (Chan, Golub, LeVeque).
__device__ __forceinline__ Summary merge(const Summary& a, const Summary& b) {
  const double n = a.n + b.n;
  if (n == 0.0) return a;
  const double d = b.mean - a.mean;
  return {n, a.mean + d * (b.n / n), a.m2 + b.m2 + d * d * (a.n * b.n / n)};
}

struct RewardConsts {
  float tau;
  float log2_base_per_minute;  // log2(decay_base) / decay_minutes
};

// The ten processed rewards z of one (step, game) from its raw rewards rho
// (time weight already applied, outcome added).
__device__ __forceinline__ void mix_game(const float (&rho)[kHeroes], float tau, float (&z)[kHeroes]) {
  const float ma = 0.2f * (rho[0] + rho[1] + rho[2] + rho[3] + rho[4]);
  const float mb = 0.2f * (rho[5] + rho[6] + rho[7] + rho[8] + rho[9]);
  const float keep = 1.0f - tau;
  // team spirit mixes in the own team's mean; zero sum takes the enemies'
  // mean (team spirit leaves a team's mean unchanged)
  const float off_a = tau * ma - mb, off_b = tau * mb - ma;
#pragma unroll
  for (int k = 0; k < 5; ++k) {
    z[k] = keep * rho[k] + off_a;
    z[5 + k] = keep * rho[5 + k] + off_b;
  }
}

// The ten processed rewards of game g at step t (item i = t * G + g), read
// with 8-byte loads (a wave covers 64 consecutive games, 2.5 KB per array).
__device__ __forceinline__ void shape_game(const float* __restrict__ shaped, const float* __restrict__ outcome,
                                           const float* __restrict__ game_time, size_t i, const RewardConsts& c,
                                           float (&z)[kHeroes]) {
  const float w = exp2f(c.log2_base_per_minute * game_time[i]);
  const float2* s2 = reinterpret_cast<const float2*>(shaped + i * kHeroes);
  float rho[kHeroes];
#pragma unroll
  for (int k = 0; k < kHeroes / 2; ++k) {
    const float2 v = s2[k];
    rho[2 * k] = v.x * w;
    rho[2 * k + 1] = v.y * w;
  }
  if (outcome) {
    const float2* o2 = reinterpret_cast<const float2*>(outcome + i * kHeroes);
#pragma unroll
    for (int k = 0; k < kHeroes / 2; ++k) {
      const float2 v = o2[k];
      rho[2 * k] += v.x;
      rho[2 * k + 1] += v.y;
    }
  }
  mix_game(rho, c.tau, z);
}

// Fixed-order tree merge of one summary per thread; the result is valid in
// thread 0.
__device__ Summary block_merge(Summary s, Summary* lds) {
  const int tid = threadIdx.x;
  lds[tid] = s;
  __syncthreads();
  for (int w = kRwThreads / 2; w > 0; w >>= 1) {
    if (tid < w) lds[tid] = merge(lds[tid], lds[tid + w]);
    __syncthreads();
  }
  return lds[0];
}

__global__ void __launch_bounds__(kRwThreads) reward_stats(size_t items, const float* __restrict__ shaped,
                                                           const float* __restrict__ outcome,
                                                           const float* __restrict__ game_time, RewardConsts c,
                                                           Summary* __restrict__ part) {
  __shared__ Summary lds[kRwThreads];
  Summary s{0.0, 0.0, 0.0};
  for (size_t i = static_cast<size_t>(blockIdx.x) * kRwThreads + threadIdx.x; i < items;
       i += static_cast<size_t>(gridDim.x) * kRwThreads) {
    float z[kHeroes];
    shape_game(shaped, outcome, game_time, i, c, z);
    double sum = 0.0;
#pragma unroll
    for (int k = 0; k < kHeroes; ++k) sum += z[k];
    const double m = sum / kHeroes;
    double q = 0.0;
#pragma unroll
    for (int k = 0; k < kHeroes; ++k) {
      const double d = z[k] - m;
      q += d * d;
    }
    s = merge(s, Summary{static_cast<double>(kHeroes), m, q});
  }
  const Summary b = block_merge(s, lds);
  if (threadIdx.x == 0) part[blockIdx.x] = b;
}

__global__ void __launch_bounds__(kRwThreads) reward_finalize(int nparts, const Summary* __restrict__ part,
                                                              double* __restrict__ stats, float eps,
                                                              float* __restrict__ scale) {
  __shared__ Summary lds[kRwThreads];
  Summary s{0.0, 0.0, 0.0};
  for (int i = threadIdx.x; i < nparts; i += kRwThreads) s = merge(s, part[i]);
  const Summary b = block_merge(s, lds);
  if (threadIdx.x == 0) {
    const Summary run = merge(Summary{stats[0], stats[1], stats[2]}, b);
    stats[0] = run.n;
    stats[1] = run.mean;
    stats[2] = run.m2;
    *scale = static_cast<float>(1.0 / sqrt(run.m2 / run.n + static_cast<double>(eps)));
  }
}

__global__ void __launch_bounds__(kRwThreads) reward_apply(size_t items, const float* __restrict__ shaped,
                                                           const float* __restrict__ outcome,
                                                           const float* __restrict__ game_time, RewardConsts c,
                                                           const float* __restrict__ scale, float* __restrict__ r) {
  const float k = *scale;
  for (size_t i = static_cast<size_t>(blockIdx.x) * kRwThreads + threadIdx.x; i < items;
       i += static_cast<size_t>(gridDim.x) * kRwThreads) {
    float z[kHeroes];
    shape_game(shaped, outcome, game_time, i, c, z);
    float2* r2 = reinterpret_cast<float2*>(r + i * kHeroes);
#pragma unroll
    for (int q = 0; q < kHeroes / 2; ++q) r2[q] = make_float2(z[2 * q] * k, z[2 * q + 1] * k);
  }
}

struct RewardWs {
  size_t part, scale, total;
  int blocks;
};

static RewardWs reward_ws(int L, int G) {
  RewardWs w;
  const size_t items = static_cast<size_t>(L) * G;
  w.blocks = static_cast<int>(std::min<size_t>((items + kRwThreads - 1) / kRwThreads, kRwMaxBlocks));
  w.part = 0;
  w.scale = align_up(static_cast<size_t>(w.blocks) * sizeof(Summary));
  w.total = w.scale + align_up(sizeof(float));
  return w;
}

}  // namespace o5

using namespace o5;

static int check_reward_shape(const char* fn, int L, int G) {
  O5_CHECK(L >= 1 && G >= 1, O5_E_SHAPE, "%s: L=%d and G=%d must be >= 1", fn, L, G);
  O5_CHECK(static_cast<long long>(L) * G < (1ll << 31) && static_cast<long long>(L) * G * kHeroes < (1ll << 31),
           O5_E_SHAPE, "%s: L*G*10 must stay below 2^31", fn);
  return O5_OK;
}

extern "C" size_t o5_reward_process_workspace_bytes(int L, int G) {
  if (check_reward_shape("o5_reward_process_workspace_bytes", L, G) != O5_OK) return 0;
  return reward_ws(L, G).total;
}

extern "C" int o5_reward_process(int L, int G, const float* shaped, const float* outcome, const float* game_time,
                                 o5_reward_hp hp, double* stats, float* r, void* ws, size_t ws_bytes,
                                 void* stream) {
  {
    const int st = check_reward_shape("o5_reward_process", L, G);
    if (st != O5_OK) return st;
  }
  O5_CHECK(hp.tau >= 0.0f && hp.tau <= 1.0f, O5_E_ARG, "o5_reward_process: tau=%g must lie in [0, 1]", hp.tau);
  O5_CHECK(hp.decay_base > 0.0f && hp.decay_base <= 1.0f && hp.decay_minutes > 0.0f && hp.eps > 0.0f, O5_E_ARG,
           "o5_reward_process: need 0 < decay_base <= 1, decay_minutes > 0 and eps > 0");
  O5_PTR(shaped, "shaped");
  O5_OPT_PTR(outcome, "outcome");
  O5_PTR(game_time, "game_time");
  O5_PTR(stats, "stats");
  O5_PTR(r, "r");
  const RewardWs w = reward_ws(L, G);
  O5_CHECK(ws != nullptr && ws_bytes >= w.total, O5_E_WORKSPACE,
           "o5_reward_process: workspace needs %zu bytes, got %zu", w.total,
           ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "o5_reward_process: 'ws' is not 16-byte aligned");
  RewardConsts c;
  c.tau = hp.tau;
  c.log2_base_per_minute = static_cast<float>(std::log2(static_cast<double>(hp.decay_base)) / hp.decay_minutes);
  const size_t items = static_cast<size_t>(L) * G;
  char* wsb = static_cast<char*>(ws);
  Summary* part = reinterpret_cast<Summary*>(wsb + w.part);
  float* scale = reinterpret_cast<float*>(wsb + w.scale);
  hipStream_t s = as_stream(stream);
  ktimer_begin(kSiteReward, s);
  hipLaunchKernelGGL(reward_stats, dim3(w.blocks), dim3(kRwThreads), 0, s, items, shaped, outcome, game_time, c,
                     part);
  hipLaunchKernelGGL(reward_finalize, dim3(1), dim3(kRwThreads), 0, s, w.blocks, part, stats, hp.eps, scale);
  hipLaunchKernelGGL(reward_apply, dim3(w.blocks), dim3(kRwThreads), 0, s, items, shaped, outcome, game_time, c,
                     scale, r);
  ktimer_end(kSiteReward, s);
  return check_launch("o5_reward_process");
}
