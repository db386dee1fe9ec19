// Unit-selection head (appendix "Neural Network Architecture": the unit
// embeddings of the observation processing are carried beside the LSTM and
// used by the action heads to choose a unit to target).  One head scores its
// nk units against per-row embeddings E [N, nk, d]:
//
//   q = h Wq^T                  GEMM (M = N, N = d, K = H), fp32 out
//   z[n, u] = <q[n] + bq, E[n, u]>          unit_logits (block per row)
//   dq[n, j] = sum_u dz[n, u] E[n, u, j]    unit_dq (block per row)
//   dWq = dq^T h,  dbq = sum_n dq           GEMM, fixed-order sums
//   dh += dq Wq                             by the caller, as extra K of its
//                                           dz Wp product
//
// On the bf16 path the two products that read dq take it as a (hi, lo) pair
// of bf16 terms (relative error ~2^-16), in row layout (written into the
// caller's dz pair, beside dz) and transposed (K-contiguous over n) for dWq,
// as the loss does for dz.  E is read twice, once per direction: N nk d
// elements each way.
#include "gemm_plan.h"
#include "heads.h"
#include "reduce.h"

namespace o5 {

constexpr int kUnitT = 64;  // transpose tile

// 8 consecutive embedding values as fp32 (one 16-byte load for bf16).
__device__ __forceinline__ void load8(const uint16_t* p, float (&f)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    f[2 * k] = __uint_as_float(w[k] << 16);
    f[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float (&f)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
  f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
}

// Block per row n.  The row's embeddings E[n] are nk * C chunks of 8 values
// (C = d / 8, a power of two up to 64); thread t takes chunks t, t + 256,
// ..., so its chunk index within a unit, t % C, never changes, and the C
// chunks of one unit sit on C consecutive lanes of one wave.  Every load is
// 16 bytes and a wave reads 1 KB of the row at a time.

// z[n, u] = sum_j (q[n, j] + bq[j]) E[n, u, j]: per-chunk partial sums, then
// a butterfly over the unit's C lanes.
template <typename E>
__global__ void __launch_bounds__(256) unit_logits(int nk, int d, const float* __restrict__ q,
                                                   const float* __restrict__ bq, const E* __restrict__ emb,
                                                   float* __restrict__ z) {
  const int n = blockIdx.x;
  const int C = d >> 3;
  const int t = threadIdx.x;
  const int jc = t & (C - 1);
  float qv[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) qv[k] = q[static_cast<size_t>(n) * d + jc * 8 + k] + bq[jc * 8 + k];
  const E* row = emb + static_cast<size_t>(n) * nk * d;
  const int chunks = nk * C;
  for (int c0 = 0; c0 < chunks; c0 += 256) {  // uniform trip count: the shuffles need every lane
    const int c = c0 + t;
    float s = 0.0f;
    if (c < chunks) {
      float f[8];
      load8(row + static_cast<size_t>(c) * 8, f);
#pragma unroll
      for (int k = 0; k < 8; ++k) s += qv[k] * f[k];
    }
    for (int w = 1; w < C; w <<= 1) s += __shfl_xor(s, w, 64);
    if (c < chunks && jc == 0) z[static_cast<size_t>(n) * nk + c / C] = s;
  }
}

// dq[n, j] = sum_u dz[n, u] E[n, u, j]: each thread accumulates its fixed
// chunk over the units it visits, then the 256 / C threads of a chunk are
// summed in order through LDS.
template <typename E>
__global__ void __launch_bounds__(256) unit_dq(int nk, int d, const float* __restrict__ dz,
                                               const E* __restrict__ emb, float* __restrict__ dq) {
  __shared__ float red[256][9];
  const int n = blockIdx.x;
  const int C = d >> 3;
  const int t = threadIdx.x;
  const E* row = emb + static_cast<size_t>(n) * nk * d;
  const float* dzn = dz + static_cast<size_t>(n) * nk;
  const int chunks = nk * C;
  float acc[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  for (int c = t; c < chunks; c += 256) {
    float f[8];
    load8(row + static_cast<size_t>(c) * 8, f);
    const float g = dzn[c / C];
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] += g * f[k];
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) red[t][k] = acc[k];
  __syncthreads();
  for (int j = t; j < d; j += 256) {
    const int jc = j >> 3, k = j & 7;
    float v = 0.0f;
    for (int r = jc; r < 256; r += C) v += red[r][k];
    dq[static_cast<size_t>(n) * d + j] = v;
  }
}

// dq [N, d] fp32 -> hi = bf16(dq), lo = bf16(dq - hi) in row layout
// (columns col0 .. col0 + dp - 1 of rows of ld elements) and transposed
// [2 dp, ldT] (hi rows, then lo rows); padding zero.  One 64 x 64 tile per
// block through LDS.
__global__ void __launch_bounds__(256) unit_pack(int N, int d, int dp, int ldT, const float* __restrict__ dq,
                                                 uint16_t* __restrict__ hi, uint16_t* __restrict__ lo, int col0, int ld,
                                                 uint16_t* __restrict__ hT) {
  __shared__ uint16_t th[kUnitT][kUnitT + 2], tl[kUnitT][kUnitT + 2];
  const int j0 = blockIdx.x * kUnitT, n0 = blockIdx.y * kUnitT;
  const int c = threadIdx.x & 63, r0 = threadIdx.x >> 6;
  for (int r = r0; r < kUnitT; r += 4) {
    const int n = n0 + r, j = j0 + c;
    const float v = (n < N && j < d) ? dq[static_cast<size_t>(n) * d + j] : 0.0f;
    const uint16_t hb = f32_to_bf16_bits(v);
    const uint16_t lb = f32_to_bf16_bits(v - bf16_bits_to_f32(hb));
    if (n < N) {
      hi[static_cast<size_t>(n) * ld + col0 + j] = hb;
      lo[static_cast<size_t>(n) * ld + col0 + j] = lb;
    }
    th[r][c] = hb;
    tl[r][c] = lb;
  }
  __syncthreads();
  for (int r = r0; r < kUnitT; r += 4) {
    const int j = j0 + r, n = n0 + c;  // transposed: row j, column n
    if (n < ldT) {
      hT[static_cast<size_t>(j) * ldT + n] = th[c][r];
      hT[static_cast<size_t>(dp + j) * ldT + n] = tl[c][r];
    }
  }
}

int check_unit(const char* fn, const HeadsMeta& hm, const o5_unit_head* u, bool loss) {
  O5_CHECK(u->head >= 0 && u->head < hm.K, O5_E_ARG, "%s: unit head %d out of range (K=%d)", fn, u->head, hm.K);
  O5_CHECK(u->d >= 8 && u->d <= 512 && (u->d & (u->d - 1)) == 0, O5_E_SHAPE,
           "%s: unit embedding width d=%d must be a power of two in 8..512", fn, u->d);
  O5_PTR(u->Wq, "unit.Wq");
  O5_PTR(u->bq, "unit.bq");
  O5_PTR(u->E, "unit.E");
  if (loss) {
    O5_PTR(u->dWq, "unit.dWq");
    O5_PTR(u->dbq, "unit.dbq");
  }
  return O5_OK;
}

UnitWs unit_ws(o5_dtype dt, int N, int H, int nk, int d, bool loss) {
  UnitWs w{};
  const bool bf = dt == O5_BF16;
  w.d = d;
  w.dp = cdiv(d, kUnitT) * kUnitT;
  w.nk = nk;
  w.ldT = cdiv(N, kUnitT) * kUnitT;
  w.nchunks = cdiv(N, 64);
  w.wsplits = 1;
  size_t o = 0;
  w.q = o;
  o += align_up(static_cast<size_t>(N) * d * 4);
  w.zext = o;
  o += align_up(static_cast<size_t>(N) * nk * 4);
  if (loss) {
    w.dzext = o;
    o += align_up(static_cast<size_t>(N) * nk * 4);
    w.dq = o;
    o += align_up(static_cast<size_t>(N) * d * 4);
    w.dbpart = o;
    o += align_up(static_cast<size_t>(w.nchunks) * d * 4);
    if (bf) {
      // dWq over K = N, split so the grid has about 256 blocks
      w.wsplits = std::max(1, std::min(cdiv(256, cdiv(2 * w.dp, 256) * cdiv(H, 256)), cdiv(N, 64) / 8));
      w.dqT = o;
      o += align_up(static_cast<size_t>(2) * w.dp * w.ldT * 2);
      w.wpart = o;
      o += align_up(static_cast<size_t>(w.wsplits) * 2 * w.dp * H * 4);
    } else {
      w.wsplits = std::max(1, std::min(cdiv(512, cdiv(d, 64) * cdiv(H, 64)), cdiv(N, 16) / 8));
      w.wpart = o;
      o += align_up(static_cast<size_t>(w.wsplits) * d * H * 4);
    }
  }
  w.total = o;
  return w;
}

void unit_forward(o5_dtype dt, int N, int H, int nk, const o5_unit_head& u, const void* h, char* ws, const UnitWs& w,
                  hipStream_t s) {
  float* q = reinterpret_cast<float*>(ws + w.q);
  float* zext = reinterpret_cast<float*>(ws + w.zext);
  const int d = w.d;
  GemmPlan plan = plan_gemm(dt == O5_BF16, N, d, H);
  plan.splits = 1;
  const dim3 grid(N);
  if (dt == O5_BF16) {
    KRows2<uint16_t> al{static_cast<const uint16_t*>(h), nullptr, nullptr, H, 0, H, H, N};
    KRows2<uint16_t> bl{static_cast<const uint16_t*>(u.Wq), nullptr, nullptr, H, 0, H, H, d};
    run_gemm(plan, al, bl, EpiStoreF32{q, d, 0}, N, d, H, s);
    hipLaunchKernelGGL(unit_logits<uint16_t>, grid, dim3(256), 0, s, nk, d, q, u.bq,
                       static_cast<const uint16_t*>(u.E), zext);
  } else {
    KRows2<float> al{static_cast<const float*>(h), nullptr, nullptr, H, 0, H, H, N};
    KRows2<float> bl{static_cast<const float*>(u.Wq), nullptr, nullptr, H, 0, H, H, d};
    run_gemm(plan, al, bl, EpiStoreF32{q, d, 0}, N, d, H, s);
    hipLaunchKernelGGL(unit_logits<float>, grid, dim3(256), 0, s, nk, d, q, u.bq, static_cast<const float*>(u.E),
                       zext);
  }
}

void unit_grad(o5_dtype dt, int N, int H, int nk, const o5_unit_head& u, const void* h, char* ws, const UnitWs& w,
               uint16_t* dzhi, uint16_t* dzlo, int col0, int ld, hipStream_t s) {
  const float* dzext = reinterpret_cast<const float*>(ws + w.dzext);
  float* dq = reinterpret_cast<float*>(ws + w.dq);
  float* dbpart = reinterpret_cast<float*>(ws + w.dbpart);
  float* wpart = reinterpret_cast<float*>(ws + w.wpart);
  const int d = w.d, dp = w.dp;
  if (dt == O5_BF16)
    hipLaunchKernelGGL(unit_dq<uint16_t>, dim3(N), dim3(256), 0, s, nk, d, dzext, static_cast<const uint16_t*>(u.E),
                       dq);
  else
    hipLaunchKernelGGL(unit_dq<float>, dim3(N), dim3(256), 0, s, nk, d, dzext, static_cast<const float*>(u.E), dq);
  // dbq: fixed-order column sums of dq (chunks of 64 rows, then a block per
  // column over the chunk sums: dq is narrow, so a thread per column alone
  // would walk too many rows)
  hipLaunchKernelGGL(colsum_chunks, dim3(cdiv(d, 256), w.nchunks), dim3(256), 0, s, N, d, 64, dq, dbpart);
  hipLaunchKernelGGL(colsum_tree, dim3(d), dim3(256), 0, s, w.nchunks, d, dbpart, u.dbq);
  if (dt == O5_BF16) {
    uint16_t* dqT = reinterpret_cast<uint16_t*>(ws + w.dqT);
    hipLaunchKernelGGL(unit_pack, dim3(dp / kUnitT, w.ldT / kUnitT), dim3(256), 0, s, N, d, dp, w.ldT, dq, dzhi, dzlo,
                       col0, ld, dqT);
    // [dWq_hi ; dWq_lo] = [hi ; lo]^T-rows . h  (M = 2 dp, N = H, K = N), split over K
    KRows2<uint16_t> al{dqT, nullptr, nullptr, w.ldT, 0, N, N, 2 * dp};
    ICols2<uint16_t> bl{static_cast<const uint16_t*>(h), nullptr, nullptr, nullptr, H, 0, H, H, N, 0};
    launch_gemm_bf16_dma(al, bl, EpiStoreF32{wpart, H, static_cast<size_t>(2) * dp * H}, 2 * dp, H, N, w.wsplits, s);
    hipLaunchKernelGGL(sum_hilo_splits, dim3(cdiv(static_cast<long long>(d) * H, 256)), dim3(256), 0, s, w.wsplits, d,
                       dp, H, wpart, u.dWq);
  } else {
    // dWq = dq^T h, split over rows, fixed-order sum
    ICols2<float> al{dq, nullptr, nullptr, nullptr, d, 0, d, d, N, 0};
    ICols2<float> bl{static_cast<const float*>(h), nullptr, nullptr, nullptr, H, 0, H, H, N, 0};
    launch_gemm_f32(al, bl, EpiStoreF32{wpart, H, static_cast<size_t>(d) * H}, d, H, N, w.wsplits, s);
    hipLaunchKernelGGL(colsum_rows, dim3(cdiv(static_cast<long long>(d) * H, 256)), dim3(256), 0, s, w.wsplits, d * H,
                       wpart, u.dWq);
  }
}

}  // namespace o5
