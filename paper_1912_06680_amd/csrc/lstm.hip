// LSTM forward pass and truncated BPTT over one minibatch of 16-step samples
// (section "Training System": a single-layer 4096-unit forget-gate LSTM;
// subsection "Optimizing the Policy": truncated BPTT over 16 timesteps).
//
// Forward, for t = 0 .. T-1:
//   GEMM  P_t = [x_t | h~_{t-1}] . [W_x | W_h]^T          (M = B, N = 4H, K = D + H)
//   cell  a = P_t + b; (i, f, g, o); c_t = f c~ + i g; h_t = o tanh(c_t)
// The concatenated-K GEMM reads x_t and the previous hidden state directly,
// so no [T, B, 4H] input projection ever goes through HBM; the reset mask is
// applied to the hidden-state half of each A row as it is loaded.
//
// Backward, for t = T-1 .. 0:
//   GEMM  R = dG_{t+1} . W_h                               (M = B, N = H, K = 4H)
//   cell  dh = dh_heads[t] + (1 - reset[t+1]) R;  dG_t and the carried dc;
//         per-block column sums of dG_t for the bias gradient
// then once:
//   GEMM  [dW_x | dW_h] = dG^T . [x | h~_prev]             (M = 4H, N = D + H, K = T B)
//   GEMM  dx = dG . W_x                                     (M = T B, N = D, K = 4H), optional
//   db    = fixed-order sum of the per-block column sums.
//
// fp32 path: the FMA engine; bf16 path: the MFMA engine, with h, the saved
// gates and dG stored in bf16 and everything else in fp32.
#include "gemm_plan.h"
#include "reduce.h"

namespace o5 {

// ------------------------------------------------------- pointwise kernels

constexpr int kPwCols = 64;  // hidden units per block
constexpr int kPwRowGroups = 4;
constexpr int kPwRows = 32;  // batch rows per block (8 per row group)

// Forward cell for one step.  pre: [S][B][4H] partial GEMM sums.
template <typename E>
__global__ void __launch_bounds__(256) lstm_fwd_cell(int B, int H, int S, const float* __restrict__ pre,
                                                     const float* __restrict__ bias, const float* __restrict__ c_prev,
                                                     const uint8_t* __restrict__ reset_t, E* __restrict__ h_out,
                                                     float* __restrict__ c_out, E* __restrict__ gates_out) {
  const int j = blockIdx.x * kPwCols + (threadIdx.x & 63);
  const int rg = threadIdx.x >> 6;
  if (j >= H) return;
  const size_t G = 4 * static_cast<size_t>(H);
  const size_t sstride = static_cast<size_t>(B) * G;
  const float bi = bias[j], bf = bias[H + j], bg = bias[2 * H + j], bo = bias[3 * H + j];
  for (int r = rg; r < kPwRows; r += kPwRowGroups) {
    const int b = blockIdx.y * kPwRows + r;
    if (b >= B) break;
    const size_t row = static_cast<size_t>(b) * G;
    float ai = bi, af = bf, ag = bg, ao = bo;
    for (int s = 0; s < S; ++s) {
      const float* p = pre + s * sstride + row;
      ai += p[j];
      af += p[H + j];
      ag += p[2 * H + j];
      ao += p[3 * H + j];
    }
    const float keep = (reset_t && reset_t[b]) ? 0.0f : 1.0f;
    const size_t hj = static_cast<size_t>(b) * H + j;
    const float cp = keep * c_prev[hj];
    const float ig = sigmoid_f(ai), fg = sigmoid_f(af), gg = tanh_f(ag), og = sigmoid_f(ao);
    const float c = fg * cp + ig * gg;
    const float h = og * tanh_f(c);
    c_out[hj] = c;
    h_out[hj] = elem<E>::from_f32(h);
    if (gates_out) {
      E* gp = gates_out + row;
      gp[j] = elem<E>::from_f32(ig);
      gp[H + j] = elem<E>::from_f32(fg);
      gp[2 * H + j] = elem<E>::from_f32(gg);
      gp[3 * H + j] = elem<E>::from_f32(og);
    }
  }
}

// Four consecutive elements as float4 (fp32 or bf16 storage).
template <typename E> struct Vec4;
template <> struct Vec4<float> {
  __device__ __forceinline__ static float4 load(const float* p) { return *reinterpret_cast<const float4*>(p); }
  __device__ __forceinline__ static void store(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
};
template <> struct Vec4<uint16_t> {
  __device__ __forceinline__ static float4 load(const uint16_t* p) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xffff0000u));
  }
  __device__ __forceinline__ static void store(uint16_t* p, float4 v) {
    uint2 u;
    u.x = f32x2_to_bf16x2(v.x, v.y);
    u.y = f32x2_to_bf16x2(v.z, v.w);
    *reinterpret_cast<uint2*>(p) = u;
  }
};

__device__ __forceinline__ float4 f4(float a) { return make_float4(a, a, a, a); }

// The forward cell fused into the epilogue of the step's GEMM.  The GEMM's B
// tile is gate-gathered (256 columns = gates i, f, g, o of 64 hidden units),
// so a wave whose tile starts at column wn0 holds gate (column / 64) of unit
// (column % 64) for 128 rows.  In two passes of 128 rows the waves of one
// row half park their accumulators in LDS ([gate][row][unit], rows padded to
// 72 floats so the two half-waves of a store hit disjoint banks), then every
// thread reads the four gates of 4 consecutive units in each of its rows and
// finishes the cell: c, h and the saved gates go straight to HBM in 16- and
// 8-byte pieces and the pre-activations never do.  The bias and the previous
// cell state of both passes are requested before the last K tile's MFMAs
// (prefetch), so their latency hides behind them.  The epilogue is bound by
// vector instruction issue (the MFMA units idle meanwhile), hence the
// hardware bf16 rounding, the bias folded into the exponent's FMA and the
// 32-bit offsets.
template <typename E>
struct EpiLstmCell {
  static constexpr int kPad = 72;
  static constexpr int kTileSmem = 4 * 128 * kPad * 4;  // 144 KB
  static constexpr int kThreads = 512;                  // the block of both engines
  static constexpr int kRS = kThreads / 16;             // rows per sweep
  static constexpr int kNR = 128 / kRS;                 // sweeps per 128-row pass
  // (thread -> 4 consecutive hidden units, quad tid % 16, of rows tid / 16 +
  // kRS * i of each pass)
  // exp(x) = 2^(x log2 e): the activations take their exponent as one FMA
  // of the pre-activation with the bias scaled in prefetch (by -log2 e for
  // the sigmoids of i, f, o; by 2 log2 e for tanh of g)
  static constexpr float kL2E = 1.44269504088896341f;
  struct Pre {
    float4 b[4];          // scaled bias of gates i, f, g, o
    float4 cp[2][kNR];    // previous cell state
    int rs[2][kNR];       // the row's reset flag (its previous state counts as zero)
  };
  const float* bias;
  const float* c_prev;
  const uint8_t* reset_t;
  E* h_out;
  float* c_out;
  E* gates_out;
  int H;

  __device__ __forceinline__ void prefetch(Pre& pre, int m0, int n0, int tid, int M) const {
    const int j = (n0 >> 2) + 4 * (tid & 15);
    const int rr = tid >> 4;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float s = g == 2 ? 2.0f * kL2E : -kL2E;
      const float4 v = *reinterpret_cast<const float4*>(bias + g * H + j);
      pre.b[g] = make_float4(v.x * s, v.y * s, v.z * s, v.w * s);
    }
    // (the flag and the state are loaded independently; the flag selects
    // when the tile uses them, so no load waits for another)
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int i = 0; i < kNR; ++i) {
        const int bidx = m0 + p * 128 + rr + i * kRS;
        pre.cp[p][i] = make_float4(0.f, 0.f, 0.f, 0.f);
        pre.rs[p][i] = 0;
        if (bidx < M) {
          pre.cp[p][i] = *reinterpret_cast<const float4*>(c_prev + static_cast<size_t>(bidx) * H + j);
          if (reset_t) pre.rs[p][i] = reset_t[bidx];
        }
      }
  }

  template <int MB, int NB>
  __device__ __forceinline__ void tile(f32x16_t (&acc)[MB][NB], char* smem, int m0, int n0, int wm, int wn0, int lane,
                                       int tid, int M, const Pre& pre) const {
    static_assert(MB * 32 == 128, "expects 128-row wave tiles");
    float* lds = reinterpret_cast<float*>(smem);
    const int uq = tid & 15;
    const int rr = tid >> 4;
    const int j = (n0 >> 2) + 4 * uq;  // first hidden unit of the quad
    const uint32_t base_hc = static_cast<uint32_t>(m0 + rr) * H + j;
    const uint32_t base_g = static_cast<uint32_t>(m0 + rr) * 4 * H + j;
    const float4 bi = pre.b[0], bf = pre.b[1], bg = pre.b[2], bo = pre.b[3];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const float4* cp = pre.cp[p];
      if (wm == p) {
#pragma unroll
        for (int a = 0; a < MB; ++a)
#pragma unroll
          for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int row = a * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
              const int col = wn0 + b * 32 + (lane & 31);  // gate col / 64, unit col % 64
              lds[((col >> 6) * 128 + row) * kPad + (col & 63)] = acc[a][b][e];
            }
      }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < kNR; ++i) {
        const int row = rr + i * kRS;
        const int bidx = m0 + p * 128 + row;
        // element offsets (B * 4H < 2^31): h and c at bidx * H + j, the gates
        // at bidx * 4H + j; the row step is uniform
        const uint32_t ohc = base_hc + static_cast<uint32_t>((p * 128 + i * kRS) * H);
        const uint32_t ogt = base_g + static_cast<uint32_t>((p * 128 + i * kRS) * 4 * H);
        if (bidx < M) {
          const float4 ai = *reinterpret_cast<const float4*>(lds + (0 * 128 + row) * kPad + 4 * uq);
          const float4 af = *reinterpret_cast<const float4*>(lds + (1 * 128 + row) * kPad + 4 * uq);
          const float4 ag = *reinterpret_cast<const float4*>(lds + (2 * 128 + row) * kPad + 4 * uq);
          const float4 ao = *reinterpret_cast<const float4*>(lds + (3 * 128 + row) * kPad + 4 * uq);
          float4 ig, fg, gg, og, c, h;
          const float* pai = &ai.x; const float* paf = &af.x; const float* pag = &ag.x; const float* pao = &ao.x;
          const float* pbi = &bi.x; const float* pbf = &bf.x; const float* pbg = &bg.x; const float* pbo = &bo.x;
          const float4 cpi = pre.rs[p][i] ? make_float4(0.f, 0.f, 0.f, 0.f) : cp[i];
          const float* pcp = &cpi.x;
          float* pig = &ig.x; float* pfg = &fg.x; float* pgg = &gg.x; float* pog = &og.x;
          float* pc = &c.x; float* ph = &h.x;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            // sigma(a + b) = 1 / (1 + 2^(-(a + b) log2 e)), tanh(a + b) =
            // 1 - 2 / (1 + 2^(2 (a + b) log2 e)), as sigmoid_f and tanh_f
            pig[q] = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(fmaf(pai[q], -kL2E, pbi[q])));
            pfg[q] = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(fmaf(paf[q], -kL2E, pbf[q])));
            pgg[q] = 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(fmaf(pag[q], 2.0f * kL2E, pbg[q])));
            pog[q] = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(fmaf(pao[q], -kL2E, pbo[q])));
            pc[q] = pfg[q] * pcp[q] + pig[q] * pgg[q];
            ph[q] = pog[q] * tanh_f(pc[q]);
          }
          *reinterpret_cast<float4*>(c_out + ohc) = c;
          Vec4<E>::store(h_out + ohc, h);
          if (gates_out) {
            E* gp = gates_out + ogt;
            Vec4<E>::store(gp, ig);
            Vec4<E>::store(gp + H, fg);
            Vec4<E>::store(gp + 2 * H, gg);
            Vec4<E>::store(gp + 3 * H, og);
          }
        }
      }
      __syncthreads();
    }
  }
  __device__ __forceinline__ void operator()(int, int, float, int) const {}
};


__device__ const uint8_t kZeroFlag = 0;

// Backward cell for step t.  rec: [S][B][H] partial sums of dG_{t+1} W_h (or
// NULL at t = T-1).  dc: in = dc arriving at c_t, out = dc for c_{t-1}.
// Block: 64 hidden units x 32 rows; each thread owns 4 consecutive units of
// 2 rows (16-byte fp32 and 8-byte bf16 accesses) and the block writes one
// partial column sum of dG per gate and unit for the bias gradient.
template <typename E, int NS>
__global__ void __launch_bounds__(256) lstm_bwd_cell(
    int B, int H, int S, const float* __restrict__ rec, const uint8_t* __restrict__ reset_next,
    const float* __restrict__ dh_t, const float* __restrict__ dh_extra, const float* dc_in,
    float* dc_out, const E* __restrict__ gates_t, const float* __restrict__ c_t,
    const float* __restrict__ c_prev, const uint8_t* __restrict__ reset_t, E* __restrict__ dG_t,
    float* __restrict__ db_part, int db_accumulate, E* __restrict__ dGT, size_t ldt, int col0) {
  constexpr int kRowGroups = 16;
  static_assert(kPwRows == 2 * kRowGroups, "two adjacent rows per thread");
  __shared__ float red[kRowGroups][4][kPwCols];
  // dG of the block transposed, [gate * 64 + unit][row] (bf16 path only)
  __shared__ __attribute__((aligned(16))) uint16_t tq[sizeof(E) == 2 ? 4 * kPwCols : 1][kPwRows + 8];
  const int jq = threadIdx.x & 15;
  const int rg = threadIdx.x >> 4;
  const int j = blockIdx.x * kPwCols + jq * 4;
  const size_t G = 4 * static_cast<size_t>(H);
  const size_t sstride = static_cast<size_t>(B) * H;
  float4 sd[4] = {f4(0.f), f4(0.f), f4(0.f), f4(0.f)};
  // this thread's dG values (bf16 bits) of its two adjacent rows, for the
  // transposed copy; rows past B stay zero
  uint32_t tbits[2][16] = {};
  constexpr int R = kPwRows / kRowGroups;  // rows per thread
  // Every load of both rows is issued before any arithmetic, so a thread has
  // all of them in flight at once (rows past B read row 0 and are dropped).
  float4 dhv[R], exv[R], dcv[R], ctv[R], cpv[R], gin[R][4];
  float4 recv[R][NS];
  bool valid[R];
  uint32_t rnb[R], rtb[R];  // reset flags of the next and this step, read like the rest
  // absent reset flags read a zero byte, so no load sits behind a branch
  const uint8_t* rnp = reset_next ? reset_next : &kZeroFlag;
  const uint8_t* rtp = reset_t ? reset_t : &kZeroFlag;
  const int rns = reset_next ? 1 : 0, rts = reset_t ? 1 : 0;
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int b = blockIdx.y * kPwRows + rg * R + i;
    valid[i] = b < B;
    const int bc = valid[i] ? b : 0;
    const size_t hj = static_cast<size_t>(bc) * H + j;
    const size_t row = static_cast<size_t>(bc) * G;
    dhv[i] = dh_t ? Vec4<float>::load(dh_t + hj) : f4(0.f);
    exv[i] = dh_extra ? Vec4<float>::load(dh_extra + hj) : f4(0.f);
#pragma unroll
    for (int q = 0; q < NS; ++q) recv[i][q] = (rec && q < S) ? Vec4<float>::load(rec + q * sstride + hj) : f4(0.f);
    rnb[i] = rnp[bc * rns];
    rtb[i] = rtp[bc * rts];
    dcv[i] = dc_in ? Vec4<float>::load(dc_in + hj) : f4(0.f);
#pragma unroll
    for (int g = 0; g < 4; ++g) gin[i][g] = Vec4<E>::load(gates_t + row + g * H + j);
    ctv[i] = Vec4<float>::load(c_t + hj);
    cpv[i] = Vec4<float>::load(c_prev + hj);
  }
#pragma unroll
  for (int i = 0; i < R; ++i) {
    if (!valid[i]) continue;
    const int b = blockIdx.y * kPwRows + rg * R + i;
    const size_t hj = static_cast<size_t>(b) * H + j;
    const size_t row = static_cast<size_t>(b) * G;
    float4 dh = dhv[i];
    if (dh_extra) dh = make_float4(dh.x + exv[i].x, dh.y + exv[i].y, dh.z + exv[i].z, dh.w + exv[i].w);
    if (rec) {
      // the split partial sums in their fixed order
      float4 acc = recv[i][0];
#pragma unroll
      for (int q = 1; q < NS; ++q)
        if (q < S) acc = make_float4(acc.x + recv[i][q].x, acc.y + recv[i][q].y, acc.z + recv[i][q].z,
                                     acc.w + recv[i][q].w);
      const float k = rnb[i] ? 0.0f : 1.0f;
      dh = make_float4(dh.x + k * acc.x, dh.y + k * acc.y, dh.z + k * acc.z, dh.w + k * acc.w);
    }
    const float4 dcin = dcv[i];
    const float4 ig = gin[i][0];
    const float4 fg = gin[i][1];
    const float4 gg = gin[i][2];
    const float4 og = gin[i][3];
    const float4 ct = ctv[i];
    const float4 cpr = cpv[i];
    const float keepf = rtb[i] ? 0.0f : 1.0f;
    const float* dhp = &dh.x;
    const float* dcp = &dcin.x;
    const float* ip = &ig.x;
    const float* fp = &fg.x;
    const float* gp = &gg.x;
    const float* op = &og.x;
    const float* cp_ = &ct.x;
    const float* pp = &cpr.x;
    float4 dco, dai, daf, dag, dao;
    float* dcop = &dco.x;
    float* aip = &dai.x;
    float* afp = &daf.x;
    float* agp = &dag.x;
    float* aop = &dao.x;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float tc = tanh_f(cp_[q]);
      const float cprev = keepf * pp[q];
      const float dc = dcp[q] + dhp[q] * op[q] * (1.0f - tc * tc);
      aip[q] = dc * gp[q] * ip[q] * (1.0f - ip[q]);
      afp[q] = dc * cprev * fp[q] * (1.0f - fp[q]);
      agp[q] = dc * ip[q] * (1.0f - gp[q] * gp[q]);
      aop[q] = dhp[q] * tc * op[q] * (1.0f - op[q]);
      dcop[q] = keepf * dc * fp[q];
    }
    Vec4<float>::store(dc_out + hj, dco);
    Vec4<E>::store(dG_t + row + j, dai);
    Vec4<E>::store(dG_t + row + H + j, daf);
    Vec4<E>::store(dG_t + row + 2 * H + j, dag);
    Vec4<E>::store(dG_t + row + 3 * H + j, dao);
    if constexpr (sizeof(E) == 2) {
      const float* gv[4] = {&dai.x, &daf.x, &dag.x, &dao.x};
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int q = 0; q < 4; ++q) tbits[i][g * 4 + q] = f32_to_bf16_bits(gv[g][q]);
    }
    sd[0] = make_float4(sd[0].x + dai.x, sd[0].y + dai.y, sd[0].z + dai.z, sd[0].w + dai.w);
    sd[1] = make_float4(sd[1].x + daf.x, sd[1].y + daf.y, sd[1].z + daf.z, sd[1].w + daf.w);
    sd[2] = make_float4(sd[2].x + dag.x, sd[2].y + dag.y, sd[2].z + dag.z, sd[2].w + dag.w);
    sd[3] = make_float4(sd[3].x + dao.x, sd[3].y + dao.y, sd[3].z + dao.z, sd[3].w + dao.w);
  }
  if constexpr (sizeof(E) == 2) {
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<uint32_t*>(&tq[g * kPwCols + jq * 4 + q][2 * rg]) =
            tbits[0][g * 4 + q] | (tbits[1][g * 4 + q] << 16);
  }
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    red[rg][g][jq * 4 + 0] = sd[g].x;
    red[rg][g][jq * 4 + 1] = sd[g].y;
    red[rg][g][jq * 4 + 2] = sd[g].z;
    red[rg][g][jq * 4 + 3] = sd[g].w;
  }
  __syncthreads();
  {
    const int g = threadIdx.x >> 6, jl = threadIdx.x & 63;
    float sum = 0.0f;
#pragma unroll
    for (int q = 0; q < kRowGroups; ++q) sum += red[q][g][jl];
    float* d = db_part + static_cast<size_t>(blockIdx.y) * G + g * H + blockIdx.x * kPwCols + jl;
    *d = db_accumulate ? *d + sum : sum;  // the same block owns this entry at every step
  }
  if constexpr (sizeof(E) == 2) {
    if (dGT) {
      // 256 rows (gate, unit) x kPwRows columns: 4 chunks of 8 rows each
      const int c = threadIdx.x & 3;
      for (int u = threadIdx.x >> 2; u < 4 * kPwCols; u += 64) {
        const int g = u / kPwCols, jl = u % kPwCols;
        const uint4 v = *reinterpret_cast<const uint4*>(&tq[u][8 * c]);
        *reinterpret_cast<uint4*>(dGT + (static_cast<size_t>(g) * H + blockIdx.x * kPwCols + jl) * ldt + col0 +
                                  blockIdx.y * kPwRows + 8 * c) = v;
      }
    }
  }
}

// Transposed, time-padded operand for the weight-gradient GEMM.  Column
// k = t * Bp + b of dst (Bp = B rounded up to 64) holds source row t * B + b;
// columns with b >= B are zero.  Source row r is s0[r] for r < split, else
// s1[r - split], and zero where mask[r] is set.  So dst row c is column c of
// [x] (split = T*B) or of the masked previous hidden state h~ (s0 = h0, s1 =
// h, split = B, mask = reset).  Each wave moves 64 source rows x 64 columns
// with no LDS: lane (rb, cb) loads the 8 x 8 block of rows 8 rb .. + 7,
// columns 8 cb .. + 7 (eight 16-byte loads in flight), transposes it in
// registers and stores 8 rows of 16 bytes, so every load and store
// instruction of a wave covers whole 128-byte lines.  A block is 4 waves
// side by side in c; the source row tiles stride by gridDim.y.  Requires C
// and Bp multiples of 64.
template <typename E>
__global__ void __launch_bounds__(256) transpose_rows(int T, int B, int Bp, int C, const E* __restrict__ s0,
                                                      const E* __restrict__ s1, int split, int lds,
                                                      const uint8_t* __restrict__ mask, E* __restrict__ dst,
                                                      size_t ldd) {
  static_assert(sizeof(E) == 2, "bf16 only");
  const int lane = threadIdx.x & 63;
  const int c0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * 64;
  if (c0 >= C) return;  // a whole wave; the kernel has no barrier
  const int rb = lane >> 3, cb = lane & 7;
  const int c = c0 + 8 * cb;
  const int nkt = static_cast<int>((static_cast<long long>(T) * Bp) / 64);
  for (int kt = blockIdx.y; kt < nkt; kt += gridDim.y) {
    const int k0 = kt * 64;
    const int t = k0 / Bp;  // one step per 64-row tile (Bp is a multiple of 64)
    const int b0 = k0 - t * Bp + 8 * rb;
    uint4 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      v[i] = make_uint4(0, 0, 0, 0);
      const int b = b0 + i;
      if (b < B) {
        const int r = t * B + b;
        if (!(mask && mask[r])) {
          const E* src = r < split ? s0 + static_cast<size_t>(r) * lds : s1 + static_cast<size_t>(r - split) * lds;
          v[i] = *reinterpret_cast<const uint4*>(src + c);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      // column c + j: 16-bit half (j & 1) of word j / 2 of each of the 8 rows
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t lo = (&v[2 * e].x)[j >> 1], hi = (&v[2 * e + 1].x)[j >> 1];
        w[e] = (j & 1) ? (lo >> 16) | (hi & 0xffff0000u) : (lo & 0xffffu) | (hi << 16);
      }
      *reinterpret_cast<uint4*>(dst + static_cast<size_t>(c + j) * ldd + k0 + 8 * rb) =
          make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// B rounded up to 64, the time padding of the weight gradient's K: column
// t * Bp + b of [x | h~]^T holds sample b of step t (zero for b >= B).
static inline int time_pad(int B) { return cdiv(B, 64) * 64; }

// Grid of transpose_rows for C columns and `rows` source rows.
static inline dim3 transpose_grid(int C, long long rows) {
  return dim3(cdiv(C, 256), static_cast<unsigned>(std::min<long long>((rows + 63) / 64, 65535)));
}

// ---------------------------------------------------------------- layouts

struct FwdWs {
  size_t pre, h0e, total;
  GemmPlan plan;
};

static FwdWs fwd_ws(o5_dtype dt, int T, int B, int D, int H) {
  (void)T;
  FwdWs w;
  w.plan = plan_gemm(dt == O5_BF16, B, 4 * H, D + H);
  size_t o = 0;
  w.pre = o;
  o += align_up(static_cast<size_t>(w.plan.splits) * B * 4 * H * sizeof(float));
  w.h0e = o;
  o += align_up(static_cast<size_t>(B) * H * dtype_size(dt));
  w.total = o;
  return w;
}

struct BwdWs {
  size_t dG, dc, rec, h0e, dbpart, dGT, XHT, WhT, total;
  int nbc;
  int Bp;       // B rounded up to the cell's row block (bf16 path: time-padded K of dW)
  size_t ldt;   // T * Bp, the leading dimension of dGT and XHT
  GemmPlan plan_dh, plan_dw, plan_dx;
};

static BwdWs bwd_ws(o5_dtype dt, int T, int B, int D, int H) {
  BwdWs w;
  const bool bf = dt == O5_BF16;
  w.Bp = time_pad(B);
  w.nbc = w.Bp / kPwRows;  // cell row blocks; those past B only write zeros
  w.ldt = static_cast<size_t>(T) * w.Bp;
  w.plan_dh = plan_gemm(bf, B, H, 4 * H);
  w.plan_dw = plan_gemm(bf, 4 * H, D + H, bf ? static_cast<int>(w.ldt) : T * B);
  w.plan_dw.splits = 1;  // dW is written directly (M x N tiles are plentiful)
  w.plan_dx = plan_gemm(bf, T * B, D, 4 * H);
  w.plan_dx.splits = 1;
  size_t o = 0;
  w.dG = o;
  o += align_up(static_cast<size_t>(T) * B * 4 * H * dtype_size(dt));
  w.dc = o;
  o += align_up(static_cast<size_t>(B) * H * sizeof(float));
  w.rec = o;
  o += align_up(static_cast<size_t>(w.plan_dh.splits) * B * H * sizeof(float));
  w.h0e = o;
  o += align_up(static_cast<size_t>(B) * H * dtype_size(dt));
  w.dbpart = o;
  o += align_up(static_cast<size_t>(w.nbc) * 4 * H * sizeof(float));
  w.dGT = w.XHT = w.WhT = o;
  if (bf) {
    // K-contiguous operands for the MFMA engine: dG^T, [x | h~]^T, W_h^T
    w.dGT = o;
    o += align_up(static_cast<size_t>(4) * H * w.ldt * sizeof(uint16_t));
    w.XHT = o;
    o += align_up(static_cast<size_t>(D + H) * w.ldt * sizeof(uint16_t));
    w.WhT = o;
    o += align_up(static_cast<size_t>(H) * 4 * H * sizeof(uint16_t));
  }
  w.total = o;
  return w;
}

constexpr int kMaxLstmB = 32767 * 64;

static int check_dims(const char* fn, o5_dtype dt, int T, int B, int D, int H) {
  O5_CHECK(dt == O5_F32 || dt == O5_BF16, O5_E_DTYPE, "%s: unknown dtype %d", fn, static_cast<int>(dt));
  O5_CHECK(T >= 1 && B >= 1, O5_E_SHAPE, "%s: T=%d and B=%d must be >= 1", fn, T, B);
  // the cell kernels' grids give a block of 32 rows to each y index (< 65535
  // after B is padded to 64)
  O5_CHECK(B <= kMaxLstmB, O5_E_SHAPE, "%s: B=%d exceeds %d", fn, B, kMaxLstmB);
  O5_CHECK(D >= 64 && H >= 64 && D % 64 == 0 && H % 64 == 0 && D <= 65536 && H <= 65536, O5_E_SHAPE,
           "%s: D=%d and H=%d must be positive multiples of 64 (<= 65536)", fn, D, H);
  O5_CHECK(static_cast<long long>(T) * B < (1ll << 31) && static_cast<long long>(T) * B * 4 * H < (1ll << 31) &&
               static_cast<long long>(T) * B * D < (1ll << 31),
           O5_E_SHAPE, "%s: T*B*4H and T*B*D must stay below 2^31", fn);
  return O5_OK;
}

// ------------------------------------------------------------- forward

template <typename E>
static int lstm_fwd_impl(int T, int B, int D, int H, const E* x, const E* Wx, const E* Wh, const float* bias,
                         const float* h0, const float* c0, const uint8_t* reset, E* h, float* c, E* gates, char* ws,
                         const FwdWs& w, hipStream_t s) {
  const size_t BH = static_cast<size_t>(B) * H;
  float* pre = reinterpret_cast<float*>(ws + w.pre);
  const E* h0e;
  if constexpr (sizeof(E) == 2) {
    E* tmp = reinterpret_cast<E*>(ws + w.h0e);
    const int st = o5_f32_to_bf16(BH, h0, reinterpret_cast<uint16_t*>(tmp), s);
    if (st != O5_OK) return st;
    h0e = tmp;
  } else {
    h0e = h0;
  }
  if constexpr (sizeof(E) == 2) {
    if (w.plan.tile == BfTile::kDma256 && w.plan.splits == 1) {
      // one launch per step: GEMM with the cell fused into its epilogue
      for (int t = 0; t < T; ++t) {
        const E* hprev = t == 0 ? h0e : h + (t - 1) * BH;
        const uint8_t* rt = reset ? reset + static_cast<size_t>(t) * B : nullptr;
        KRows2<E> al{x + static_cast<size_t>(t) * B * D, hprev, rt, D, H, D, D + H, B};
        KRows2<E> bl{Wx, Wh, nullptr, D, H, D, D + H, 4 * H};
        bl.gstride = H;
        const float* cprev = t == 0 ? c0 : c + (t - 1) * BH;
        E* gt = gates ? gates + static_cast<size_t>(t) * B * 4 * H : nullptr;
        EpiLstmCell<E> epi{bias, cprev, rt, h + t * BH, c + t * BH, gt, H};
        ktimer_begin(kSiteLstmFwdGemm, s);
        if (kk_fits(al) && kk_fits(bl))
          launch_gemm_kk(al, bl, epi, B, 4 * H, D + H, 1, s);
        else
          launch_gemm_bf16_dma(al, bl, epi, B, 4 * H, D + H, 1, s);
        ktimer_end(kSiteLstmFwdGemm, s);
      }
      return check_launch("o5_lstm_fwd");
    }
  }
  const dim3 pw_grid(cdiv(H, kPwCols), cdiv(B, kPwRows));
  for (int t = 0; t < T; ++t) {
    const E* hprev = t == 0 ? h0e : h + (t - 1) * BH;
    const uint8_t* rt = reset ? reset + static_cast<size_t>(t) * B : nullptr;
    KRows2<E> al{x + static_cast<size_t>(t) * B * D, hprev, rt, D, H, D, D + H, B};
    KRows2<E> bl{Wx, Wh, nullptr, D, H, D, D + H, 4 * H};
    EpiStoreF32 epi{pre, 4 * H, static_cast<size_t>(B) * 4 * H};
    ktimer_begin(kSiteLstmFwdGemm, s);
    run_gemm(w.plan, al, bl, epi, B, 4 * H, D + H, s);
    ktimer_end(kSiteLstmFwdGemm, s);
    const float* cprev = t == 0 ? c0 : c + (t - 1) * BH;
    E* gt = gates ? gates + static_cast<size_t>(t) * B * 4 * H : nullptr;
    ktimer_begin(kSiteLstmFwdCell, s);
    hipLaunchKernelGGL(lstm_fwd_cell<E>, pw_grid, dim3(256), 0, s, B, H, w.plan.splits, pre, bias, cprev, rt,
                       h + t * BH, c + t * BH, gt);
    ktimer_end(kSiteLstmFwdCell, s);
  }
  return check_launch("o5_lstm_fwd");
}

// ------------------------------------------------------------ backward

template <typename E>
static int lstm_bptt_impl(int T, int B, int D, int H, const E* x, const E* Wx, const E* Wh, const float* h0,
                          const float* c0, const uint8_t* reset, const E* h, const float* c, const E* gates,
                          const float* dh, const float* dhT, const float* dcT, float* dWx, float* dWh, float* db,
                          E* dx, char* ws, const BwdWs& w, hipStream_t s, const E* P = nullptr,
                          const E* Wf = nullptr, int ldp = 0) {
  // P, Wf (bf16 only): the heads' gradient in factored form, dh_t = P_t Wf^T
  // with P [T*B][ldp] and Wf [H][ldp], instead of dh
  constexpr bool kBf = sizeof(E) == 2;
  const size_t BH = static_cast<size_t>(B) * H;
  const size_t BG = static_cast<size_t>(B) * 4 * H;
  E* dG = reinterpret_cast<E*>(ws + w.dG);
  float* dc = reinterpret_cast<float*>(ws + w.dc);
  float* rec = reinterpret_cast<float*>(ws + w.rec);
  float* dbpart = reinterpret_cast<float*>(ws + w.dbpart);
  E* dGT = kBf ? reinterpret_cast<E*>(ws + w.dGT) : nullptr;
  E* XHT = kBf ? reinterpret_cast<E*>(ws + w.XHT) : nullptr;
  E* WhT = kBf ? reinterpret_cast<E*>(ws + w.WhT) : nullptr;
  const E* h0e;
  if constexpr (kBf) {
    E* tmp = reinterpret_cast<E*>(ws + w.h0e);
    const int st = o5_f32_to_bf16(BH, h0, reinterpret_cast<uint16_t*>(tmp), s);
    if (st != O5_OK) return st;
    h0e = tmp;
    // W_h^T [H][4H]: the recurrent GEMM's second operand, K-contiguous
    hipLaunchKernelGGL(transpose_rows<E>, transpose_grid(H, 4 * H), dim3(256), 0, s, 1, 4 * H, 4 * H, H, Wh,
                       Wh, 4 * H, H, nullptr, WhT, static_cast<size_t>(4 * H));
  } else {
    h0e = h0;
  }
  const dim3 pw_grid(cdiv(H, kPwCols), w.nbc);
  // the cell unrolls its loads of the recurrent GEMM's split partials up to NS
  auto cell = w.plan_dh.splits <= 2 ? lstm_bwd_cell<E, 2>
              : w.plan_dh.splits <= 8 ? lstm_bwd_cell<E, 8>
                                      : lstm_bwd_cell<E, 16>;
  const bool fact = P != nullptr;
  for (int t = T - 1; t >= 0; --t) {
    const float* recp = nullptr;
    int S = w.plan_dh.splits;  // partial sums the cell adds
    if (fact) {
      if constexpr (kBf) {
        // R = [P_t | dG_{t+1}] . [Wf | W_h^T]^T: the heads' dh_t plus, for the
        // rows whose state carried into step t + 1 (the reset mask zeroes the
        // second source's rows), dG_{t+1} W_h; the last step has the first
        // part only
        const int K = t < T - 1 ? ldp + 4 * H : ldp;
        const uint8_t* rn = (reset && t < T - 1) ? reset + static_cast<size_t>(t + 1) * B : nullptr;
        KRows2<E> al{P + static_cast<size_t>(t) * B * ldp, t < T - 1 ? dG + (t + 1) * BG : nullptr, rn, ldp,
                     t < T - 1 ? 4 * H : 0, ldp, K, B};
        KRows2<E> bl{Wf, t < T - 1 ? WhT : nullptr, nullptr, ldp, t < T - 1 ? 4 * H : 0, ldp, K, H};
        EpiStoreF32 epi{rec, H, BH};
        GemmPlan plan = w.plan_dh;
        if (t == T - 1) plan.splits = 1;
        S = plan.splits;
        ktimer_begin(kSiteLstmDhGemm, s);
        run_gemm(plan, al, bl, epi, B, H, K, s);
        ktimer_end(kSiteLstmDhGemm, s);
        recp = rec;
      }
    } else if (t < T - 1) {
      // R = dG_{t+1} . W_h :  A(i=b, k=n) = dG_{t+1}[b, n];  B(j, k=n) = W_h[n, j]
      KRows2<E> al{dG + (t + 1) * BG, nullptr, nullptr, 4 * H, 0, 4 * H, 4 * H, B};
      EpiStoreF32 epi{rec, H, BH};
      ktimer_begin(kSiteLstmDhGemm, s);
      if constexpr (kBf) {
        KRows2<E> bl{WhT, nullptr, nullptr, 4 * H, 0, 4 * H, 4 * H, H};
        run_gemm(w.plan_dh, al, bl, epi, B, H, 4 * H, s);
      } else {
        ICols2<E> bl{Wh, nullptr, nullptr, nullptr, H, 0, H, H, 4 * H, 0};
        run_gemm(w.plan_dh, al, bl, epi, B, H, 4 * H, s);
      }
      ktimer_end(kSiteLstmDhGemm, s);
      recp = rec;
    }
    const uint8_t* rt = reset ? reset + static_cast<size_t>(t) * B : nullptr;
    // (the factored path has applied the next step's reset inside its product)
    const uint8_t* rn = (reset && t < T - 1 && !fact) ? reset + static_cast<size_t>(t + 1) * B : nullptr;
    const float* dcin = t == T - 1 ? dcT : dc;
    const float* dhx = t == T - 1 ? dhT : nullptr;
    const float* cprev = t == 0 ? c0 : c + (t - 1) * BH;
    ktimer_begin(kSiteLstmBwdCell, s);
    hipLaunchKernelGGL(cell, pw_grid, dim3(256), 0, s, B, H, S, recp, rn, fact ? nullptr : dh + t * BH, dhx,
                       dcin, dc, gates + t * BG, c + t * BH, cprev, rt, dG + t * BG, dbpart, t < T - 1 ? 1 : 0, dGT,
                       w.ldt, t * w.Bp);
    ktimer_end(kSiteLstmBwdCell, s);
  }
  // [dW_x | dW_h] = dG^T . [x | h~_prev] over the T*B rows r = t*B + b
  {
    EpiStoreF32Split2 epi{dWx, dWh, D, H, D};
    if constexpr (kBf) {
      // both operands K-contiguous over the time-padded K = T * Bp
      const int K = static_cast<int>(w.ldt);
      const int ldt = static_cast<int>(w.ldt);
      hipLaunchKernelGGL(transpose_rows<E>, transpose_grid(D, K), dim3(256), 0, s, T, B, w.Bp, D, x, x, T * B, D,
                         nullptr, XHT, w.ldt);
      hipLaunchKernelGGL(transpose_rows<E>, transpose_grid(H, K), dim3(256), 0, s, T, B, w.Bp, H, h0e, h, B, H,
                         reset, XHT + static_cast<size_t>(D) * w.ldt, w.ldt);
      KRows2<E> al{dGT, nullptr, nullptr, ldt, 0, K, K, 4 * H};
      KRows2<E> bl{XHT, nullptr, nullptr, ldt, 0, K, K, D + H};
      ktimer_begin(kSiteLstmDwGemm, s);
      run_gemm(w.plan_dw, al, bl, epi, 4 * H, D + H, K, s);
      ktimer_end(kSiteLstmDwGemm, s);
    } else {
      const int R = T * B;
      ICols2<E> al{dG, nullptr, nullptr, nullptr, 4 * H, 0, 4 * H, 4 * H, R, 0};
      ICols2<E> bl{x, h0e, h, reset, D, H, D, D + H, R, B};
      ktimer_begin(kSiteLstmDwGemm, s);
      run_gemm(w.plan_dw, al, bl, epi, 4 * H, D + H, R, s);
      ktimer_end(kSiteLstmDwGemm, s);
    }
  }
  hipLaunchKernelGGL(colsum_rows4, dim3(cdiv(4 * H, 64)), dim3(256), 0, s, w.nbc, 4 * H, dbpart, db);
  if (dx) {
    // dx = dG . W_x :  A(i=r, k=n) = dG[r, n];  B(j=d, k=n) = W_x[n, d]
    const int R = T * B;
    KRows2<E> al{dG, nullptr, nullptr, 4 * H, 0, 4 * H, 4 * H, R};
    ICols2<E> bl{Wx, nullptr, nullptr, nullptr, D, 0, D, D, 4 * H, 0};
    EpiStoreElem<E> epi{dx, D};
    ktimer_begin(kSiteLstmDxGemm, s);
    run_gemm(w.plan_dx, al, bl, epi, R, D, 4 * H, s);
    ktimer_end(kSiteLstmDxGemm, s);
  }
  return check_launch("o5_lstm_bptt");
}

}  // namespace o5

using namespace o5;

extern "C" size_t o5_lstm_fwd_workspace_bytes(o5_dtype dt, int T, int B, int D, int H) {
  if (check_dims("o5_lstm_fwd_workspace_bytes", dt, T, B, D, H) != O5_OK) return 0;
  return fwd_ws(dt, T, B, D, H).total;
}

extern "C" int o5_lstm_fwd(o5_dtype dt, int T, int B, int D, int H, const void* x, const void* Wx, const void* Wh,
                           const float* b, const float* h0, const float* c0, const uint8_t* reset, void* h, float* c,
                           void* gates, void* ws, size_t ws_bytes, void* stream) {
  int st = check_dims("o5_lstm_fwd", dt, T, B, D, H);
  if (st != O5_OK) return st;
  O5_PTR(x, "x");
  O5_PTR(Wx, "Wx");
  O5_PTR(Wh, "Wh");
  O5_PTR(b, "b");
  O5_PTR(h0, "h0");
  O5_PTR(c0, "c0");
  O5_OPT_PTR(reset, "reset");
  O5_PTR(h, "h");
  O5_PTR(c, "c");
  O5_OPT_PTR(gates, "gates");
  const FwdWs w = fwd_ws(dt, T, B, D, H);
  O5_CHECK(ws != nullptr && ws_bytes >= w.total, O5_E_WORKSPACE, "o5_lstm_fwd: workspace needs %zu bytes, got %zu",
           w.total, ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "o5_lstm_fwd: ws is not 16-byte aligned");
  char* wsp = static_cast<char*>(ws);
  hipStream_t s = as_stream(stream);
  ktimer_begin(kSiteLstmFwdCall, s);
  const int rc =
      dt == O5_BF16
          ? lstm_fwd_impl<uint16_t>(T, B, D, H, static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(Wx),
                                    static_cast<const uint16_t*>(Wh), b, h0, c0, reset, static_cast<uint16_t*>(h), c,
                                    static_cast<uint16_t*>(gates), wsp, w, s)
          : lstm_fwd_impl<float>(T, B, D, H, static_cast<const float*>(x), static_cast<const float*>(Wx),
                                 static_cast<const float*>(Wh), b, h0, c0, reset, static_cast<float*>(h), c,
                                 static_cast<float*>(gates), wsp, w, s);
  ktimer_end(kSiteLstmFwdCall, s);
  return rc;
}

extern "C" size_t o5_lstm_bptt_workspace_bytes(o5_dtype dt, int T, int B, int D, int H) {
  if (check_dims("o5_lstm_bptt_workspace_bytes", dt, T, B, D, H) != O5_OK) return 0;
  return bwd_ws(dt, T, B, D, H).total;
}

// Validation shared by the two backward calls (all but the heads' gradient).
static int bptt_check(const char* fn, o5_dtype dt, int T, int B, int D, int H, const void* x, const void* Wx,
                      const void* Wh, const float* h0, const float* c0, const uint8_t* reset, const void* h,
                      const float* c, const void* gates, const float* dhT, const float* dcT, float* dWx, float* dWh,
                      float* db, void* dx, void* ws, size_t ws_bytes, BwdWs* w) {
  int st = check_dims(fn, dt, T, B, D, H);
  if (st != O5_OK) return st;
  O5_PTR_IN(fn, x, "x");
  O5_PTR_IN(fn, Wx, "Wx");
  O5_PTR_IN(fn, Wh, "Wh");
  O5_PTR_IN(fn, h0, "h0");
  O5_PTR_IN(fn, c0, "c0");
  O5_OPT_PTR_IN(fn, reset, "reset");
  O5_PTR_IN(fn, h, "h");
  O5_PTR_IN(fn, c, "c");
  O5_PTR_IN(fn, gates, "gates");
  O5_OPT_PTR_IN(fn, dhT, "dhT");
  O5_OPT_PTR_IN(fn, dcT, "dcT");
  O5_PTR_IN(fn, dWx, "dWx");
  O5_PTR_IN(fn, dWh, "dWh");
  O5_PTR_IN(fn, db, "db");
  O5_OPT_PTR_IN(fn, dx, "dx");
  *w = bwd_ws(dt, T, B, D, H);
  O5_CHECK(ws != nullptr && ws_bytes >= w->total, O5_E_WORKSPACE, "%s: workspace needs %zu bytes, got %zu", fn,
           w->total, ws ? ws_bytes : static_cast<size_t>(0));
  O5_CHECK(aligned16(ws), O5_E_ALIGN, "%s: ws is not 16-byte aligned", fn);
  return O5_OK;
}

extern "C" int o5_lstm_bptt(o5_dtype dt, int T, int B, int D, int H, const void* x, const void* Wx, const void* Wh,
                            const float* h0, const float* c0, const uint8_t* reset, const void* h, const float* c,
                            const void* gates, const float* dh, const float* dhT, const float* dcT, float* dWx,
                            float* dWh, float* db, void* dx, void* ws, size_t ws_bytes, void* stream) {
  BwdWs w;
  const int st = bptt_check("o5_lstm_bptt", dt, T, B, D, H, x, Wx, Wh, h0, c0, reset, h, c, gates, dhT, dcT, dWx,
                            dWh, db, dx, ws, ws_bytes, &w);
  if (st != O5_OK) return st;
  O5_PTR(dh, "dh");
  char* wsp = static_cast<char*>(ws);
  hipStream_t s = as_stream(stream);
  if (dt == O5_BF16)
    return lstm_bptt_impl<uint16_t>(T, B, D, H, static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(Wx),
                                    static_cast<const uint16_t*>(Wh), h0, c0, reset,
                                    static_cast<const uint16_t*>(h), c, static_cast<const uint16_t*>(gates), dh, dhT,
                                    dcT, dWx, dWh, db, static_cast<uint16_t*>(dx), wsp, w, s);
  return lstm_bptt_impl<float>(T, B, D, H, static_cast<const float*>(x), static_cast<const float*>(Wx),
                               static_cast<const float*>(Wh), h0, c0, reset, static_cast<const float*>(h), c,
                               static_cast<const float*>(gates), dh, dhT, dcT, dWx, dWh, db,
                               static_cast<float*>(dx), wsp, w, s);
}

extern "C" int o5_lstm_bptt_factored(o5_dtype dt, int T, int B, int D, int H, const void* x, const void* Wx,
                                     const void* Wh, const float* h0, const float* c0, const uint8_t* reset,
                                     const void* h, const float* c, const void* gates, const uint16_t* P,
                                     const uint16_t* W, int ld, const float* dhT, const float* dcT, float* dWx,
                                     float* dWh, float* db, void* dx, void* ws, size_t ws_bytes, void* stream) {
  O5_CHECK(dt == O5_BF16, O5_E_DTYPE, "o5_lstm_bptt_factored: the factored gradient is bf16 only (dt=%d)",
           static_cast<int>(dt));
  BwdWs w;
  const int st = bptt_check("o5_lstm_bptt_factored", dt, T, B, D, H, x, Wx, Wh, h0, c0, reset, h, c, gates, dhT,
                            dcT, dWx, dWh, db, dx, ws, ws_bytes, &w);
  if (st != O5_OK) return st;
  O5_CHECK(ld >= 64 && ld % 64 == 0 && ld <= 4096, O5_E_SHAPE,
           "o5_lstm_bptt_factored: ld=%d must be a multiple of 64 in 64..4096", ld);
  O5_PTR(P, "P");
  O5_PTR(W, "W");
  return lstm_bptt_impl<uint16_t>(T, B, D, H, static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(Wx),
                                  static_cast<const uint16_t*>(Wh), h0, c0, reset, static_cast<const uint16_t*>(h), c,
                                  static_cast<const uint16_t*>(gates), nullptr, dhT, dcT, dWx, dWh, db,
                                  static_cast<uint16_t*>(dx), static_cast<char*>(ws), w, as_stream(stream), P, W, ld);
}
