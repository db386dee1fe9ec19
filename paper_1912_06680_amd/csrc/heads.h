// Head layout shared by the loss and the sampler: K categorical heads whose
// logits occupy consecutive columns, followed by one value column.
#pragma once

#include "common.h"

namespace o5 {

constexpr int kMaxHeads = 8;
constexpr int kMaxA1 = 1024;

struct HeadsMeta {
  int K;
  int A;  // total logits; column A is the value
  int off[kMaxHeads + 1];
};

// Validates (dt, N, H, K, head_sizes) and fills hm.  Returns O5_OK or an
// O5_E_* code with the message set.
int check_heads(const char* fn, o5_dtype dt, int N, int H, int K, const int* head_sizes, HeadsMeta* hm);

// out[a, j] = sum over splits s of part[s, a, j] + part[s, A1p + a, j] (the
// hi and lo halves of a product taken on a (hi; lo) bf16 pair), fixed order.
static __global__ void __launch_bounds__(256) sum_hilo_splits(int S, int A1, int A1p, int H, const float* __restrict__ part,
                                                       float* __restrict__ out) {
  const size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= static_cast<size_t>(A1) * H) return;
  const size_t hs = static_cast<size_t>(A1p) * H;  // offset of the lo half
  float v = 0.0f;
  for (int s2 = 0; s2 < S; ++s2) {
    const float* p = part + static_cast<size_t>(s2) * 2 * hs;
    v += p[i] + p[hs + i];
  }
  out[i] = v;
}

// ------------------------------------------------- unit-selection head
// Head `unit->head` scored against per-row unit embeddings (o5_unit_head):
// q = h Wq^T + bq, logits <q[n], E[n, u]>.  Scratch of the loss and the
// sampler, laid out by unit_ws; unit_forward leaves the head's logits in
// zext [N, nk]; unit_grad takes their gradient dzext [N, nk] to dq, writes
// dWq and dbq, and (bf16) leaves dq as a (hi, lo) pair in columns col0 ..
// col0 + dp - 1 of the caller's dz pair (rows of ld elements), so that the
// caller's dz Wp product also forms dq Wq.  The fp32 path leaves dq at dq.

struct UnitWs {
  size_t q, zext, dzext, dq, dqT, wpart, dbpart, total;
  int d, dp, nk, ldT, wsplits, nchunks;
};

// Validates the head description (loss: with the gradient outputs).
int check_unit(const char* fn, const HeadsMeta& hm, const o5_unit_head* u, bool loss);
UnitWs unit_ws(o5_dtype dt, int N, int H, int nk, int d, bool loss);
void unit_forward(o5_dtype dt, int N, int H, int nk, const o5_unit_head& u, const void* h, char* ws, const UnitWs& w,
                  hipStream_t s);
void unit_grad(o5_dtype dt, int N, int H, int nk, const o5_unit_head& u, const void* h, char* ws, const UnitWs& w,
               uint16_t* dzhi, uint16_t* dzlo, int col0, int ld, hipStream_t s);

// ------------------------------------------------ rollout sampling
// The two halves of o5_policy_sample: argument validation (everything but
// the workspace; fills hm and the scratch bytes needed) and the enqueueing
// of its kernels with a scratch buffer of at least that size.
int policy_sample_check(const char* fn, o5_dtype dt, int B, int H, int K, const int* head_sizes, const void* h,
                        const void* Wp, const float* bp, const uint8_t* avail, const o5_unit_head* unit,
                        const int32_t* act, const float* logp, const float* value, HeadsMeta* hm, size_t* need);
int policy_sample_run(o5_dtype dt, int B, int H, const HeadsMeta& hm, const void* h, const void* Wp, const float* bp,
                      const uint8_t* avail, const o5_unit_head* unit, uint64_t seed, uint64_t counter, int32_t* act,
                      float* logp, float* value, char* ws, hipStream_t s);

}  // namespace o5
