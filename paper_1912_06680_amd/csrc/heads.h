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

}  // namespace o5
