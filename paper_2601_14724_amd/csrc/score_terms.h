// Per-candidate terms of the attention score shared by the kernels that
// produce W (attention.hip) and the kernels that score and select
// (select.hip).  Device code only.
#pragma once
#include "hermes_internal.h"

namespace hermes {

// alpha_i W_i (Sec. 3.1): W_i divided by the number of the chunk's queries
// that can see candidate i (all C for cached rows, C - (i - T0) for the
// chunk's own row i under the causal mask) when mode is 0; W_i itself when
// mode is 1 (a guidance prompt, whose rows all see every candidate, or the
// plain sum).
__device__ __forceinline__ double mass_over_observers(float w, int i, int T0, int C, int mode) {
  if (mode != 0) return (double)w;
  const int n = i < T0 ? C : C - (i - T0);
  return (double)w / (double)n;
}

}  // namespace hermes
