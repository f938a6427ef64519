// Group advantage of App. D.2, shared by rb_group_advantage and rb_push.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace rbp {

// A_i = (r_i - mean) / (std + eps) over the rewards reward[lo .. hi) of one
// group, std with ddof = 0 or 1; A = 0 for every member when the rewards are
// all equal or n - ddof <= 0.  out(i, A_i) receives member i's value.  Fixed
// summation order (one thread per group).
template <class Out>
__device__ __forceinline__ void group_advantage(const float* __restrict__ reward, int32_t lo,
                                                int32_t hi, int32_t ddof, float eps, Out out) {
  const int32_t n = hi - lo;
  if (n <= 0) return;
  float sum = 0.0f;
  for (int32_t i = lo; i < hi; ++i) sum += reward[i];
  const float mean = sum / (float)n;
  float ss = 0.0f;
  for (int32_t i = lo; i < hi; ++i) {
    const float dv = reward[i] - mean;
    ss = fmaf(dv, dv, ss);
  }
  if (ss == 0.0f || n - ddof <= 0) {
    for (int32_t i = lo; i < hi; ++i) out(i, 0.0f);
    return;
  }
  const float sd = __fsqrt_rn(ss / (float)(n - ddof));
  const float denom = sd + eps;
  for (int32_t i = lo; i < hi; ++i) out(i, (reward[i] - mean) / denom);
}

}  // namespace rbp
