// Group advantage of App. D.2, shared by rb_group_advantage and rb_push.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace rbp {

// A_i = (r_i - mean) / (std + eps) over the rewards reward[lo .. hi) of one
// group, std with ddof = 0 or 1; A = 0 for every member when the rewards are
// all equal or n - ddof <= 0.  out(i, A_i) receives member i's value.  Fixed
// summation order (one thread per group).
//
// The mean, the spread and the quotient are formed in fp64 and only A is
// rounded to fp32.  fp32 inputs sum exactly in fp64 (a group is far shorter
// than 2^29 rewards of similar magnitude), so a group of equal rewards has a
// mean equal to each of them and deviations of exactly zero; an fp32 mean of
// rewards such as 0.7 is off by an ulp, which the eps of 1e-6 then turns
// into an advantage of order 0.1 instead of 0.  Equality is also decided
// directly on the inputs before any arithmetic.
template <class Out>
__device__ __forceinline__ void group_advantage(const float* __restrict__ reward, int32_t lo,
                                                int32_t hi, int32_t ddof, float eps, Out out) {
  const int32_t n = hi - lo;
  if (n <= 0) return;
  const float first = reward[lo];
  bool equal = true;
  double sum = 0.0;
  for (int32_t i = lo; i < hi; ++i) {
    const float r = reward[i];
    equal = equal && (r == first);
    sum += (double)r;
  }
  const double mean = sum / (double)n;
  double ss = 0.0;
  for (int32_t i = lo; i < hi; ++i) {
    const double dv = (double)reward[i] - mean;
    ss = fma(dv, dv, ss);
  }
  if (equal || ss == 0.0 || n - ddof <= 0) {
    for (int32_t i = lo; i < hi; ++i) out(i, 0.0f);
    return;
  }
  const double denom = sqrt(ss / (double)(n - ddof)) + (double)eps;
  for (int32_t i = lo; i < hi; ++i) out(i, (float)(((double)reward[i] - mean) / denom));
}

}  // namespace rbp
