// Softmax weights of the top-k state composition (Sec. 5.4 Eq. smc-fusion;
// the multi-chunk injection of Fig. 1):
//
//   w_j = exp((s_j - m) / tau) / sum_i exp((s_i - m) / tau),  m = max_i s_i,
//
// formed in fp64 from the exact retrieval scores, the sum taken in rank
// order i = 0..k-1, and rounded once to fp32.  Every weight is a function of
// the k scores alone, computed the same way by whichever thread needs it, so
// the composition kernel and a scan that starts from a composed state get the
// same bits.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace precog {

struct SoftmaxDen {
  double mx;   // largest score
  double den;  // sum_i exp((s_i - mx) * inv_tau), rank order
};

__device__ __forceinline__ SoftmaxDen softmax_den(const double* s, int k, double inv_tau) {
  double mx = s[0];
  for (int i = 1; i < k; ++i) mx = fmax(mx, s[i]);
  double den = 0.0;
  for (int i = 0; i < k; ++i) den += exp((s[i] - mx) * inv_tau);
  return SoftmaxDen{mx, den};
}

__device__ __forceinline__ float softmax_weight(double sj, const SoftmaxDen& d, double inv_tau) {
  return static_cast<float>(exp((sj - d.mx) * inv_tau) / d.den);
}

}  // namespace precog
