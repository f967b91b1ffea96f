// Head-wise budgets of the policy function (paper §3.1: the policy maps each
// head's Selected Aggregation Score and the inference state to its sparsity-
// ratio scheme; §4 policy study: budget negatively correlated with the score).
//
// For the listed heads h_0..h_{n-1}: w_k = 1 / AS(h_k) (0 when AS <= 0),
// W = w_0 + ... + w_{n-1} added in list order by one thread, and
// k_k = clamp(floor(n k_dyn w_k / W + 1/2), 1, NB) (W = 0: clamp(k_dyn, 1, NB)).
// Every step is a correctly rounded fp64 operation in a fixed order, so the
// result does not depend on the launch.
#include "spade_internal.h"

namespace spade {
namespace {

constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads)
    policy_budgets_kernel(const double* __restrict__ as_best, HeadMap hm, int k_dyn, int NB,
                          int* __restrict__ k_out) {
  __shared__ double w_sum;
  const int n = hm.n;
  auto score = [&](int k) { return as_best[hm.ident ? k : hm.h[k]]; };
  if (threadIdx.x == 0) {
    double W = 0.0;
    for (int k = 0; k < n; ++k) {
      const double a = score(k);
      W += a > 0.0 ? 1.0 / a : 0.0;
    }
    w_sum = W;
  }
  __syncthreads();
  const double W = w_sum;
  const double total = double(n) * double(k_dyn);
  for (int k = threadIdx.x; k < n; k += kThreads) {
    int kk = k_dyn;
    if (W > 0.0) {
      const double a = score(k);
      const double w = a > 0.0 ? 1.0 / a : 0.0;
      const double x = floor(total * w / W + 0.5);
      kk = x > double(NB) ? NB : int(x);
    }
    k_out[k] = min(max(kk, 1), NB);
  }
}

}  // namespace

hipError_t launch_policy_budgets(const double* as_best, const HeadMap& hm, int k_dyn, int NB,
                                 int* k_out, hipStream_t s) {
  policy_budgets_kernel<<<1, kThreads, 0, s>>>(as_best, hm, k_dyn, NB, k_out);
  return hipGetLastError();
}

}  // namespace spade
