// The policy function (paper §3.1: the policy maps each head's Selected
// Aggregation Score and the inference state to its sparsity-ratio scheme; §4:
// Func 0 / Func 1 budgets, the dense warm-up, the policy study's budgets
// negatively correlated with the score): the per-head budgets on the device, and
// the warm-up schedule and the static/dynamic budget split on the host.
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

// Per-head Top-P mass: e_k = (n (1 - tau)) a_k / S with a_k = max(AS(h_k), 0) and
// S = a_0 + ... + a_{n-1} added in list order by one thread; tau_k = 1 - e_k
// (S = 0: tau for every head).
__global__ void __launch_bounds__(kThreads)
    policy_tau_kernel(const double* __restrict__ as_best, HeadMap hm, double tau,
                      double* __restrict__ tau_out) {
  __shared__ double s_sum;
  const int n = hm.n;
  auto score = [&](int k) { return fmax(as_best[hm.ident ? k : hm.h[k]], 0.0); };
  if (threadIdx.x == 0) {
    double S = 0.0;
    for (int k = 0; k < n; ++k) S += score(k);
    s_sum = S;
  }
  __syncthreads();
  const double S = s_sum;
  const double total = double(n) * (1.0 - tau);
  for (int k = threadIdx.x; k < n; k += kThreads)
    tau_out[k] = S > 0.0 ? 1.0 - total * score(k) / S : tau;
}

}  // namespace

// Warm-up: the first ceil(0.3 n) steps (text-to-video) or ceil(n / 4) steps
// (image-to-video) of n, in integer arithmetic; Turbo: the first step only.
bool policy_dense(int step, int n_steps, int task, bool turbo) {
  if (turbo) return step < 1;
  const int warm = task == 0 ? (3 * n_steps + 9) / 10 : (n_steps + 3) / 4;
  return step < warm;
}

// Static/dynamic split of a per-row budget: the static share (Func 0: 1 of 31
// blocks, the 30:1 dynamic:static budget; Func 1: 1 of 5, ~80% dynamic) rounded
// half up in integers, then the largest window of the radius ladder that fits it.
void policy_split(int k_total, int func, int window[3], int* window_blocks, int* k_dyn) {
  // (t, y, x) radii of growing windows: 1, 3, 9, 27, 45, 75, 125 blocks
  static const int kLadder[][3] = {{0, 0, 0}, {0, 0, 1}, {0, 1, 1}, {1, 1, 1},
                                   {1, 1, 2}, {1, 2, 2}, {2, 2, 2}};
  const int k_static = func == 0 ? (2 * k_total + 31) / 62 : (2 * k_total + 5) / 10;
  int best = -1;
  for (int w = 0; w < int(sizeof(kLadder) / sizeof(kLadder[0])); ++w) {
    const int size = (2 * kLadder[w][0] + 1) * (2 * kLadder[w][1] + 1) * (2 * kLadder[w][2] + 1);
    if (size <= k_static) best = w;
  }
  if (best < 0) {
    window[0] = window[1] = window[2] = -1;
    *window_blocks = 0;
    *k_dyn = k_total;
    return;
  }
  int size = 1;
  for (int a = 0; a < 3; ++a) {
    window[a] = kLadder[best][a];
    size *= 2 * kLadder[best][a] + 1;
  }
  *window_blocks = size;
  *k_dyn = k_total - size;
}

hipError_t launch_policy_tau(const double* as_best, const HeadMap& hm, double tau,
                             double* tau_out, hipStream_t s) {
  policy_tau_kernel<<<1, kThreads, 0, s>>>(as_best, hm, tau, tau_out);
  return hipGetLastError();
}

hipError_t launch_policy_budgets(const double* as_best, const HeadMap& hm, int k_dyn, int NB,
                                 int* k_out, hipStream_t s) {
  policy_budgets_kernel<<<1, kThreads, 0, s>>>(as_best, hm, k_dyn, NB, k_out);
  return hipGetLastError();
}

}  // namespace spade
