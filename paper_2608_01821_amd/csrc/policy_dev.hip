// The closed-loop part of the allocation policy on the GPU (Sec. 4.2): after
// step t's commitment, the risk signals of every sample (mean confidence c̄
// over the positions still masked, prediction churn χ against step t-1) and
// the allocation of step t+1 (risk Eq. 7, envelope allocation Eq. 8, K-level
// quantisation Eq. 9).  Bit-identical to davet_step_stats followed by
// davet_policy_step on the host: the same float64 operations in the same
// order (a sequential sum over positions in index order), no contraction
// into fused multiply-adds, IEEE-rounded division.
//
// One wavefront per sample: the lanes stage each position's contribution to
// the sum in LDS with coalesced loads (its confidence as a double where the
// position is still masked, +0.0 elsewhere: the running sum starts at +0.0
// and x + 0.0 == x for every x it can take, so this is the masked-only sum
// bit for bit) and count the masked and changed positions with wavefront
// sums; lane 0 runs the ordered sum, branch-free so its LDS reads pipeline,
// and the policy arithmetic.  The outputs may live in pinned host memory (the
// schedule loop reads the next levels from there without a copy, and polls a
// completion stamp instead of a stream synchronisation).

#include "common.h"

namespace davet {
namespace {

struct PolArgs {
  double alpha[DAVET_MAX_SEQS];
  double lower[DAVET_MAX_SEQS];   // envelope bounds of step t+1, per sample
  double upper[DAVET_MAX_SEQS];
};

// One workgroup of 16 wavefronts; wavefront w serves samples w, w+16, ...
// When every sample is done, thread 0 publishes `stamp` to *done (if given)
// after a system-scope fence, so a host that polls *done in pinned memory
// sees the levels and budgets complete.
constexpr int POL_WAVES = 16;

__global__ void __launch_bounds__(64 * POL_WAVES)
policy_step_kernel(int n_seqs, int L, int K, const float* __restrict__ conf,
                   const int32_t* __restrict__ argmax,
                   const int32_t* __restrict__ argmax_prev,
                   const uint8_t* __restrict__ masked_after, PolArgs pa,
                   int32_t* level_out, double* budget_out, double* r_out,
                   double* cbar_out, double* churn_out, int32_t* done,
                   int32_t stamp) {
#pragma clang fp contract(off)
  __shared__ double s_term[POL_WAVES][DAVET_MAX_RESP];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int s = w; s < n_seqs; s += POL_WAVES) {
    const size_t o = (size_t)s * L;
    int n = 0, changed = 0;
    for (int i = lane; i < L; i += 64) {
      const bool m = masked_after[o + i] != 0;
      s_term[w][i] = m ? (double)conf[o + i] : 0.0;
      n += m;
      changed += m && argmax_prev && argmax[o + i] != argmax_prev[o + i];
    }
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) {
      n += __shfl_xor(n, d, 64);
      changed += __shfl_xor(changed, d, 64);
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    if (lane == 0) {
      double sum = 0.0;
#pragma unroll 16
      for (int i = 0; i < L; ++i) sum = sum + s_term[w][i];
      const double cbar = n ? sum / (double)n : 0.0;
      const double churn =
          (n && argmax_prev) ? (double)changed / (double)n : 0.0;
      // Eq. (7) with the signals of step t, for step t+1 > 1
      const double r = 1.0 - ((pa.alpha[s] * cbar) * (1.0 - churn));
      // Eq. (8)
      const double lo = pa.lower[s], up = pa.upper[s];
      const double b = lo + r * (up - lo);
      // Eq. (9): the thresholds j/K that b reaches
      int lv = 0;
      for (int j = 1; j < K; ++j)
        if ((double)j / (double)K <= b) ++lv;
      level_out[s] = lv;
      budget_out[s] = b;
      if (r_out) r_out[s] = r;
      if (cbar_out) cbar_out[s] = cbar;
      if (churn_out) churn_out[s] = churn;
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  }
  if (done) {
    __syncthreads();
    if (threadIdx.x == 0) {
      __threadfence_system();
      *reinterpret_cast<volatile int32_t*>(done) = stamp;
    }
  }
}

}  // namespace

int launch_policy_step(int n_seqs, int L, int K, const double* alpha,
                       const double* lower, const double* upper,
                       const float* conf, const int32_t* argmax,
                       const int32_t* argmax_prev, const uint8_t* masked_after,
                       int32_t* level_out, double* budget_out, double* r_out,
                       double* cbar_out, double* churn_out, int32_t* done,
                       int32_t stamp, hipStream_t s) {
  PolArgs pa{};
  for (int i = 0; i < n_seqs; ++i) {
    pa.alpha[i] = alpha[i];
    pa.lower[i] = lower[i];
    pa.upper[i] = upper[i];
  }
  hipLaunchKernelGGL(policy_step_kernel, dim3(1), dim3(64 * POL_WAVES), 0, s,
                     n_seqs, L, K, conf, argmax, argmax_prev, masked_after, pa,
                     level_out, budget_out, r_out, cbar_out, churn_out, done,
                     stamp);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

}  // namespace davet

extern "C" int davet_policy_step_device(
    int32_t n_seqs, int32_t L, int32_t t, int32_t T, const davet_policy* pols,
    const double* lower, const double* upper, const float* conf,
    const int32_t* argmax, const int32_t* argmax_prev,
    const uint8_t* masked_after, int32_t* level_out, double* budget_out,
    double* r_out, hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(pols && lower && upper && conf && argmax && masked_after &&
                      level_out && budget_out,
                  DAVET_EINVAL, "davet_policy_step_device: null argument");
  DAVET_CHECK_ARG(n_seqs >= 1 && n_seqs <= DAVET_MAX_SEQS, DAVET_ESHAPE,
                  "davet_policy_step_device: n_seqs out of range");
  DAVET_CHECK_ARG(L >= 1 && L <= DAVET_MAX_RESP, DAVET_ESHAPE,
                  "davet_policy_step_device: L out of range");
  DAVET_CHECK_ARG(t >= 1 && t < T, DAVET_EINVAL,
                  "davet_policy_step_device: t must be in [1, T)");
  DAVET_CHECK_ARG((t == 1) == (argmax_prev == nullptr), DAVET_EINVAL,
                  "davet_policy_step_device: argmax_prev is NULL exactly at "
                  "t = 1");
  const int K = pols[0].K;
  double alpha[DAVET_MAX_SEQS], lo[DAVET_MAX_SEQS], up[DAVET_MAX_SEQS];
  for (int i = 0; i < n_seqs; ++i) {
    DAVET_CHECK_ARG(pols[i].K == K && K >= 1 && K <= DAVET_MAX_LEVELS,
                    DAVET_EINVAL,
                    "davet_policy_step_device: every policy needs the same K "
                    "in [1, 4]");
    alpha[i] = pols[i].alpha;
    lo[i] = lower[(size_t)i * T + t];          // step t+1 (0-based index t)
    up[i] = upper[(size_t)i * T + t];
  }
  return launch_policy_step(n_seqs, L, K, alpha, lo, up, conf, argmax,
                            argmax_prev, masked_after, level_out, budget_out,
                            r_out, nullptr, nullptr, nullptr, 0, stream);
}
