// Confidence-ranked commitment, Eq. (2) (Sec. 5.1: positions are committed by
// confidence ranking).  One workgroup per sequence.  Every masked position
// computes its rank under the total order (confidence descending, NaN treated
// as -inf, then position ascending) by counting the masked positions ahead of
// it; the first min(k, |M|) ranks commit.  Comparisons only: the selection is
// exact and independent of scheduling.

#include "common.h"

namespace davet {
namespace {

__device__ __forceinline__ float rank_key(float c) {
  return (c != c) ? -INFINITY : c;
}

__global__ void __launch_bounds__(256)
unmask_kernel(int L, int k, const float* __restrict__ conf,
              const int32_t* __restrict__ argmax, int32_t* __restrict__ ids,
              uint8_t* __restrict__ masked, int32_t* __restrict__ selected) {
  __shared__ float key[DAVET_MAX_RESP];
  __shared__ uint8_t msk[DAVET_MAX_RESP];
  __shared__ int cnt;
  const int s = blockIdx.x;
  const size_t base = (size_t)s * L;
  if (threadIdx.x == 0) cnt = 0;
  __syncthreads();
  int local = 0;
  for (int i = threadIdx.x; i < L; i += blockDim.x) {
    const uint8_t m = masked[base + i] != 0;
    msk[i] = m;
    key[i] = rank_key(conf[base + i]);
    local += m;
  }
  atomicAdd(&cnt, local);
  __syncthreads();
  const int kt = min(k, cnt);
  for (int i = threadIdx.x; i < L; i += blockDim.x) {
    if (!msk[i]) continue;
    const float ki = key[i];
    int rank = 0;
    for (int j = 0; j < L; ++j) {
      const float kj = key[j];
      rank += msk[j] && (kj > ki || (kj == ki && j < i));
    }
    if (rank < kt) {
      ids[base + i] = argmax[base + i];
      masked[base + i] = 0;
      if (selected) selected[(size_t)s * k + rank] = i;
    }
  }
  if (selected)
    for (int r = kt + threadIdx.x; r < k; r += blockDim.x)
      selected[(size_t)s * k + r] = -1;
}

}  // namespace

int launch_unmask(int n_seqs, int L, int k, const float* conf,
                  const int32_t* argmax, int32_t* ids, uint8_t* masked,
                  int32_t* selected, hipStream_t s) {
  ProfScope ps(KC_UNMASK, s);
  hipLaunchKernelGGL(unmask_kernel, dim3(n_seqs), dim3(256), 0, s, L, k, conf,
                     argmax, ids, masked, selected);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

}  // namespace davet

extern "C" int davet_unmask(int32_t n_seqs, int32_t L, int32_t k,
                            const float* conf, const int32_t* argmax,
                            int32_t* resp_ids, uint8_t* resp_masked,
                            int32_t* selected, hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(conf && argmax && resp_ids && resp_masked, DAVET_EINVAL,
                  "davet_unmask: null pointer");
  DAVET_CHECK_ARG(k >= 1, DAVET_EINVAL, "davet_unmask: k must be >= 1");
  DAVET_CHECK_ARG(n_seqs >= 1 && n_seqs <= 65535, DAVET_ESHAPE,
                  "davet_unmask: n_seqs out of range");
  DAVET_CHECK_ARG(L >= 1 && L <= DAVET_MAX_RESP, DAVET_ESHAPE,
                  "davet_unmask: L out of range [1, 1024]");
  return launch_unmask(n_seqs, L, k, conf, argmax, resp_ids, resp_masked,
                       selected, stream);
}
