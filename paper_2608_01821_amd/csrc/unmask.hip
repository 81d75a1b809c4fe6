// Confidence-ranked commitment, Eq. (2) (Sec. 5.1: positions are committed by
// confidence ranking).  One workgroup per sequence.  Every masked position
// computes its rank under the total order (confidence descending, NaN treated
// as -inf, then position ascending) by counting the masked positions ahead of
// it; the first min(k, |M|) ranks commit.  Comparisons only: the selection is
// exact and independent of scheduling.

#include "common.h"

namespace davet {
namespace {

// Rank key of a position: NaN ranks as -inf and -0 as +0 (equal floats tie
// and fall back to the position), encoded so that unsigned order is
// (confidence descending, position ascending); committed positions get the
// largest key and are never counted.
__device__ __forceinline__ uint64_t rank_code(float c, int i) {
  if (c != c) c = -INFINITY;
  if (c == 0.f) c = 0.f;
  uint32_t u = __float_as_uint(c);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);   // ascending float order
  return ((uint64_t)(~u) << 32) | (uint32_t)i;
}

constexpr int kPer = DAVET_MAX_RESP / 256;   // positions per thread

__global__ void __launch_bounds__(256)
unmask_kernel(int L, int k, const float* __restrict__ conf,
              const int32_t* __restrict__ argmax, int32_t* __restrict__ ids,
              uint8_t* __restrict__ masked, int32_t* __restrict__ selected) {
  __shared__ uint64_t code[DAVET_MAX_RESP];
  __shared__ int wcnt[4];
  const int s = blockIdx.x;
  const size_t base = (size_t)s * L;
  uint64_t mine[kPer];
  int local = 0;
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int i = threadIdx.x + q * 256;
    mine[q] = ~0ull;
    if (i < L) {
      if (masked[base + i]) {
        mine[q] = rank_code(conf[base + i], i);
        ++local;
      }
      code[i] = mine[q];
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) local += __shfl_xor(local, o, 64);
  if ((threadIdx.x & 63) == 0) wcnt[threadIdx.x >> 6] = local;
  __syncthreads();
  const int kt = min(k, wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3]);
  int rank[kPer];
#pragma unroll
  for (int q = 0; q < kPer; ++q) rank[q] = 0;
  for (int j = 0; j < L; ++j) {
    const uint64_t cj = code[j];
#pragma unroll
    for (int q = 0; q < kPer; ++q) rank[q] += cj < mine[q];
  }
#pragma unroll
  for (int q = 0; q < kPer; ++q) {
    const int i = threadIdx.x + q * 256;
    if (i < L && mine[q] != ~0ull && rank[q] < kt) {
      ids[base + i] = argmax[base + i];
      masked[base + i] = 0;
      if (selected) selected[(size_t)s * k + rank[q]] = i;
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
