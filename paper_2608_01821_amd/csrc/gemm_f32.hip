// float32 GEMMs for the fp32 configuration: C[M,N] = A[M,K] * B[N,K]^T on the
// vector ALUs (fp32 FMA), 64 x 64 tiles, 16-deep K slabs staged in LDS, each
// of 256 threads accumulating a 4 x 4 block.  Same epilogues as the bf16
// path; the SwiGLU form accumulates gate and up blocks side by side.  Rows at
// or beyond *m_count (when given) are skipped, for the vocabulary head whose
// live row count is known only on the device.

#include "common.h"

namespace davet {
namespace {

constexpr int TB = 64, TK = 16;

template <int EPI>
__global__ void __launch_bounds__(256)
gemm_f32_kernel(const float* __restrict__ A, const float* __restrict__ B,
                const float* __restrict__ B2, float* __restrict__ C, int M,
                int N, int K, int ldc, const int32_t* __restrict__ m_count) {
  constexpr bool DUAL = EPI == EPI_SWIGLU;
  __shared__ float As[TK][TB + 4];
  __shared__ float Bs[TK][TB + 4];
  __shared__ float B2s[DUAL ? TK : 1][TB + 4];
  const int m_live = m_count ? m_count[0] : M;
  const int m0 = blockIdx.y * TB, n0 = blockIdx.x * TB;
  if (m0 >= m_live) return;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {}, acc2[4][4] = {};
  // loader: each thread moves 4 elements of A and of B per slab
  const int lr = threadIdx.x >> 2;          // 0..63
  const int lk = (threadIdx.x & 3) * 4;     // 0,4,8,12
  const int am = min(m0 + lr, m_live - 1);
  const int bn = min(n0 + lr, N - 1);
  for (int k0 = 0; k0 < K; k0 += TK) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = k0 + lk + e;
      As[lk + e][lr] = k < K ? A[(size_t)am * K + k] : 0.f;
      Bs[lk + e][lr] = k < K ? B[(size_t)bn * K + k] : 0.f;
      if constexpr (DUAL) B2s[lk + e][lr] = k < K ? B2[(size_t)bn * K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4], b2[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = As[kk][ty * 4 + i];
        b[i] = Bs[kk][tx * 4 + i];
        if constexpr (DUAL) b2[i] = B2s[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
          if constexpr (DUAL) acc2[i][j] = fmaf(a[i], b2[j], acc2[i][j]);
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= m_live) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col >= N) continue;
      float* c = C + (size_t)row * ldc + col;
      if constexpr (EPI == EPI_STORE) *c = acc[i][j];
      else if constexpr (EPI == EPI_ADD_F32) *c += acc[i][j];
      else {
        const float g = acc[i][j];
        *c = g / (1.0f + expf(-g)) * acc2[i][j];
      }
    }
  }
}

}  // namespace

// For EPI_SWIGLU, N is the number of output columns (= ffn) and B/B2 are the
// gate and up weights.
int launch_gemm_f32(int epi, const float* A, const float* B, const float* B2,
                    float* C, int M, int N, int K, int ldc, int cls,
                    const int32_t* m_count, hipStream_t s) {
  if (M <= 0) return DAVET_OK;
  ProfScope ps(cls, s);
  dim3 grid((N + TB - 1) / TB, (M + TB - 1) / TB);
  switch (epi) {
    case EPI_STORE:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE>, grid, dim3(256), 0, s, A,
                         B, B2, C, M, N, K, ldc, m_count); break;
    case EPI_ADD_F32:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_ADD_F32>, grid, dim3(256), 0, s,
                         A, B, B2, C, M, N, K, ldc, m_count); break;
    case EPI_SWIGLU:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, dim3(256), 0, s, A,
                         B, B2, C, M, N, K, ldc, m_count); break;
    default:
      return set_error(DAVET_EINVAL, "gemm_f32: unknown epilogue");
  }
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

}  // namespace davet
