// 16-bit (bf16 or fp16) matrix-core GEMMs of the denoiser: C[M,N] = A[M,K] * B[N,K]^T with both
// operands K-contiguous (activations row-major, weights [out, in]).
//
// Tiling for CDNA4: a 256-thread workgroup (4 wavefronts, 2 x 2) owns a
// BM x BN output tile; each wavefront issues v_mfma_f32_32x32x16_bf16 on a
// (BM/2) x (BN/2) sub-tile.  K advances in slabs of 64 staged through LDS with
// double buffering (global loads of slab k+1 are in flight while slab k feeds
// the matrix cores; one barrier per slab).  LDS rows are padded by 16 bytes so
// the 16-byte fragment reads of a half-wavefront hit distinct banks.
// Workgroup ids are remapped so each XCD (ids congruent mod 8) walks a
// contiguous run of tiles with the M index fastest: a weight tile is fetched
// into one XCD's L2 and reused by every M tile of that column.
//
// Epilogues (fused, no extra pass over C):
//   EPI_STORE    C (16-bit) = acc
//   EPI_ADD_F32  C f32 += acc           (residual stream update)
//   EPI_SWIGLU   dual weight: the tile's first BN/2 columns come from B (gate),
//                the last BN/2 from B2 (up) at the same output index; the wave
//                layout puts gate and up of one column in the same lane, so
//                C (16-bit) = silu(gate) * up is formed in registers.
//   head         vocabulary slab reduction: per row, (max, first argmax, sum of
//                exp(l - max)) over the slab's columns with [MASK] excluded.

#include "common.h"

namespace davet {
namespace {

constexpr int BK = 64;
constexpr int LDS_STRIDE = BK + 8;     // elements; 144-byte rows
constexpr int EPI_HEAD = 3;

struct HeadArgs {
  const int32_t* list;   // list[0] = live rows, list[1+j] = global position
  int vocab;
  int mask_id;
  int n_slabs;
  float* pmax;
  float* psum;
  int32_t* parg;
  float* logits_out;     // nullable
};

__device__ __forceinline__ int remap_xcd(int bid, int nwg) {
  const int full = nwg & ~7;
  if (bid >= full) return bid;
  const int per = full >> 3;
  return (bid & 7) * per + (bid >> 3);
}

template <typename Fmt, int BM, int BN, int EPI>
__global__ void __launch_bounds__(256, 1)
gemm16_kernel(const uint16_t* __restrict__ A, const uint16_t* __restrict__ B,
                 const uint16_t* __restrict__ B2, void* __restrict__ C, int M,
                 int N, int K, int ldc, int n_mtiles, HeadArgs ha) {
  constexpr int TM = BM / 64;            // 32-row sub-tiles per wave
  constexpr int TN = BN / 64;            // 32-col sub-tiles per wave
  constexpr int A_LD = BM / 32;          // 16-byte loads per thread
  constexpr int B_LD = BN / 32;
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LDS_STRIDE];

  const int nwg = gridDim.x;
  const int tile = remap_xcd(blockIdx.x, nwg);
  const int mb = tile % n_mtiles;
  const int nb = tile / n_mtiles;
  int m_live = M;
  if constexpr (EPI == EPI_HEAD) m_live = ha.list[0];
  const int m0 = mb * BM;
  if (m0 >= m_live) return;
  const int n0 = nb * BN;

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // global source pointers of this thread's 16-byte chunks
  const uint16_t* a_src[A_LD];
  const uint16_t* b_src[B_LD];
#pragma unroll
  for (int q = 0; q < A_LD; ++q) {
    const int r = q * 32 + (t >> 3);
    const int gm = min(m0 + r, m_live - 1);
    a_src[q] = A + (size_t)gm * K + (t & 7) * 8;
  }
#pragma unroll
  for (int q = 0; q < B_LD; ++q) {
    const int r = q * 32 + (t >> 3);
    const uint16_t* base;
    int gn;
    if constexpr (EPI == EPI_SWIGLU) {
      const int half = BN / 2;
      base = r < half ? B : B2;
      gn = nb * half + (r < half ? r : r - half);
    } else {
      base = B;
      gn = min(n0 + r, N - 1);
    }
    b_src[q] = base + (size_t)gn * K + (t & 7) * 8;
  }

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  u32x4 ra[A_LD], rb[B_LD];
  auto gload = [&](int k0) {
#pragma unroll
    for (int q = 0; q < A_LD; ++q)
      ra[q] = *reinterpret_cast<const u32x4*>(a_src[q] + k0);
#pragma unroll
    for (int q = 0; q < B_LD; ++q)
      rb[q] = *reinterpret_cast<const u32x4*>(b_src[q] + k0);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int q = 0; q < A_LD; ++q)
      *reinterpret_cast<u32x4*>(&As[buf][(q * 32 + (t >> 3)) * LDS_STRIDE +
                                         (t & 7) * 8]) = ra[q];
#pragma unroll
    for (int q = 0; q < B_LD; ++q)
      *reinterpret_cast<u32x4*>(&Bs[buf][(q * 32 + (t >> 3)) * LDS_STRIDE +
                                         (t & 7) * 8]) = rb[q];
  };

  const int nk = K / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  const int lr = lane & 31;           // row inside a 32-row fragment
  const int lk = (lane >> 5) * 8;     // k offset inside a 16-wide k-step
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      typename Fmt::v8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm * (BM / 2) + i * 32 + lr;
        af[i] = __builtin_bit_cast(
            typename Fmt::v8, *reinterpret_cast<const u32x4*>(
                        &As[cur][row * LDS_STRIDE + kk * 16 + lk]));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = j * 64 + wn * 32 + lr;
        bfr[j] = __builtin_bit_cast(
            typename Fmt::v8, *reinterpret_cast<const u32x4*>(
                        &Bs[cur][row * LDS_STRIDE + kk * 16 + lk]));
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = Fmt::mfma32(af[i], bfr[j], acc[i][j]);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // acc[i][j][e]: row = wm*BM/2 + i*32 + (e/4)*8 + (lane/32)*4 + e%4,
  //               col = j*64 + wn*32 + lane%32   (tile-local)
  const int hrow = (lane >> 5) * 4;
  if constexpr (EPI == EPI_STORE || EPI == EPI_ADD_F32) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = n0 + j * 64 + wn * 32 + lr;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * (BM / 2) + i * 32 + (e >> 2) * 8 + hrow +
                          (e & 3);
          if (row < M) {
            if constexpr (EPI == EPI_STORE)
              reinterpret_cast<uint16_t*>(C)[(size_t)row * ldc + col] =
                  Fmt::store(acc[i][j][e]);
            else
              reinterpret_cast<float*>(C)[(size_t)row * ldc + col] +=
                  acc[i][j][e];
          }
        }
      }
  } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN / 2; ++j) {
        const int col = nb * (BN / 2) + j * 64 + wn * 32 + lr;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * (BM / 2) + i * 32 + (e >> 2) * 8 + hrow +
                          (e & 3);
          if (row < M) {
            const float g = acc[i][j][e];
            const float u = acc[i][j + TN / 2][e];
            const float h = g / (1.0f + __expf(-g)) * u;
            reinterpret_cast<uint16_t*>(C)[(size_t)row * ldc + col] =
                Fmt::store(h);
          }
        }
      }
  } else {   // EPI_HEAD
    __shared__ float red_m[2][BM];
    __shared__ float red_s[2][BM];
    __shared__ int red_a[2][BM];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int lrow = wm * (BM / 2) + i * 32 + (e >> 2) * 8 + hrow + (e & 3);
        const int row = m0 + lrow;
        float m = -INFINITY, s = 0.f;
        int a = 0x7fffffff;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int col = n0 + j * 64 + wn * 32 + lr;
          float v = acc[i][j][e];
          if (ha.logits_out && row < m_live && col < ha.vocab)
            ha.logits_out[(size_t)ha.list[1 + row] * ha.vocab + col] = v;
          if (col == ha.mask_id || col >= ha.vocab) v = -INFINITY;
          if (v > m) {              // columns ascend with j: keeps the first
            s = s * __expf(m - v) + 1.0f;
            m = v; a = col;
          } else if (v != -INFINITY) {
            s += __expf(v - m);
          }
        }
        // combine over the 32 lanes of this half-wave (same row)
#pragma unroll
        for (int o = 1; o < 32; o <<= 1) {
          const float m2 = __shfl_xor(m, o, 64);
          const float s2 = __shfl_xor(s, o, 64);
          const int a2 = __shfl_xor(a, o, 64);
          const float mm = fmaxf(m, m2);
          float ns = 0.f;
          if (m != -INFINITY) ns += s * __expf(m - mm);
          if (m2 != -INFINITY) ns += s2 * __expf(m2 - mm);
          const int na = (m2 > m || (m2 == m && a2 < a)) ? a2 : a;
          m = mm; s = ns; a = na;
        }
        if (lr == 0) {
          red_m[wn][lrow] = m;
          red_s[wn][lrow] = s;
          red_a[wn][lrow] = a;
        }
      }
    }
    __syncthreads();
    for (int r = t; r < BM; r += 256) {
      const int row = m0 + r;
      if (row >= m_live) continue;
      const float m1 = red_m[0][r], m2 = red_m[1][r];
      const float mm = fmaxf(m1, m2);
      float s = 0.f;
      if (m1 != -INFINITY) s += red_s[0][r] * __expf(m1 - mm);
      if (m2 != -INFINITY) s += red_s[1][r] * __expf(m2 - mm);
      const int a1 = red_a[0][r], a2 = red_a[1][r];
      const int a = (m2 > m1 || (m2 == m1 && a2 < a1)) ? a2 : a1;
      const size_t o = (size_t)row * ha.n_slabs + nb;
      ha.pmax[o] = mm;
      ha.psum[o] = s;
      ha.parg[o] = a;
    }
  }
}

template <typename Fmt, int BM, int BN, int EPI>
int launch(const uint16_t* A, const uint16_t* B, const uint16_t* B2, void* C,
           int M, int N, int K, int ldc, int n_ntiles, const HeadArgs& ha,
           hipStream_t s) {
  const int mt = (M + BM - 1) / BM;
  const int nwg = mt * n_ntiles;
  hipLaunchKernelGGL((gemm16_kernel<Fmt, BM, BN, EPI>), dim3(nwg), dim3(256),
                     0, s, A, B, B2, C, M, N, K, ldc, mt, ha);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

template <typename Fmt>
int gemm_dispatch(int epi, const uint16_t* A, const uint16_t* B,
                  const uint16_t* B2, void* C, int M, int N, int K, int ldc,
                  hipStream_t s) {
  HeadArgs ha{};
  switch (epi) {
    case EPI_STORE:
      return launch<Fmt, 128, 128, EPI_STORE>(A, B, B2, C, M, N, K, ldc,
                                              N / 128, ha, s);
    case EPI_ADD_F32:
      return launch<Fmt, 128, 128, EPI_ADD_F32>(A, B, B2, C, M, N, K, ldc,
                                                N / 128, ha, s);
    case EPI_SWIGLU:   // N = 2 * ffn output columns of gate|up
      return launch<Fmt, 128, 128, EPI_SWIGLU>(A, B, B2, C, M, N, K, ldc,
                                               N / 128, ha, s);
  }
  return set_error(DAVET_EINVAL, "gemm16: unknown epilogue");
}

}  // namespace

int launch_gemm16(int dtype, int epi, const uint16_t* A, const uint16_t* B,
                  const uint16_t* B2, void* C, int M, int N, int K, int ldc,
                  int cls, hipStream_t s) {
  if (M <= 0) return DAVET_OK;
  if (N % 128 || K % BK)
    return set_error(DAVET_ESHAPE, "gemm16: N % 128 or K % 64 != 0");
  ProfScope ps(cls, s);
  return dtype == DAVET_F16
             ? gemm_dispatch<F16>(epi, A, B, B2, C, M, N, K, ldc, s)
             : gemm_dispatch<BF16>(epi, A, B, B2, C, M, N, K, ldc, s);
}

int head16_slabs(int vocab) { return (vocab + 127) / 128; }

int launch_head16(int dtype, const uint16_t* Hm, const uint16_t* W,
                  const int32_t* list, int max_rows, int vocab, int d,
                  int mask_id, float* pmax, float* psum, int32_t* parg,
                  float* logits_out, hipStream_t s) {
  if (d % BK) return set_error(DAVET_ESHAPE, "head16: d % 64 != 0");
  ProfScope ps(KC_HEAD, s);
  HeadArgs ha{list, vocab, mask_id, head16_slabs(vocab), pmax, psum, parg,
              logits_out};
  return dtype == DAVET_F16
             ? launch<F16, 128, 128, EPI_HEAD>(Hm, W, nullptr, nullptr,
                                               max_rows, vocab, d, 0,
                                               ha.n_slabs, ha, s)
             : launch<BF16, 128, 128, EPI_HEAD>(Hm, W, nullptr, nullptr,
                                                max_rows, vocab, d, 0,
                                                ha.n_slabs, ha, s);
}

}  // namespace davet
