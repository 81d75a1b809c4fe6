// Bidirectional (non-causal) attention over a packed batch of independent
// sequences (Sec. 1 and Sec. 3.1: dVLMs refine all answer positions in
// parallel through bidirectional attention).  Every query of a sequence sees
// every key of the same sequence; sequences never mix.
//
// 16-bit path (bf16 or fp16 operands), head_dim 128, CDNA4 matrix cores.  A
// workgroup of 4 wavefronts owns 128 queries of one head; each wavefront owns
// 32 queries.  Keys stream in tiles of 64 staged in LDS: K row-major, V
// transposed.  Per tile a wavefront computes S^T = K Q^T (2 x 8
// v_mfma_f32_32x32x16 ops), so every lane holds the scores of ONE query: the
// online-softmax rescale is a per-lane scalar and the probabilities, rounded
// to 16 bits, are already laid out as the B operand of O^T += V^T P^T (4 x 4
// MFMAs) -- no LDS round trip for P.  Scores,
// running max and normaliser stay in fp32 (exp2 with log2(e) folded into the
// 1/sqrt(D) scale).  Ragged tails: keys past the sequence end score -inf;
// queries past it are computed on clamped rows and never stored.

#include "common.h"

namespace davet {
namespace {

constexpr int HD = 128;           // head dim of the matrix-core path
constexpr int QT = 128;           // queries per workgroup
constexpr int KT = 64;            // keys per tile
constexpr int K_STRIDE = HD + 8;  // 272-byte K rows
constexpr int V_STRIDE = KT + 4;  // 136-byte V^T rows (conflict-free b64 reads)

__device__ __forceinline__ void locate_tile(const SeqPack& sp, int tile,
                                            int qtile, int& s, int& qt) {
  s = 0;
  int acc = 0;
  for (;;) {
    const int n = sp.row0[s + 1] - sp.row0[s];
    const int nt = (n + qtile - 1) / qtile;
    if (tile < acc + nt || s + 1 >= sp.n_seqs) break;
    acc += nt;
    ++s;
  }
  qt = tile - acc;
}

template <typename Fmt>
__global__ void __launch_bounds__(256, 1)
attn16_kernel(const uint16_t* __restrict__ qkv, uint16_t* __restrict__ out,
              SeqPack sp, int n_heads, float scale_log2) {
  using v8 = typename Fmt::v8;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[KT * K_STRIDE];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[HD * V_STRIDE];
  int s, qt;
  locate_tile(sp, blockIdx.x, QT, s, qt);
  const int h = blockIdx.y;
  const int d = n_heads * HD;
  const size_t ld = (size_t)3 * d;
  const int row0 = sp.row0[s];
  const int N = sp.row0[s + 1] - row0;
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int q = qt * QT + wave * 32 + l32;         // this lane's query
  const int qc = min(q, N - 1);

  // Q^T fragments (B operand): 8 k-steps of 16 head dims
  v8 qf[HD / 16];
  {
    const uint16_t* qp = qkv + (size_t)(row0 + qc) * ld + (size_t)h * HD + hh * 8;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks)
      qf[ks] = __builtin_bit_cast(v8,
                                  *reinterpret_cast<const u32x4*>(qp + ks * 16));
  }
  f32x16 o[HD / 32];
#pragma unroll
  for (int i = 0; i < HD / 32; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[i][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const uint16_t* kbase = qkv + (size_t)row0 * ld + d + (size_t)h * HD;
  const uint16_t* vbase = qkv + (size_t)row0 * ld + 2 * d + (size_t)h * HD;
  const int n_kt = (N + KT - 1) / KT;
  for (int kb = 0; kb < n_kt; ++kb) {
    const int k0 = kb * KT;
    // ---- stage K (row-major) and V (transposed) tiles in LDS
#pragma unroll
    for (int it = 0; it < KT * HD / 8 / 256; ++it) {
      const int w = t + it * 256;
      const int key = w >> 4, ch = w & 15;
      const int gk = min(k0 + key, N - 1);
      *reinterpret_cast<u32x4*>(&Ks[key * K_STRIDE + ch * 8]) =
          *reinterpret_cast<const u32x4*>(kbase + (size_t)gk * ld + ch * 8);
    }
#pragma unroll
    for (int it = 0; it < KT * HD / 16 / 256; ++it) {
      const int w = t + it * 256;
      const int kp = w >> 4, dc = w & 15;
      const int g0 = min(k0 + 2 * kp, N - 1), g1 = min(k0 + 2 * kp + 1, N - 1);
      const u32x4 a = *reinterpret_cast<const u32x4*>(vbase + (size_t)g0 * ld + dc * 8);
      const u32x4 b = *reinterpret_cast<const u32x4*>(vbase + (size_t)g1 * ld + dc * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t lo = (a[e] & 0xffffu) | (b[e] << 16);
        const uint32_t hi = (a[e] >> 16) | (b[e] & 0xffff0000u);
        *reinterpret_cast<uint32_t*>(&Vt[(dc * 8 + 2 * e) * V_STRIDE + 2 * kp]) = lo;
        *reinterpret_cast<uint32_t*>(&Vt[(dc * 8 + 2 * e + 1) * V_STRIDE + 2 * kp]) = hi;
      }
    }
    __syncthreads();

    // ---- S^T = K Q^T for 64 keys x 32 queries (two 32-key halves)
    f32x16 sc[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[mt][e] = 0.f;
#pragma unroll
      for (int ks = 0; ks < HD / 16; ++ks) {
        const v8 kf = __builtin_bit_cast(
            v8, *reinterpret_cast<const u32x4*>(
                    &Ks[(mt * 32 + l32) * K_STRIDE + ks * 16 + hh * 8]));
        sc[mt] = Fmt::mfma32(kf, qf[ks], sc[mt]);
      }
    }
    // ---- online softmax for this lane's query over its 32 keys + partner's 32
    float tmax = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = k0 + mt * 32 + (e >> 2) * 8 + hh * 4 + (e & 3);
        const float v = key < N ? sc[mt][e] * scale_log2 : -INFINITY;
        sc[mt][e] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = exp2f(m_run - m_new);
    float psum = 0.f;
    uint16_t pb[4][8];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = exp2f(sc[mt][e] - m_new);
        psum += p;
        pb[mt * 2 + (e >> 3)][e & 7] = Fmt::store(p);
      }
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < HD / 32; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[i][e] *= alpha;

    // ---- O^T += V^T P^T: k-step ps covers keys 16*ps .. 16*ps+15
#pragma unroll
    for (int ps = 0; ps < 4; ++ps) {
      const int kbase_l = ps * 16 + hh * 4;
#pragma unroll
      for (int dt = 0; dt < HD / 32; ++dt) {
        const uint16_t* vr = &Vt[(dt * 32 + l32) * V_STRIDE + kbase_l];
        const u32x2 v0 = *reinterpret_cast<const u32x2*>(vr);
        const u32x2 v1 = *reinterpret_cast<const u32x2*>(vr + 8);
        u32x4 vv;
        vv[0] = v0[0]; vv[1] = v0[1]; vv[2] = v1[0]; vv[3] = v1[1];
        u32x4 pw;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          pw[q] = (uint32_t)pb[ps][2 * q] | ((uint32_t)pb[ps][2 * q + 1] << 16);
        o[dt] = Fmt::mfma32(__builtin_bit_cast(v8, vv),
                            __builtin_bit_cast(v8, pw), o[dt]);
      }
    }
    __syncthreads();
  }

  if (q < N) {
    const float inv = 1.0f / l_run;
    uint16_t* op = out + (size_t)(row0 + q) * d + (size_t)h * HD;
#pragma unroll
    for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int dd = dt * 32 + g * 8 + hh * 4;
        u32x2 w;
        w[0] = (uint32_t)Fmt::store(o[dt][g * 4 + 0] * inv) |
               ((uint32_t)Fmt::store(o[dt][g * 4 + 1] * inv) << 16);
        w[1] = (uint32_t)Fmt::store(o[dt][g * 4 + 2] * inv) |
               ((uint32_t)Fmt::store(o[dt][g * 4 + 3] * inv) << 16);
        *reinterpret_cast<u32x2*>(op + dd) = w;
      }
  }
}

// fp32 path: one thread per (query, head), keys streamed with an online
// softmax; used by the small fp32 configuration.
template <int D>
__global__ void __launch_bounds__(64)
attn_f32_kernel(const float* __restrict__ qkv, float* __restrict__ out,
                SeqPack sp, int n_heads, float scale) {
  const int row = blockIdx.x * 64 + threadIdx.x;
  if (row >= sp.total) return;
  const int h = blockIdx.y;
  int s = 0;
  while (s + 1 < sp.n_seqs && sp.row0[s + 1] <= row) ++s;
  const int r0 = sp.row0[s], r1 = sp.row0[s + 1];
  const int d = n_heads * D;
  const size_t ld = (size_t)3 * d;
  float qv[D], acc[D];
  const float* qp = qkv + (size_t)row * ld + (size_t)h * D;
#pragma unroll
  for (int e = 0; e < D; ++e) { qv[e] = qp[e] * scale; acc[e] = 0.f; }
  float m = -INFINITY, l = 0.f;
  for (int j = r0; j < r1; ++j) {
    const float* kp = qkv + (size_t)j * ld + d + (size_t)h * D;
    float sc = 0.f;
#pragma unroll
    for (int e = 0; e < D; ++e) sc = fmaf(qv[e], kp[e], sc);
    const float mn = fmaxf(m, sc);
    const float a = expf(m - mn), p = expf(sc - mn);
    l = l * a + p;
    const float* vp = qkv + (size_t)j * ld + 2 * d + (size_t)h * D;
#pragma unroll
    for (int e = 0; e < D; ++e) acc[e] = acc[e] * a + p * vp[e];
    m = mn;
  }
  float* op = out + (size_t)row * d + (size_t)h * D;
  const float inv = 1.0f / l;
#pragma unroll
  for (int e = 0; e < D; ++e) op[e] = acc[e] * inv;
}

}  // namespace

int launch_attention16(int dtype, const uint16_t* qkv, uint16_t* o,
                       const SeqPack& sp, int n_heads, int head_dim,
                       hipStream_t s) {
  if (head_dim != HD)
    return set_error(DAVET_ESHAPE, "attention16: head_dim must be 128");
  int tiles = 0;
  for (int i = 0; i < sp.n_seqs; ++i)
    tiles += (sp.row0[i + 1] - sp.row0[i] + QT - 1) / QT;
  if (tiles == 0) return DAVET_OK;
  ProfScope ps(KC_ATTN, s);
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)head_dim);
  if (dtype == DAVET_F16)
    hipLaunchKernelGGL(attn16_kernel<F16>, dim3(tiles, n_heads), dim3(256), 0,
                       s, qkv, o, sp, n_heads, scale_log2);
  else
    hipLaunchKernelGGL(attn16_kernel<BF16>, dim3(tiles, n_heads), dim3(256), 0,
                       s, qkv, o, sp, n_heads, scale_log2);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_attention_f32(const float* qkv, float* o, const SeqPack& sp,
                         int n_heads, int head_dim, hipStream_t s) {
  if (sp.total == 0) return DAVET_OK;
  ProfScope ps(KC_ATTN_F32, s);
  dim3 grid((sp.total + 63) / 64, n_heads);
  const float scale = 1.0f / sqrtf((float)head_dim);
  if (head_dim == 64)
    hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(64), 0, s, qkv, o, sp,
                       n_heads, scale);
  else if (head_dim == 128)
    hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(64), 0, s, qkv, o, sp,
                       n_heads, scale);
  else
    return set_error(DAVET_ESHAPE, "attention_f32: head_dim must be 64 or 128");
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

}  // namespace davet
