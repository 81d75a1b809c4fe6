// Row-wise kernels of the denoiser step: sequence assembly + embedding gather
// fused with the first RMSNorm, RMSNorm, rotary embedding, masked-row
// compaction, final norm of the masked rows, and the vocabulary-reduction
// merge.  One workgroup (4 wavefronts) per row; reductions are wavefront
// butterflies followed by a 4-entry LDS combine.

#include <algorithm>

#include "common.h"

namespace davet {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float block_sum(float v, float* red) {
  v = warp_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) t += red[i];
  return t;
}

__device__ __forceinline__ int find_seq(const SeqPack& sp, int row) {
  int s = 0;
  while (s + 1 < sp.n_seqs && sp.row0[s + 1] <= row) ++s;
  return s;
}

// Rows are moved in chunks of 8 elements (16 bytes of a 16-bit format, 32 of
// fp32): d is a multiple of 64, every row start is 16-byte aligned.  A thread
// owns chunks t, t + 256, ... (at most 4: d <= 8192).
constexpr int kMaxChunks = 4;

template <typename Fmt>
__device__ __forceinline__ void load8(const typename Fmt::st* p, float* v) {
  if constexpr (Fmt::dtype == DAVET_F32) {
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  } else {
    const u32x4 w = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = Fmt::load((uint16_t)(w[i] & 0xffffu));
      v[2 * i + 1] = Fmt::load((uint16_t)(w[i] >> 16));
    }
  }
}

template <typename Fmt>
__device__ __forceinline__ void store8(typename Fmt::st* p, const float* v) {
  if constexpr (Fmt::dtype == DAVET_F32) {
    reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
  } else {
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)Fmt::store(v[2 * i]) |
             ((uint32_t)Fmt::store(v[2 * i + 1]) << 16);
    *reinterpret_cast<u32x4*>(p) = w;
  }
}

// store8 for 16-bit formats that also counts the non-finite values stored
template <typename Fmt>
__device__ __forceinline__ int store8_count(typename Fmt::st* p,
                                            const float* v) {
  u32x4 w;
  int nf = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint16_t a = Fmt::store(v[2 * i]), b = Fmt::store(v[2 * i + 1]);
    nf += Fmt::nonfinite(a) + Fmt::nonfinite(b);
    w[i] = (uint32_t)a | ((uint32_t)b << 16);
  }
  *reinterpret_cast<u32x4*>(p) = w;
  return nf;
}

__device__ __forceinline__ void load8f(const float* p, float* v) {
  load8<F32S>(p, v);
}
__device__ __forceinline__ void store8f(float* p, const float* v) {
  store8<F32S>(p, v);
}

// gain chunk (1.0 where no gain vector is given)
__device__ __forceinline__ void gain8(const float* g, int e, float* v) {
  if (g) {
    load8f(g + e, v);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = 1.0f;
  }
}

// A[row] = 16-bit or fp32 RMSNorm of the row chunks x (sum of squares ss of
// this thread's part).
template <typename Fmt, typename T = typename Fmt::st>
__device__ __forceinline__ void norm_store(float (*x)[8], float ss, int d,
                                           const float* __restrict__ gain,
                                           float eps, T* __restrict__ out,
                                           float* red) {
  const float tot = block_sum(ss, red);
  const float rstd = 1.0f / sqrtf(tot / (float)d + eps);
  const int nc = d / 8;
#pragma unroll
  for (int n = 0; n < kMaxChunks; ++n) {
    const int c = threadIdx.x + n * kThreads;
    if (c >= nc) break;
    float g[8], y[8];
    gain8(gain, c * 8, g);
#pragma unroll
    for (int i = 0; i < 8; ++i) y[i] = x[n][i] * rstd * g[i];
    store8<Fmt>(out + (size_t)c * 8, y);
  }
}

// One workgroup: ordered list of masked response positions (global index
// s*L + i) with the count in list[0], and (if slot is given) each position's
// index in that list, -1 for committed ones; committed positions get conf =
// -inf and argmax = -1.  Each thread takes a contiguous run of positions; the
// run offsets come from a workgroup prefix sum (wavefront scan + LDS).
__device__ __forceinline__ void build_row_list(const RowList& rl,
                                               const uint8_t* __restrict__ masked) {
  __shared__ int wsum[kThreads / 64];
  const int total = rl.total;
  const int per = (total + kThreads - 1) / kThreads;
  const int lo = min(total, (int)threadIdx.x * per);
  const int hi = min(total, lo + per);
  int c = 0;
  for (int i = lo; i < hi; ++i) c += masked[i] != 0;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int incl = c;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  int base = 0, all = 0;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) {
    if (i < w) base += wsum[i];
    all += wsum[i];
  }
  if (threadIdx.x == 0) {
    rl.list[0] = all;
    if (rl.overflow && rl.clear_overflow) *rl.overflow = 0;
  }
  int o = base + incl - c;
  for (int i = lo; i < hi; ++i) {
    if (masked[i]) {
      if (rl.slot) rl.slot[i] = o;
      rl.list[1 + o++] = i;
    } else {
      if (rl.slot) rl.slot[i] = -1;
      rl.conf[i] = -INFINITY;
      rl.argmax[i] = -1;
    }
  }
}

// X[row] = [view | E[prompt] | E[resp or mask]] row; A[row] = RMSNorm(X[row]).
// One extra workgroup after the rows builds the masked-row list meanwhile.
template <typename Fmt, typename T = typename Fmt::st>
__global__ void __launch_bounds__(kThreads)
assemble_norm_kernel(SeqPack sp, ViewPtrs vp, const T* __restrict__ embed,
                     const int32_t* __restrict__ prompt_ids,
                     const int32_t* __restrict__ resp_ids,
                     const uint8_t* __restrict__ masked, int mask_id,
                     int vocab, int d, const float* __restrict__ gain,
                     float eps, float* __restrict__ X, T* __restrict__ A,
                     int32_t* __restrict__ pos, RowList rl) {
  __shared__ float red[kThreads / 64];
  const int row = blockIdx.x;
  if (row == sp.total) {
    build_row_list(rl, masked);
    return;
  }
  const int s = find_seq(sp, row);
  const int j = row - sp.row0[s];
  if (threadIdx.x == 0 && pos) pos[row] = j;     // rotary position
  const T* src;
  if (j < sp.nview[s]) {
    src = reinterpret_cast<const T*>(vp.p[s]) + (size_t)j * d;
  } else if (j < sp.nview[s] + sp.plen[s]) {
    // ids outside [0, vocab) are clamped, never read out of bounds
    const int id = min(max(prompt_ids[sp.pstart[s] + j - sp.nview[s]], 0),
                       vocab - 1);
    src = embed + (size_t)id * d;
  } else {
    const int i = j - sp.nview[s] - sp.plen[s];
    const size_t q = (size_t)s * sp.L + i;
    const int id = masked[q] ? mask_id : min(max(resp_ids[q], 0), vocab - 1);
    src = embed + (size_t)id * d;
  }
  const int nc = d / 8;
  float x[kMaxChunks][8];
  float ss = 0.f;
#pragma unroll
  for (int n = 0; n < kMaxChunks; ++n) {
    const int c = threadIdx.x + n * kThreads;
    if (c < nc) {
      load8<Fmt>(src + (size_t)c * 8, x[n]);
      store8f(X + (size_t)row * d + c * 8, x[n]);
#pragma unroll
      for (int i = 0; i < 8; ++i) ss += x[n][i] * x[n][i];
    }
  }
  norm_store<Fmt>(x, ss, d, gain, eps, A + (size_t)row * d, red);
}

template <typename Fmt, typename T = typename Fmt::st>
__global__ void __launch_bounds__(kThreads)
rmsnorm_kernel(const float* __restrict__ X, int d,
               const float* __restrict__ gain, float eps, T* __restrict__ A) {
  __shared__ float red[kThreads / 64];
  const int row = blockIdx.x;
  const float* x = X + (size_t)row * d;
  const int nc = d / 8;
  float v[kMaxChunks][8];
  float ss = 0.f;
#pragma unroll
  for (int n = 0; n < kMaxChunks; ++n) {
    const int c = threadIdx.x + n * kThreads;
    if (c < nc) {
      load8f(x + c * 8, v[n]);
#pragma unroll
      for (int i = 0; i < 8; ++i) ss += v[n][i] * v[n][i];
    }
  }
  norm_store<Fmt>(v, ss, d, gain, eps, A + (size_t)row * d, red);
}

// cos/sin of pos * theta^(-2i/D), evaluated in float64 and rounded once.
__global__ void rope_table_kernel(int max_pos, int head_dim, double theta,
                                  float2* __restrict__ cs) {
  const int half = head_dim / 2;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= max_pos * half) return;
  const int pos = idx / half, i = idx % half;
  const double inv = pow(theta, -(2.0 * i) / (double)head_dim);
  const double a = (double)pos * inv;
  cs[idx] = make_float2((float)cos(a), (float)sin(a));
}

// In-place rotary embedding of the query and key parts of qkv [rows, 3d]:
// dim i pairs with dim i + D/2 inside each head (rotate-half form).
template <typename Fmt, typename T = typename Fmt::st>
__global__ void __launch_bounds__(kThreads)
rope_kernel(T* __restrict__ qkv, SeqPack sp, int n_heads, int head_dim,
            const float2* __restrict__ cs) {
  const int row = blockIdx.x;
  const int s = find_seq(sp, row);
  const int pos = row - sp.row0[s];
  const int d = n_heads * head_dim;
  const int half = head_dim / 2;
  T* base = qkv + (size_t)row * 3 * d;
  // 2 * n_heads * half pairs: queries then keys
  for (int p = threadIdx.x; p < 2 * n_heads * half; p += kThreads) {
    const int which = p / (n_heads * half);
    const int h = (p / half) % n_heads;
    const int i = p % half;
    T* x = base + which * d + h * head_dim;
    const float2 c = cs[(size_t)pos * half + i];
    const float a = Fmt::load(x[i]), b = Fmt::load(x[i + half]);
    x[i] = Fmt::store(a * c.x - b * c.y);
    x[i + half] = Fmt::store(b * c.x + a * c.y);
  }
}

// Hm[j] = RMSNorm_final(X[packed row of masked position list[1+j]]).
template <typename Fmt, typename T = typename Fmt::st>
__global__ void __launch_bounds__(kThreads)
final_norm_gather_kernel(const float* __restrict__ X, SeqPack sp,
                         const int32_t* __restrict__ list, int d,
                         const float* __restrict__ gain, float eps,
                         T* __restrict__ Hm) {
  __shared__ float red[kThreads / 64];
  const int j = blockIdx.x;
  if (j >= list[0]) return;
  const int g = list[1 + j];
  const int s = g / sp.L, i = g % sp.L;
  const int row = sp.row0[s] + sp.nview[s] + sp.plen[s] + i;
  const float* x = X + (size_t)row * d;
  const int nc = d / 8;
  float v[kMaxChunks][8];
  float ss = 0.f;
#pragma unroll
  for (int n = 0; n < kMaxChunks; ++n) {
    const int c = threadIdx.x + n * kThreads;
    if (c < nc) {
      load8f(x + c * 8, v[n]);
#pragma unroll
      for (int q = 0; q < 8; ++q) ss += v[n][q] * v[n][q];
    }
  }
  norm_store<Fmt>(v, ss, d, gain, eps, Hm + (size_t)j * d, red);
}

// (max, first argmax, sum of exp(l - max)) partials over vocabulary slabs ->
// argmax (lowest id: slabs are in id order) and confidence 1 / sum.
__global__ void __launch_bounds__(kThreads)
head_merge_kernel(const int32_t* __restrict__ list, int n_slabs,
                  const float* __restrict__ pmax, const float* __restrict__ psum,
                  const int32_t* __restrict__ parg, float* __restrict__ conf_out,
                  int32_t* __restrict__ argmax_out) {
  __shared__ float rm[kThreads / 64];
  __shared__ int ra[kThreads / 64];
  __shared__ float red[kThreads / 64];
  const int j = blockIdx.x;
  if (j >= list[0]) return;
  const float* mx = pmax + (size_t)j * n_slabs;
  const float* sm = psum + (size_t)j * n_slabs;
  const int32_t* ag = parg + (size_t)j * n_slabs;
  float m = -INFINITY;
  int a = 0x7fffffff;
  for (int t = threadIdx.x; t < n_slabs; t += kThreads) {
    const float v = mx[t];
    const int id = ag[t];
    if (v > m || (v == m && id < a)) { m = v; a = id; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float v = __shfl_xor(m, o, 64);
    const int id = __shfl_xor(a, o, 64);
    if (v > m || (v == m && id < a)) { m = v; a = id; }
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { rm[w] = m; ra[w] = a; }
  __syncthreads();
  m = rm[0]; a = ra[0];
  for (int i = 1; i < kThreads / 64; ++i)
    if (rm[i] > m || (rm[i] == m && ra[i] < a)) { m = rm[i]; a = ra[i]; }
  float s = 0.f;
  for (int t = threadIdx.x; t < n_slabs; t += kThreads)
    s += sm[t] * __expf(mx[t] - m);
  s = block_sum(s, red);
  if (threadIdx.x == 0) {
    const int g = list[1 + j];
    conf_out[g] = 1.0f / s;
    argmax_out[g] = a;
  }
}

// Float32 path: per masked row, reduce a full logits row.
__global__ void __launch_bounds__(kThreads)
head_reduce_f32_kernel(const float* __restrict__ logits,
                       const int32_t* __restrict__ list, int V, int mask_id,
                       float* __restrict__ conf_out,
                       int32_t* __restrict__ argmax_out,
                       float* __restrict__ logits_out) {
  __shared__ float rm[kThreads / 64];
  __shared__ int ra[kThreads / 64];
  __shared__ float red[kThreads / 64];
  const int j = blockIdx.x;
  if (j >= list[0]) return;
  const int g = list[1 + j];
  const float* lg = logits + (size_t)j * V;
  float m = -INFINITY;
  int a = 0x7fffffff;
  for (int t = threadIdx.x; t < V; t += kThreads) {
    const float v = lg[t];
    if (logits_out) logits_out[(size_t)g * V + t] = v;
    if (t == mask_id) continue;
    if (v > m || (v == m && t < a)) { m = v; a = t; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float v = __shfl_xor(m, o, 64);
    const int id = __shfl_xor(a, o, 64);
    if (v > m || (v == m && id < a)) { m = v; a = id; }
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { rm[w] = m; ra[w] = a; }
  __syncthreads();
  m = rm[0]; a = ra[0];
  for (int i = 1; i < kThreads / 64; ++i)
    if (rm[i] > m || (rm[i] == m && ra[i] < a)) { m = rm[i]; a = ra[i]; }
  float s = 0.f;
  for (int t = threadIdx.x; t < V; t += kThreads)
    if (t != mask_id) s += expf(lg[t] - m);
  s = block_sum(s, red);
  if (threadIdx.x == 0) {
    conf_out[g] = 1.0f / s;
    argmax_out[g] = a;
  }
}

// ---- split-K reductions: partial tiles P[k][row][col] summed in k order
// (fixed order: deterministic), 8-column chunks, every load of a chunk issued
// before the first add.
template <int KS>
__device__ __forceinline__ void sum_parts(const float* __restrict__ p,
                                          size_t stride, float* v) {
  float t[KS][8];
#pragma unroll
  for (int k = 0; k < KS; ++k) load8f(p + k * stride, t[k]);
#pragma unroll
  for (int k = 0; k < KS; ++k)
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += t[k][i];
}

// X[row] += sum_k P[k][row]; then A[row] = RMSNorm(X[row]) * gain if A given.
template <typename Fmt, int KS, typename T = typename Fmt::st>
__global__ void __launch_bounds__(kThreads)
reduce_add_norm_kernel(const float* __restrict__ P, int rows, int d,
                       float* __restrict__ X, const float* __restrict__ gain,
                       float eps, T* __restrict__ A) {
  __shared__ float red[kThreads / 64];
  const int row = blockIdx.x;
  const size_t stride = (size_t)rows * d;
  const int nc = d / 8;
  float v[kMaxChunks][8];
  float ss = 0.f;
#pragma unroll
  for (int n = 0; n < kMaxChunks; ++n) {
    const int c = threadIdx.x + n * kThreads;
    if (c < nc) {
      float* xr = X + (size_t)row * d + c * 8;
      load8f(xr, v[n]);
      sum_parts<KS>(P + (size_t)row * d + c * 8, stride, v[n]);
      store8f(xr, v[n]);
#pragma unroll
      for (int i = 0; i < 8; ++i) ss += v[n][i] * v[n][i];
    }
  }
  if (!A) return;
  norm_store<Fmt>(v, ss, d, gain, eps, A + (size_t)row * d, red);
}

// X[row] += sum_k P[k][row]; a masked response row also gets
// Hm[slot] = RMSNorm(X[row]) * gain (slot: its index in the masked-row list):
// the final norm and gather of the masked rows, fused into the split-K
// reduction of the last layer.
template <typename Fmt, int KS, typename T = typename Fmt::st>
__global__ void __launch_bounds__(kThreads)
reduce_add_gather_kernel(const float* __restrict__ P, int rows, int d,
                         float* __restrict__ X, SeqPack sp,
                         const int32_t* __restrict__ slot,
                         const float* __restrict__ gain, float eps,
                         T* __restrict__ Hm) {
  __shared__ float red[kThreads / 64];
  const int row = blockIdx.x;
  const size_t stride = (size_t)rows * d;
  const int nc = d / 8;
  float v[kMaxChunks][8];
  float ss = 0.f;
#pragma unroll
  for (int n = 0; n < kMaxChunks; ++n) {
    const int c = threadIdx.x + n * kThreads;
    if (c < nc) {
      float* xr = X + (size_t)row * d + c * 8;
      load8f(xr, v[n]);
      sum_parts<KS>(P + (size_t)row * d + c * 8, stride, v[n]);
      store8f(xr, v[n]);
#pragma unroll
      for (int i = 0; i < 8; ++i) ss += v[n][i] * v[n][i];
    }
  }
  // the same for every thread of the workgroup: the row's response index
  const int s = find_seq(sp, row);
  const int i = row - (sp.row0[s] + sp.nview[s] + sp.plen[s]);
  if (i < 0 || i >= sp.L) return;
  const int j = slot[s * sp.L + i];
  if (j < 0) return;
  norm_store<Fmt>(v, ss, d, gain, eps, Hm + (size_t)j * d, red);
}

// columns < rope_cols hold heads of 128 dims rotated as (i, i + 64)
template <typename Fmt, int KS, typename T = typename Fmt::st>
__global__ void __launch_bounds__(kThreads)
reduce_store_rope_kernel(const float* __restrict__ P, int rows, int ncols,
                         int rope_cols, const int32_t* __restrict__ pos,
                         const float2* __restrict__ cs, T* __restrict__ out,
                         int32_t* __restrict__ overflow) {
  int nf = 0;
  const int row = blockIdx.x;
  const size_t stride = (size_t)rows * ncols;
  const float* pr = P + (size_t)row * ncols;
  T* o = out + (size_t)row * ncols;
  const int p0 = pos[row];
  // rotated pairs: chunk q covers dims i0..i0+7 and i0+64..i0+71 of a head
  const int npairs = rope_cols / 16;
  for (int q = threadIdx.x; q < npairs; q += kThreads) {
    const int i0 = (q % 8) * 8;
    const int c1 = (q / 8) * 128 + i0, c2 = c1 + 64;
    float x[8] = {0, 0, 0, 0, 0, 0, 0, 0}, y[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    sum_parts<KS>(pr + c1, stride, x);
    sum_parts<KS>(pr + c2, stride, y);
    float cv[8], sv[8];
    const float4* cp = reinterpret_cast<const float4*>(cs + (size_t)p0 * 64 + i0);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float4 t = cp[u];
      cv[2 * u] = t.x; sv[2 * u] = t.y; cv[2 * u + 1] = t.z; sv[2 * u + 1] = t.w;
    }
    float a[8], b[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[i] = x[i] * cv[i] - y[i] * sv[i];
      b[i] = y[i] * cv[i] + x[i] * sv[i];
    }
    nf += store8_count<Fmt>(o + c1, a);
    nf += store8_count<Fmt>(o + c2, b);
  }
  for (int c = rope_cols + threadIdx.x * 8; c < ncols; c += kThreads * 8) {
    float x[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    sum_parts<KS>(pr + c, stride, x);
    nf += store8_count<Fmt>(o + c, x);
  }
  if (nf && overflow) atomicAdd(overflow, nf);
}

template <typename Fmt, int KS, typename T = typename Fmt::st>
__global__ void __launch_bounds__(kThreads)
reduce_swiglu_kernel(const float* __restrict__ P, int rows, int ffn,
                     T* __restrict__ out, int32_t* __restrict__ overflow) {
  int nf = 0;
  const int row = blockIdx.x;
  const size_t ld = (size_t)2 * ffn;
  const size_t stride = (size_t)rows * ld;
  const float* pr = P + (size_t)row * ld;
  for (int c = threadIdx.x * 8; c < ffn; c += kThreads * 8) {
    float g[8] = {0, 0, 0, 0, 0, 0, 0, 0}, u[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    sum_parts<KS>(pr + c, stride, g);
    sum_parts<KS>(pr + ffn + c, stride, u);
    float h[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = g[i] / (1.0f + __expf(-g[i])) * u[i];
    nf += store8_count<Fmt>(out + (size_t)row * ffn + c, h);
  }
  if (nf && overflow) atomicAdd(overflow, nf);
}

// Element-type conversion through float32 (exact for the 16-bit sources),
// rounding to nearest even into the destination format.
template <typename Src, typename Dst>
__global__ void __launch_bounds__(256)
convert_kernel(const typename Src::st* __restrict__ src,
               typename Dst::st* __restrict__ dst, size_t n) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += stride)
    dst[i] = Dst::store(Src::load(src[i]));
}

// Tiled vocabulary head: thread q writes the 16 bytes (8 elements) at
// tiled[8q .. 8q+8): tile (c, s), row r, elements 8u .. 8u+7 of the 64.
__global__ void __launch_bounds__(256)
pack_head_kernel(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst,
                 int vocab, int d, int n_slabs, size_t n_vec) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t q = (size_t)blockIdx.x * blockDim.x + threadIdx.x; q < n_vec;
       q += stride) {
    const int u = (int)(q & 7);
    const size_t rq = q >> 3;                   // row of a tile, globally
    const int r = (int)(rq & 127);
    const size_t tile = rq >> 7;                // c * n_slabs + s
    const int sl = (int)(tile % n_slabs);
    const int c = (int)(tile / n_slabs);
    const int n = sl * 128 + r;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (n < vocab)
      v = *reinterpret_cast<const u32x4*>(src + (size_t)n * d + c * 64 + u * 8);
    *reinterpret_cast<u32x4*>(dst + q * 8) = v;
  }
}

template <typename Src>
int convert_from(const void* src, void* dst, int dst_dtype, size_t n,
                 hipStream_t s) {
  const size_t blocks = std::min<size_t>((n + 255) / 256, 65536);
#define CV(D)                                                           \
  hipLaunchKernelGGL((convert_kernel<Src, D>), dim3(blocks), dim3(256), 0, s, \
                     (const typename Src::st*)src, (D::st*)dst, n)
  if (dst_dtype == DAVET_F16) CV(F16S);
  else if (dst_dtype == DAVET_BF16) CV(BF16S);
  else CV(F32S);
#undef CV
  return DAVET_OK;
}

}  // namespace

int launch_convert(const void* src, int src_dtype, void* dst, int dst_dtype,
                   size_t n, hipStream_t s) {
  if (n == 0) return DAVET_OK;
  ProfScope ps(KC_MISC, s);
  if (src_dtype == DAVET_BF16) convert_from<BF16S>(src, dst, dst_dtype, n, s);
  else if (src_dtype == DAVET_F16) convert_from<F16S>(src, dst, dst_dtype, n, s);
  else convert_from<F32S>(src, dst, dst_dtype, n, s);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

#define DISPATCH16(dtype, F_BODY)                                           \
  do {                                                                      \
    if ((dtype) == DAVET_F16) { using F = F16S; F_BODY; }                   \
    else { using F = BF16S; F_BODY; }                                       \
  } while (0)

#define DISPATCH_KS(ksplit, BODY)                                           \
  do {                                                                      \
    switch (ksplit) {                                                       \
      case 2: { constexpr int KS = 2; BODY; } break;                        \
      case 3: { constexpr int KS = 3; BODY; } break;                        \
      case 4: { constexpr int KS = 4; BODY; } break;                        \
      case 5: { constexpr int KS = 5; BODY; } break;                        \
      case 6: { constexpr int KS = 6; BODY; } break;                        \
      case 8: { constexpr int KS = 8; BODY; } break;                        \
      default: return set_error(DAVET_EINVAL,                              \
                                "split-K: ksplit must be 2, 3, 4, 5, 6 or 8"); \
    }                                                                       \
  } while (0)

int launch_reduce_add_norm(int dtype, const float* P, int ksplit, int rows,
                           int d, float* X, const float* gain, float eps,
                           void* A, hipStream_t s) {
  if (rows <= 0) return DAVET_OK;
  ProfScope ps(KC_RMSNORM, s);
  DISPATCH16(dtype, DISPATCH_KS(ksplit, hipLaunchKernelGGL(
      (reduce_add_norm_kernel<F, KS>), dim3(rows), dim3(kThreads), 0, s, P,
      rows, d, X, gain, eps, (F::st*)A)));
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_reduce_add_gather(int dtype, const float* P, int ksplit, int rows,
                             int d, float* X, const SeqPack& sp,
                             const int32_t* slot, const float* gain, float eps,
                             void* Hm, hipStream_t s) {
  if (rows <= 0) return DAVET_OK;
  ProfScope ps(KC_RMSNORM, s);
  DISPATCH16(dtype, DISPATCH_KS(ksplit, hipLaunchKernelGGL(
      (reduce_add_gather_kernel<F, KS>), dim3(rows), dim3(kThreads), 0, s, P,
      rows, d, X, sp, slot, gain, eps, (F::st*)Hm)));
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_reduce_store_rope(int dtype, const float* P, int ksplit, int rows,
                             int ncols, int rope_cols, const int32_t* pos,
                             const float* cs, void* out, hipStream_t s,
                             int32_t* overflow) {
  if (rows <= 0) return DAVET_OK;
  if (rope_cols % 128 || ncols % 8)
    return set_error(DAVET_ESHAPE, "reduce_store_rope: column counts");
  ProfScope ps(KC_ROPE, s);
  DISPATCH16(dtype, DISPATCH_KS(ksplit, hipLaunchKernelGGL(
      (reduce_store_rope_kernel<F, KS>), dim3(rows), dim3(kThreads), 0, s, P,
      rows, ncols, rope_cols, pos, (const float2*)cs, (F::st*)out,
      overflow)));
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_reduce_swiglu(int dtype, const float* P, int ksplit, int rows,
                         int ffn, void* out, hipStream_t s, int32_t* overflow) {
  if (rows <= 0) return DAVET_OK;
  if (ffn % 8) return set_error(DAVET_ESHAPE, "reduce_swiglu: ffn % 8 != 0");
  ProfScope ps(KC_MISC, s);
  DISPATCH16(dtype, DISPATCH_KS(ksplit, hipLaunchKernelGGL(
      (reduce_swiglu_kernel<F, KS>), dim3(rows), dim3(kThreads), 0, s, P, rows,
      ffn, (F::st*)out, overflow)));
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}
#undef DISPATCH_KS

int launch_assemble_norm(const SeqPack& sp, const ViewPtrs& vp, int dtype,
                         const void* embed, const int32_t* prompt_ids,
                         const int32_t* resp_ids, const uint8_t* masked,
                         int mask_id, int vocab, int d, const float* gain,
                         float eps, float* X, void* A, int32_t* pos,
                         const RowList& rl, hipStream_t s) {
  ProfScope ps(KC_ASSEMBLE, s);
#define ASM(F)                                                               \
  hipLaunchKernelGGL(assemble_norm_kernel<F>, dim3(sp.total + 1),             \
                     dim3(kThreads), 0, s, sp, vp, (const F::st*)embed,       \
                     prompt_ids, resp_ids, masked, mask_id, vocab, d, gain,   \
                     eps, X, (F::st*)A, pos, rl)
  if (dtype == DAVET_BF16) ASM(BF16S);
  else if (dtype == DAVET_F16) ASM(F16S);
  else ASM(F32S);
#undef ASM
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_rmsnorm(const float* X, int rows, int d, const float* gain,
                   float eps, int dtype, void* A, hipStream_t s) {
  ProfScope ps(KC_RMSNORM, s);
#define RMS(F)                                                             \
  hipLaunchKernelGGL(rmsnorm_kernel<F>, dim3(rows), dim3(kThreads), 0, s, X, \
                     d, gain, eps, (F::st*)A)
  if (dtype == DAVET_BF16) RMS(BF16S);
  else if (dtype == DAVET_F16) RMS(F16S);
  else RMS(F32S);
#undef RMS
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_rope_table(int max_pos, int head_dim, float theta, float* cs,
                      hipStream_t s) {
  ProfScope ps(KC_MISC, s);
  const int n = max_pos * (head_dim / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3((n + 255) / 256), dim3(256), 0, s,
                     max_pos, head_dim, (double)theta, (float2*)cs);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_rope(void* qkv, int rows, int n_heads, int head_dim, int dtype,
                const SeqPack& sp, const float* cs, hipStream_t s) {
  ProfScope ps(KC_ROPE, s);
#define ROPE(F)                                                             \
  hipLaunchKernelGGL(rope_kernel<F>, dim3(rows), dim3(kThreads), 0, s,        \
                     (F::st*)qkv, sp, n_heads, head_dim, (const float2*)cs)
  if (dtype == DAVET_BF16) ROPE(BF16S);
  else if (dtype == DAVET_F16) ROPE(F16S);
  else ROPE(F32S);
#undef ROPE
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_final_norm_gather(const float* X, const SeqPack& sp,
                             const int32_t* list, int max_rows, int d,
                             const float* gain, float eps, int dtype, void* Hm,
                             hipStream_t s) {
  ProfScope ps(KC_HEAD_PREP, s);
#define FNG(F)                                                              \
  hipLaunchKernelGGL(final_norm_gather_kernel<F>, dim3(max_rows),            \
                     dim3(kThreads), 0, s, X, sp, list, d, gain, eps,         \
                     (F::st*)Hm)
  if (dtype == DAVET_BF16) FNG(BF16S);
  else if (dtype == DAVET_F16) FNG(F16S);
  else FNG(F32S);
#undef FNG
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_head_merge(const int32_t* list, int max_rows, int n_slabs,
                      const float* pmax, const float* psum, const int32_t* parg,
                      float* conf_out, int32_t* argmax_out, hipStream_t s) {
  ProfScope ps(KC_HEAD_MERGE, s);
  hipLaunchKernelGGL(head_merge_kernel, dim3(max_rows), dim3(kThreads), 0, s,
                     list, n_slabs, pmax, psum, parg, conf_out, argmax_out);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_head_reduce_f32(const float* logits, const int32_t* list,
                           int max_rows, int vocab, int mask_id,
                           float* conf_out, int32_t* argmax_out,
                           float* logits_out, hipStream_t s) {
  ProfScope ps(KC_HEAD_MERGE, s);
  hipLaunchKernelGGL(head_reduce_f32_kernel, dim3(max_rows), dim3(kThreads), 0,
                     s, logits, list, vocab, mask_id, conf_out, argmax_out,
                     logits_out);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_pack_head(const uint16_t* src, uint16_t* dst, int vocab, int d,
                     hipStream_t s) {
  ProfScope ps(KC_MISC, s);
  const int n_slabs = (vocab + 127) / 128;
  const size_t n_vec = (size_t)n_slabs * 128 * d / 8;
  const size_t blocks = std::min<size_t>((n_vec + 255) / 256, 65536);
  hipLaunchKernelGGL(pack_head_kernel, dim3(blocks), dim3(256), 0, s, src, dst,
                     vocab, d, n_slabs, n_vec);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

}  // namespace davet

extern "C" size_t davet_head_tiled_elems(int32_t vocab, int32_t d) {
  if (vocab < 1 || d < 1) return 0;
  return (size_t)((vocab + 127) / 128) * 128 * (size_t)d;
}

extern "C" int davet_pack_head(const void* src, void* dst, int32_t vocab,
                               int32_t d, int32_t dtype, hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(src && dst, DAVET_EINVAL, "davet_pack_head: null pointer");
  DAVET_CHECK_ARG(is16(dtype), DAVET_EDTYPE,
                  "davet_pack_head: dtype must be DAVET_BF16 or DAVET_F16");
  DAVET_CHECK_ARG(vocab >= 1 && d >= 64 && d % 64 == 0, DAVET_ESHAPE,
                  "davet_pack_head: vocab >= 1, d >= 64 and d % 64 == 0");
  DAVET_CHECK_ARG(((uintptr_t)src & 15) == 0 && ((uintptr_t)dst & 15) == 0,
                  DAVET_EINVAL, "davet_pack_head: buffers must be 16-byte aligned");
  const char* s0 = static_cast<const char*>(src);
  const char* d0 = static_cast<const char*>(dst);
  const size_t sb = (size_t)vocab * d * 2;
  const size_t db = davet_head_tiled_elems(vocab, d) * 2;
  DAVET_CHECK_ARG(s0 + sb <= d0 || d0 + db <= s0, DAVET_EINVAL,
                  "davet_pack_head: src and dst overlap");
  return launch_pack_head(static_cast<const uint16_t*>(src),
                          static_cast<uint16_t*>(dst), vocab, d, stream);
}

extern "C" int davet_convert(const void* src, int32_t src_dtype, void* dst,
                             int32_t dst_dtype, size_t n, hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(n == 0 || (src && dst), DAVET_EINVAL,
                  "davet_convert: null pointer");
  auto ok = [](int t) {
    return t == DAVET_F32 || t == DAVET_BF16 || t == DAVET_F16;
  };
  DAVET_CHECK_ARG(ok(src_dtype) && ok(dst_dtype), DAVET_EDTYPE,
                  "davet_convert: unknown dtype");
  const char* s0 = static_cast<const char*>(src);
  const char* d0 = static_cast<const char*>(dst);
  const size_t sb = n * dtype_size(src_dtype), db = n * dtype_size(dst_dtype);
  DAVET_CHECK_ARG(s0 + sb <= d0 || d0 + db <= s0, DAVET_EINVAL,
                  "davet_convert: src and dst overlap");
  return launch_convert(src, src_dtype, dst, dst_dtype, n, stream);
}
