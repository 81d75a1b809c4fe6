// Internal helpers shared by the HIP sources of the DAVET library (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string>

#include "davet.h"

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

namespace davet {

// ---- error reporting (host) ------------------------------------------------
int set_error(int status, const std::string& msg);
#define DAVET_CHECK_ARG(cond, status, msg) \
  do { if (!(cond)) return ::davet::set_error((status), (msg)); } while (0)
#define DAVET_HIP(call)                                                     \
  do {                                                                      \
    hipError_t e_ = (call);                                                 \
    if (e_ != hipSuccess)                                                   \
      return ::davet::set_error(DAVET_EHIP, std::string(#call) + ": " +    \
                                hipGetErrorString(e_));                     \
  } while (0)

// ---- per-kernel-class launch timing (host) ---------------------------------
enum KernelClass {
  KC_VIEWS = 0, KC_VIEW_MAPS, KC_ASSEMBLE, KC_RMSNORM, KC_GEMM_QKV, KC_ROPE,
  KC_ATTN, KC_GEMM_O, KC_GEMM_GATEUP, KC_GEMM_DOWN, KC_HEAD_PREP, KC_HEAD,
  KC_HEAD_MERGE, KC_UNMASK, KC_GEMM_F32, KC_ATTN_F32, KC_MISC,
  KC_REALIZER_KEYS, KC_REALIZER_MAPS, KC_COUNT
};
const char* kernel_class_name(int c);
// Brackets a launch with events when profiling is on; cheap no-op otherwise.
struct ProfScope {
  ProfScope(int cls, hipStream_t s);
  ~ProfScope();
  int slot;
  hipStream_t stream;
};

// ---- bf16 helpers (device) -------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}
// float32 -> bf16, round to nearest even (finite values; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
// float64 -> bf16 in a single rounding step (nearest, ties to even); normal
// range values.  Keeps 7 of the 52 explicit mantissa bits of the double.
__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
  uint64_t b = (uint64_t)__double_as_longlong(x);
  uint64_t lsb = (b >> 45) & 1ull;
  b = (b + ((1ull << 44) - 1ull) + lsb) & ~((1ull << 45) - 1ull);
  float f = (float)__longlong_as_double((long long)b);   // exact
  return (uint16_t)(__float_as_uint(f) >> 16);
}

// float64 -> float32 with round-to-odd: truncate toward zero and set the last
// mantissa bit when inexact.  A later round-to-nearest-even to a format with
// at least 2 fewer mantissa bits then equals one correct rounding of x.
__device__ __forceinline__ float f64_to_f32_odd(double x) {
  float f = (float)x;
  const double back = (double)f;
  if (back == x || x != x) return f;
  if (fabs(back) > fabs(x))                       // rounded away from zero
    f = __uint_as_float(__float_as_uint(f) - 1u);
  return __uint_as_float(__float_as_uint(f) | 1u);
}
__device__ __forceinline__ uint16_t f32_to_f16(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);   // RNE
}
__device__ __forceinline__ float f16_to_f32(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}
// float64 -> fp16 with a single rounding (nearest even), subnormals included.
__device__ __forceinline__ uint16_t f64_to_f16(double x) {
  return f32_to_f16(f64_to_f32_odd(x));
}

// 16-bit operand formats of the matrix-core path.  Both are stored as
// uint16_t bit patterns; fp32 accumulation in both.
struct BF16 {
  using v8 = bf16x8;
  static constexpr int dtype = DAVET_BF16;
  __device__ static __forceinline__ float load(uint16_t b) { return bf16_to_f32(b); }
  __device__ static __forceinline__ uint16_t store(float f) { return f32_to_bf16(f); }
  // two values rounded (nearest even) into one word, a in the low half
  __device__ static __forceinline__ uint32_t store2(float a, float b) {
    return (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
  }
  __device__ static __forceinline__ uint16_t from_f64(double x) { return f64_to_bf16(x); }
  // 1 when a stored value is not finite (all exponent bits set)
  __device__ static __forceinline__ int nonfinite(uint16_t h) {
    return (h & 0x7f80u) == 0x7f80u;
  }
  __device__ static __forceinline__ f32x16 mfma32(v8 a, v8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ f32x4 mfma16(v8 a, v8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
struct F16 {
  using v8 = f16x8;
  static constexpr int dtype = DAVET_F16;
  __device__ static __forceinline__ float load(uint16_t h) { return f16_to_f32(h); }
  __device__ static __forceinline__ uint16_t store(float f) { return f32_to_f16(f); }
  // two values rounded (nearest even) into one word, a in the low half: one
  // packed conversion (v_cvt_pk_f16_f32) instead of two and a merge
  __device__ static __forceinline__ uint32_t store2(float a, float b) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    const f2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
  }
  __device__ static __forceinline__ uint16_t from_f64(double x) { return f64_to_f16(x); }
  // 1 when a stored value is not finite: for fp16 a result above 65504 in
  // magnitude (after rounding) became +-inf
  __device__ static __forceinline__ int nonfinite(uint16_t h) {
    return (h & 0x7c00u) == 0x7c00u;
  }
  __device__ static __forceinline__ f32x16 mfma32(v8 a, v8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ f32x4 mfma16(v8 a, v8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
};

// Storage formats for row kernels: element type in memory plus conversions.
struct F32S {
  using st = float;
  static constexpr int dtype = DAVET_F32;
  __device__ static __forceinline__ float load(float x) { return x; }
  __device__ static __forceinline__ float store(float x) { return x; }
};
struct BF16S : BF16 { using st = uint16_t; };
struct F16S : F16 { using st = uint16_t; };

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float warp_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

inline size_t dtype_size(int dt) { return dt == DAVET_F32 ? 4 : 2; }
inline bool is16(int dt) { return dt == DAVET_BF16 || dt == DAVET_F16; }
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---- kernel launchers (host, defined next to their kernels) ----------------
// Views
int launch_views(const davet_view_geom& g, const void* v, void* const* levels,
                 hipStream_t s);
int launch_view_maps(const davet_view_geom& g, int32_t* const* offs,
                     int32_t* const* mem, hipStream_t s);
// Geometry checks shared by every view entry point (EINVAL/ESHAPE).
int check_view_geom(const davet_view_geom* g, const char* who);
// Prune / merge realizers: scratch size and the whole build (keys, maps,
// levels) into caller scratch.
size_t realizer_scratch_bytes(const davet_view_geom& g);
int build_views_realizer(const davet_view_geom& g, const void* v,
                         void* const* levels, int32_t* const* offs,
                         int32_t* const* mem, void* scratch,
                         size_t scratch_bytes, hipStream_t s);

// Packed-batch description passed by value to kernels.
struct SeqPack {
  int32_t n_seqs;
  int32_t L;
  int32_t total;                       // sum of N_s
  int32_t row0[DAVET_MAX_SEQS + 1];    // first packed row of each sequence
  int32_t nview[DAVET_MAX_SEQS];
  int32_t pstart[DAVET_MAX_SEQS];      // offset into prompt_ids
  int32_t plen[DAVET_MAX_SEQS];
};
struct ViewPtrs { const void* p[DAVET_MAX_SEQS]; };

// Row kernels
// The masked response positions of a step (total = n_seqs * L): list[0] =
// their count, list[1 + j] = the j-th in index order; slot[i] = i's index in
// the list or -1 (may be null); committed positions get conf = -inf and
// argmax = -1.
struct RowList {
  int total;
  int32_t* list;
  float* conf;
  int32_t* argmax;
  int32_t* slot;
  int32_t* overflow;      // the step's 16-bit overflow counter (may be null)
  int clear_overflow;     // the list builder zeroes it first
};
// assembly + first norm of every packed row; one extra workgroup builds the
// masked-row list alongside
int launch_assemble_norm(const SeqPack& sp, const ViewPtrs& vp, int dtype,
                         const void* embed, const int32_t* prompt_ids,
                         const int32_t* resp_ids, const uint8_t* masked,
                         int mask_id, int vocab, int d, const float* gain,
                         float eps, float* X, void* A, int32_t* pos,
                         const RowList& rl, hipStream_t s);
int launch_rmsnorm(const float* X, int rows, int d, const float* gain,
                   float eps, int dtype, void* A, hipStream_t s);
int launch_rope_table(int max_pos, int head_dim, float theta, float* cs,
                      hipStream_t s);
int launch_rope(void* qkv, int rows, int n_heads, int head_dim, int dtype,
                const SeqPack& sp, const float* cs, hipStream_t s);
int launch_final_norm_gather(const float* X, const SeqPack& sp,
                             const int32_t* list, int max_rows, int d,
                             const float* gain, float eps, int dtype, void* Hm,
                             hipStream_t s);
int launch_head_merge(const int32_t* list, int max_rows, int n_slabs,
                      const float* pmax, const float* psum, const int32_t* parg,
                      float* conf_out, int32_t* argmax_out, hipStream_t s);
int launch_head_reduce_f32(const float* logits, const int32_t* list,
                           int max_rows, int vocab, int mask_id,
                           float* conf_out, int32_t* argmax_out,
                           float* logits_out, hipStream_t s);

// GEMMs: C[M,N] = A[M,K] * B[N,K]^T
enum Epilogue { EPI_STORE = 0, EPI_ADD_F32 = 1, EPI_SWIGLU = 2 };
struct GemmPlan {
  int tile;      // kernel variant (tile shape, K slab, stages, waves)
  int ksplit;    // > 1: fp32 partials [ksplit][M][N] + a reduction kernel
};
// Tile shape and K split for an M x N x K product (N = 2*ffn for SwiGLU).
GemmPlan plan_gemm16(int M, int N, int K);
// 16-bit GEMM with fused epilogue.  EPI_STORE applies the rotary embedding to
// columns < rope_cols using pos[row] and the cos/sin table cs when pos is
// given.  With plan.ksplit > 1 the kernel writes fp32 partials to `partials`
// and the caller runs the matching reduce kernel below.
// overflow (may be null): every 16-bit value the EPI_STORE / EPI_SWIGLU
// epilogue stores as non-finite adds 1 to *overflow.
int launch_gemm16(int dtype, int epi, const GemmPlan& plan, const uint16_t* A,
                  const uint16_t* B, const uint16_t* B2, void* C, int M, int N,
                  int K, int ldc, const int32_t* pos, const float* cs,
                  int rope_cols, float* partials, size_t partial_cap, int cls,
                  hipStream_t s, int32_t* overflow = nullptr);
// Largest fp32 split-K partial buffer (bytes) plan_gemm16 may ask for with
// M <= max_M rows of an N x K product.
size_t gemm16_partial_bound(int max_M, int N, int K);
// Split-K reductions (fixed summation order over the splits):
//   X[r] += sum_s P[s][r]; then A[r] = RMSNorm(X[r]) * gain when A is given
int launch_reduce_add_norm(int dtype, const float* P, int ksplit, int rows,
                           int d, float* X, const float* gain, float eps,
                           void* A, hipStream_t s);
//   X[r] += sum_s P[s][r]; then Hm[slot] = RMSNorm(X[r]) * gain for a masked
//   response row r (the last layer's final norm and gather)
int launch_reduce_add_gather(int dtype, const float* P, int ksplit, int rows,
                             int d, float* X, const SeqPack& sp,
                             const int32_t* slot, const float* gain, float eps,
                             void* Hm, hipStream_t s);
//   out16[r][c] = rope(sum_s P[s][r][c]) for c < rope_cols, plain otherwise
int launch_reduce_store_rope(int dtype, const float* P, int ksplit, int rows,
                             int ncols, int rope_cols, const int32_t* pos,
                             const float* cs, void* out, hipStream_t s,
                             int32_t* overflow = nullptr);
//   out16[r][c] = silu(sum_s P[s][r][c]) * sum_s P[s][r][F + c]
int launch_reduce_swiglu(int dtype, const float* P, int ksplit, int rows,
                         int ffn, void* out, hipStream_t s,
                         int32_t* overflow = nullptr);
// Vocabulary head over the masked rows: the tile follows the weight layout
// (tiled: davet_pack_head blocks) and live_bound, a host-side bound on the
// live rows (-1: max_rows)
int launch_head16(int dtype, const uint16_t* Hm, const uint16_t* W,
                  const int32_t* list, int max_rows, int vocab, int d,
                  int mask_id, float* pmax, float* psum, int32_t* parg,
                  float* logits_out, hipStream_t s, int tiled = 0,
                  int live_bound = -1);
// vocabulary slabs per row (pmax/psum/parg columns) the head launch for this
// layout and live-row bound writes; at most ceil(V / 128)
int head16_slabs(int vocab, int tiled = 0, int live_bound = 1);
int launch_gemm_f32(int epi, const float* A, const float* B, const float* B2,
                    float* C, int M, int N, int K, int ldc, int cls,
                    const int32_t* m_count, hipStream_t s);

// Attention over the packed batch: qkv [total, 3d] -> o [total, d]
// Key-range split of the 16-bit attention: a query tile's keys may be
// divided among up to ATT_MAX_SPLIT workgroups, each writing one partial slot
// of ATT_SLOT_FLOATS floats (O^T as [128 dims][128 queries], then max and
// normaliser as [2][128]) into `part`; at most ATT_MAX_SLOTS slots.
constexpr int ATT_MAX_SPLIT = 8;
constexpr int ATT_MAX_SLOTS = 1024;
constexpr int ATT_SLOT_FLOATS = 128 * 128 + 2 * 128;
// Partial bytes a launch over at most `tokens` rows in `seqs` sequences may use.
size_t attention_part_bytes(int64_t tokens, int64_t seqs, int n_heads);
int launch_attention16(int dtype, const uint16_t* qkv, uint16_t* o,
                       const SeqPack& sp, int n_heads, int head_dim,
                       float* part, size_t part_bytes, hipStream_t s);
int launch_convert(const void* src, int src_dtype, void* dst, int dst_dtype,
                   size_t n, hipStream_t s);
int launch_attention_f32(const float* qkv, float* o, const SeqPack& sp,
                         int n_heads, int head_dim, hipStream_t s);

int launch_unmask(int n_seqs, int L, int k, const float* conf,
                  const int32_t* argmax, int32_t* ids, uint8_t* masked,
                  int32_t* selected, hipStream_t s);

}  // namespace davet
