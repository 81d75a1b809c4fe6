// Evidence hierarchy by per-crop average pooling (Sec. 4.3, "Ordered evidence
// hierarchy"; v^(K) = v).  One pass over v builds every pooled level: a thread
// owns 2 to 8 consecutive features of one coarsest window and visits that
// window's tokens once, in row-major order, adding each into the running
// float64 sum of the sub-window it belongs to at every finer level.  Each
// level token is then (sum / member count) rounded once to the view dtype.
// HBM-bound: v is read once, the levels are written once.  Every token of a
// thread's window is loaded before any is summed, so a thread has the whole
// window in flight.
//
// Mixed view (K = 3, stride S): level 1 becomes, per crop, the level-0 tokens
// followed by the raw tokens on the lattice (o + aS, o + bS), o = S/2.  The
// same pass writes each level-0 token twice and copies each lattice token's
// bits from v; the 2x2 sums are not formed.

#include "common.h"

namespace davet {
namespace {

struct LevelOut { void* p[DAVET_MAX_LEVELS]; };


// lattice length of a crop: #{o, o + S, ... < G}, o = S / 2
__host__ __device__ inline int lattice_len(int G, int S) {
  const int o = S / 2;
  return o < G ? (G - o + S - 1) / S : 0;
}

template <int K, int VEC, typename Fmt, bool MIXED>
__global__ void __launch_bounds__(256)
pool_views_kernel(const typename Fmt::st* __restrict__ v, LevelOut out,
                  int n_crops, int G, int d, int S) {
  static_assert(!MIXED || K == 3, "the mixed view is defined for K = 3");
  using T = typename Fmt::st;
  constexpr int F = 1 << (K - 1);                 // coarsest window side
  const int Wc = (G + F - 1) / F;
  const int win = blockIdx.x;                     // coarsest window id
  const int c = win / (Wc * Wc);
  const int I = (win / Wc) % Wc;
  const int J = win % Wc;
  const int e0 = (blockIdx.y * blockDim.x + threadIdx.x) * VEC;
  if (e0 >= d) return;

  // accumulators: level l has (F / f_l)^2 sub-windows, f_l = 2^(K-1-l)
  constexpr int NACC = (K == 2) ? 1 : (K == 3) ? 5 : 21;
  double acc[NACC][VEC];
#pragma unroll
  for (int a = 0; a < NACC; ++a)
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[a][e] = 0.0;

  const int r0 = I * F, s0 = J * F;
  // Every token of the window is loaded before any is summed (F*F loads in
  // flight per thread instead of one memory round trip per token); tokens
  // past the grid edge load a clamped in-bounds row and add +0.0, an exact
  // no-op on a sum that starts at +0.0, so the sums are the member sums in
  // member order bit for bit.
  constexpr int WORDS = VEC * (int)sizeof(T) / 4;   // 32-bit words per load
  uint32_t raw[F * F][WORDS];
#pragma unroll
  for (int dr = 0; dr < F; ++dr) {
#pragma unroll
    for (int ds = 0; ds < F; ++ds) {
      const int r = min(r0 + dr, G - 1), s = min(s0 + ds, G - 1);
      const T* src = v + ((size_t)c * G * G + (size_t)r * G + s) * d + e0;
      if constexpr (WORDS % 4 == 0) {
#pragma unroll
        for (int q4 = 0; q4 < WORDS / 4; ++q4) {
          const u32x4 w = reinterpret_cast<const u32x4*>(src)[q4];
#pragma unroll
          for (int q = 0; q < 4; ++q) raw[dr * F + ds][q4 * 4 + q] = w[q];
        }
      } else if constexpr (WORDS == 2) {
        const u32x2 w = *reinterpret_cast<const u32x2*>(src);
        raw[dr * F + ds][0] = w[0];
        raw[dr * F + ds][1] = w[1];
      } else {
        static_assert(WORDS == 1, "load width");
        raw[dr * F + ds][0] = *reinterpret_cast<const uint32_t*>(src);
      }
    }
  }
  // Fully unrolled so every accumulator index is a compile-time constant.
#pragma unroll
  for (int dr = 0; dr < F; ++dr) {
#pragma unroll
    for (int ds = 0; ds < F; ++ds) {
      const int r = r0 + dr, s = s0 + ds;
      const bool inb = r < G && s < G;
      const T* src = v + ((size_t)c * G * G + (size_t)r * G + s) * d + e0;
      double x[VEC];
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int q = 0; q < VEC / 2; ++q) {
          const uint32_t w = raw[dr * F + ds][q];
          x[2 * q] = inb ? (double)Fmt::load((uint16_t)(w & 0xffffu)) : 0.0;
          x[2 * q + 1] = inb ? (double)Fmt::load((uint16_t)(w >> 16)) : 0.0;
        }
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          x[e] = inb ? (double)__uint_as_float(raw[dr * F + ds][e]) : 0.0;
      }
      if constexpr (MIXED) {
        const int o = S / 2;
        if (inb && r % S == o && s % S == o) {    // lattice token: copy bits
          const int m = lattice_len(G, S);
          const size_t tok = (size_t)c * (Wc * Wc + m * m) + Wc * Wc +
                             (size_t)(r / S) * m + (s / S);
          T* dst = reinterpret_cast<T*>(out.p[1]) + tok * d + e0;
#pragma unroll
          for (int e = 0; e < VEC; ++e) dst[e] = src[e];
        }
      }
      int base = 0;
#pragma unroll
      for (int l = 0; l < (MIXED ? 1 : K - 1); ++l) {
        const int f = F >> l;                      // window side of level l
        const int per = F / f;                     // sub-windows per side
        const int a = base + (dr / f) * per + (ds / f);
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[a][e] += x[e];
        base += per * per;
      }
    }
  }
  int base = 0;
#pragma unroll
  for (int l = 0; l < (MIXED ? 1 : K - 1); ++l) {
    const int f = F >> l;
    const int per = F / f;
    const int W = (G + f - 1) / f;
#pragma unroll
    for (int a = 0; a < per; ++a) {
      const int i = I * per + a;
      if (i >= W) continue;
      const int rows = min(f, G - i * f);
#pragma unroll
      for (int b = 0; b < per; ++b) {
        const int j = J * per + b;
        if (j >= W) continue;
        const int cols = min(f, G - j * f);
        const double cnt = (double)(rows * cols);
        const size_t tok = (size_t)c * W * W + (size_t)i * W + j;
        double* ac = acc[base + a * per + b];
        // level-0 tokens of the mixed view sit at the head of their crop
        size_t tok_mix = 0;
        if constexpr (MIXED) {
          const int m = lattice_len(G, S);
          tok_mix = (size_t)c * (W * W + m * m) + (size_t)i * W + j;
        }
        if constexpr (sizeof(T) == 2) {
          uint16_t* dst = reinterpret_cast<uint16_t*>(out.p[l]) + tok * d + e0;
          uint16_t h[VEC];
#pragma unroll
          for (int e = 0; e < VEC; ++e) h[e] = Fmt::from_f64(ac[e] / cnt);
          if constexpr (VEC == 8) {
            u32x4 w;
#pragma unroll
            for (int q = 0; q < 4; ++q)
              w[q] = (uint32_t)h[2 * q] | ((uint32_t)h[2 * q + 1] << 16);
            *reinterpret_cast<u32x4*>(dst) = w;
            if constexpr (MIXED)
              *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(out.p[1]) +
                                        tok_mix * d + e0) = w;
          } else if constexpr (VEC == 4) {
            u32x2 w;
            w[0] = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
            w[1] = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
            *reinterpret_cast<u32x2*>(dst) = w;
            if constexpr (MIXED)
              *reinterpret_cast<u32x2*>(reinterpret_cast<uint16_t*>(out.p[1]) +
                                        tok_mix * d + e0) = w;
          } else {
            static_assert(VEC == 2, "store width");
            const uint32_t w = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
            *reinterpret_cast<uint32_t*>(dst) = w;
            if constexpr (MIXED)
              *reinterpret_cast<uint32_t*>(reinterpret_cast<uint16_t*>(out.p[1]) +
                                           tok_mix * d + e0) = w;
          }
        } else {
          float* dst = reinterpret_cast<float*>(out.p[l]) + tok * d + e0;
#pragma unroll
          for (int e = 0; e < VEC; e += 2) {
            float2 w;
            w.x = (float)(ac[e] / cnt);
            w.y = (float)(ac[e + 1] / cnt);
            *reinterpret_cast<float2*>(dst + e) = w;
            if constexpr (MIXED)
              *reinterpret_cast<float2*>(reinterpret_cast<float*>(out.p[1]) +
                                         tok_mix * d + e0 + e) = w;
          }
        }
      }
    }
    base += per * per;
  }
}

struct MapOut { int32_t* offs[DAVET_MAX_LEVELS]; int32_t* mem[DAVET_MAX_LEVELS]; };

// One thread per token of v; for every level it writes the token's slot in
// that level's member list and, for a window's first token, the window offset.
// The mixed level (S > 0, level 1) repeats level 0's lists crop by crop
// (crop stride G^2 + m^2 members, W^2 + m^2 tokens) and appends each lattice
// token as a one-member window.
__global__ void __launch_bounds__(256)
view_maps_kernel(MapOut mo, int n_crops, int G, int K, int S) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  const int total = n_crops * G * G;
  if (p >= total) return;
  const int c = p / (G * G);
  const int r = (p / G) % G;
  const int s = p % G;
  const int m = S > 0 ? lattice_len(G, S) : 0;
  for (int l = 0; l < K; ++l) {
    const bool mixed = S > 0 && l == 1;
    const int f = 1 << (K - 1 - (mixed ? 0 : l));
    const int W = (G + f - 1) / f;
    const int i = r / f, j = s / f;
    const int rows = min(f, G - i * f), cols = min(f, G - j * f);
    const int mem_crop = mixed ? G * G + m * m : G * G;   // members per crop
    const int tok_crop = mixed ? W * W + m * m : W * W;   // tokens per crop
    const int off = c * mem_crop + i * f * G + rows * j * f;
    const int a = r - i * f, b = s - j * f;
    if (mo.mem[l]) mo.mem[l][off + a * cols + b] = p;
    if (mo.offs[l]) {
      if (a == 0 && b == 0) mo.offs[l][c * tok_crop + i * W + j] = off;
      if (p == 0) mo.offs[l][n_crops * tok_crop] = n_crops * mem_crop;
    }
    if (mixed && r % S == S / 2 && s % S == S / 2) {
      const int k = (r / S) * m + (s / S);
      const int slot = c * mem_crop + G * G + k;
      if (mo.mem[l]) mo.mem[l][slot] = p;
      if (mo.offs[l]) mo.offs[l][c * tok_crop + W * W + k] = slot;
    }
  }
}

template <int K, int VEC, typename Fmt, bool MIXED = false>
void launch_pool(const davet_view_geom& g, const void* v, const LevelOut& lo,
                 hipStream_t s) {
  constexpr int F = 1 << (K - 1);
  const int Wc = (g.grid + F - 1) / F;
  dim3 grid(g.n_crops * Wc * Wc, (g.d / VEC + 255) / 256);
  hipLaunchKernelGGL((pool_views_kernel<K, VEC, Fmt, MIXED>), grid, dim3(256),
                     0, s, reinterpret_cast<const typename Fmt::st*>(v), lo,
                     g.n_crops, g.grid, g.d, g.mixed_stride);
}

template <typename Fmt>
void launch_pool_k(const davet_view_geom& g, const void* v, const LevelOut& lo,
                   hipStream_t s) {
  switch (g.K) {
    case 2: launch_pool<2, 8, Fmt>(g, v, lo, s); break;
    case 3:
      if (g.mixed_stride > 0) launch_pool<3, 8, Fmt, true>(g, v, lo, s);
      // two features per thread: twice the threads of four-wide loads, and
      // measured on MI355X 5-7 % faster at four and five 27 x 27 crops
      // (eight-wide loads 15-20 % slower; non-temporal loads no change)
      else launch_pool<3, 2, Fmt>(g, v, lo, s);
      break;
    default: launch_pool<4, 2, Fmt>(g, v, lo, s); break;
  }
}

}  // namespace

int launch_views(const davet_view_geom& g, const void* v, void* const* levels,
                 hipStream_t s) {
  if (g.K < 2) return DAVET_OK;
  LevelOut lo{};
  for (int l = 0; l < g.K - 1; ++l) lo.p[l] = levels[l];
  ProfScope ps(KC_VIEWS, s);
  if (g.dtype == DAVET_BF16) launch_pool_k<BF16S>(g, v, lo, s);
  else if (g.dtype == DAVET_F16) launch_pool_k<F16S>(g, v, lo, s);
  else launch_pool_k<F32S>(g, v, lo, s);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_view_maps(const davet_view_geom& g, int32_t* const* offs,
                     int32_t* const* mem, hipStream_t s) {
  MapOut mo{};
  bool any = false;
  for (int l = 0; l < g.K; ++l) {
    mo.offs[l] = offs ? offs[l] : nullptr;
    mo.mem[l] = mem ? mem[l] : nullptr;
    any = any || mo.offs[l] || mo.mem[l];
  }
  if (!any) return DAVET_OK;
  const int total = g.n_crops * g.grid * g.grid;
  ProfScope ps(KC_VIEW_MAPS, s);
  hipLaunchKernelGGL(view_maps_kernel, dim3((total + 255) / 256), dim3(256), 0,
                     s, mo, g.n_crops, g.grid, g.K, g.mixed_stride);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

}  // namespace davet

namespace davet {
int check_view_geom(const davet_view_geom* g, const char* who) {
  DAVET_CHECK_ARG(g->K >= 1 && g->K <= DAVET_MAX_LEVELS, DAVET_ESHAPE,
                  std::string(who) + ": K out of range [1, 4]");
  DAVET_CHECK_ARG(g->grid >= 1 && g->n_crops >= 1, DAVET_ESHAPE,
                  std::string(who) + ": grid and n_crops must be >= 1");
  DAVET_CHECK_ARG(g->realizer >= DAVET_REALIZER_POOL &&
                      g->realizer <= DAVET_REALIZER_MERGE, DAVET_EINVAL,
                  std::string(who) + ": unknown realizer");
  DAVET_CHECK_ARG(g->mixed_stride == 0 ||
                      (g->mixed_stride >= 2 && g->K == 3 &&
                       g->realizer == DAVET_REALIZER_POOL),
                  DAVET_ESHAPE,
                  std::string(who) + ": mixed_stride must be 0, or >= 2 with "
                  "K = 3 and the pooling realizer");
  DAVET_CHECK_ARG(g->realizer == DAVET_REALIZER_POOL ||
                      g->grid <= DAVET_MAX_REALIZER_GRID, DAVET_ESHAPE,
                  std::string(who) + ": grid above DAVET_MAX_REALIZER_GRID "
                  "for the prune / merge realizer");
  DAVET_CHECK_ARG((long long)g->n_crops * g->grid * g->grid * 2 < (1ll << 31),
                  DAVET_ESHAPE, std::string(who) + ": too many tokens");
  return DAVET_OK;
}
}  // namespace davet

extern "C" int davet_view_sizes(const davet_view_geom* g, int32_t* n_tokens) {
  using namespace davet;
  DAVET_CHECK_ARG(g && n_tokens, DAVET_EINVAL, "davet_view_sizes: null argument");
  int rc = check_view_geom(g, "davet_view_sizes");
  if (rc) return rc;
  for (int l = 0; l < g->K; ++l) {
    const int f = 1 << (g->K - 1 - l);
    const int W = (g->grid + f - 1) / f;
    n_tokens[l] = g->n_crops * W * W;
  }
  if (g->mixed_stride > 0) {
    const int W0 = (g->grid + 3) / 4;
    const int m = lattice_len(g->grid, g->mixed_stride);
    n_tokens[1] = g->n_crops * (W0 * W0 + m * m);
  }
  return DAVET_OK;
}

extern "C" int davet_view_map_sizes(const davet_view_geom* g,
                                    int32_t* n_members) {
  using namespace davet;
  DAVET_CHECK_ARG(g && n_members, DAVET_EINVAL,
                  "davet_view_map_sizes: null argument");
  int rc = check_view_geom(g, "davet_view_map_sizes");
  if (rc) return rc;
  for (int l = 0; l < g->K; ++l) n_members[l] = g->n_crops * g->grid * g->grid;
  if (g->realizer == DAVET_REALIZER_PRUNE) {        // one member per token
    for (int l = 0; l + 1 < g->K; ++l) {
      const int f = 1 << (g->K - 1 - l);
      const int W = (g->grid + f - 1) / f;
      n_members[l] = g->n_crops * W * W;
    }
  }
  if (g->mixed_stride > 0) {
    const int m = lattice_len(g->grid, g->mixed_stride);
    n_members[1] = g->n_crops * (g->grid * g->grid + m * m);
  }
  return DAVET_OK;
}

extern "C" int davet_views_scratch_bytes(const davet_view_geom* g,
                                         size_t* bytes) {
  using namespace davet;
  DAVET_CHECK_ARG(g && bytes, DAVET_EINVAL,
                  "davet_views_scratch_bytes: null argument");
  int rc = check_view_geom(g, "davet_views_scratch_bytes");
  if (rc) return rc;
  *bytes = realizer_scratch_bytes(*g);
  return DAVET_OK;
}

extern "C" int davet_build_views(const davet_view_geom* g, const void* v,
                                 void* const* levels,
                                 int32_t* const* idx_offsets,
                                 int32_t* const* idx_members, void* scratch,
                                 size_t scratch_bytes, hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(g && v, DAVET_EINVAL, "davet_build_views: null geometry or v");
  {
    int rc = check_view_geom(g, "davet_build_views");
    if (rc) return rc;
  }
  DAVET_CHECK_ARG(g->d >= 8 && g->d % 8 == 0, DAVET_ESHAPE,
                  "davet_build_views: d must be a positive multiple of 8");
  DAVET_CHECK_ARG(g->dtype == DAVET_F32 || g->dtype == DAVET_BF16 ||
                      g->dtype == DAVET_F16, DAVET_EDTYPE,
                  "davet_build_views: dtype must be DAVET_F32, BF16 or F16");
  DAVET_CHECK_ARG(((uintptr_t)v & 15) == 0, DAVET_EINVAL,
                  "davet_build_views: v must be 16-byte aligned");
  if (g->K > 1) {
    DAVET_CHECK_ARG(levels != nullptr, DAVET_EINVAL,
                    "davet_build_views: levels is null");
    for (int l = 0; l < g->K - 1; ++l) {
      DAVET_CHECK_ARG(levels[l] != nullptr, DAVET_EINVAL,
                      "davet_build_views: null pooled level pointer");
      DAVET_CHECK_ARG(((uintptr_t)levels[l] & 15) == 0, DAVET_EINVAL,
                      "davet_build_views: level buffers must be 16-byte aligned");
    }
  }
  if (g->realizer != DAVET_REALIZER_POOL)
    return build_views_realizer(*g, v, levels, idx_offsets, idx_members,
                                scratch, scratch_bytes, stream);
  int rc = launch_views(*g, v, levels, stream);
  if (rc != DAVET_OK) return rc;
  return launch_view_maps(*g, idx_offsets, idx_members, stream);
}
