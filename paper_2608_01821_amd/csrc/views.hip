// Evidence hierarchy by per-crop average pooling (Sec. 4.3, "Ordered evidence
// hierarchy"; v^(K) = v).  One pass over v builds every pooled level: a thread
// owns 8 (or 2) consecutive features of one coarsest window and visits that
// window's tokens once, in row-major order, adding each into the running
// float64 sum of the sub-window it belongs to at every finer level.  Each
// level token is then (sum / member count) rounded once to the view dtype.
// HBM-bound: v is read once, the levels are written once.

#include "common.h"

namespace davet {
namespace {

struct LevelOut { void* p[DAVET_MAX_LEVELS]; };


template <int K, int VEC, typename Fmt>
__global__ void __launch_bounds__(256)
pool_views_kernel(const typename Fmt::st* __restrict__ v, LevelOut out,
                  int n_crops, int G, int d) {
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
  // Fully unrolled so every accumulator index is a compile-time constant.
#pragma unroll
  for (int dr = 0; dr < F; ++dr) {
#pragma unroll
    for (int ds = 0; ds < F; ++ds) {
      const int r = r0 + dr, s = s0 + ds;
      if (r >= G || s >= G) continue;
      const T* src = v + ((size_t)c * G * G + (size_t)r * G + s) * d + e0;
      float x[VEC];
      if constexpr (sizeof(T) == 2) {
        if constexpr (VEC == 8) {
          u32x4 w = *reinterpret_cast<const u32x4*>(src);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            x[2 * q] = Fmt::load((uint16_t)(w[q] & 0xffffu));
            x[2 * q + 1] = Fmt::load((uint16_t)(w[q] >> 16));
          }
        } else {
          uint32_t w = *reinterpret_cast<const uint32_t*>(src);
          x[0] = Fmt::load((uint16_t)(w & 0xffffu));
          x[1] = Fmt::load((uint16_t)(w >> 16));
        }
      } else {
#pragma unroll
        for (int e = 0; e < VEC; e += 2) {
          float2 w = *reinterpret_cast<const float2*>(src + e);
          x[e] = w.x; x[e + 1] = w.y;
        }
      }
      int base = 0;
#pragma unroll
      for (int l = 0; l < K - 1; ++l) {
        const int f = F >> l;                      // window side of level l
        const int per = F / f;                     // sub-windows per side
        const int a = base + (dr / f) * per + (ds / f);
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[a][e] += (double)x[e];
        base += per * per;
      }
    }
  }
  int base = 0;
#pragma unroll
  for (int l = 0; l < K - 1; ++l) {
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
          } else {
            *reinterpret_cast<uint32_t*>(dst) =
                (uint32_t)h[0] | ((uint32_t)h[1] << 16);
          }
        } else {
          float* dst = reinterpret_cast<float*>(out.p[l]) + tok * d + e0;
#pragma unroll
          for (int e = 0; e < VEC; e += 2) {
            float2 w;
            w.x = (float)(ac[e] / cnt);
            w.y = (float)(ac[e + 1] / cnt);
            *reinterpret_cast<float2*>(dst + e) = w;
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
__global__ void __launch_bounds__(256)
view_maps_kernel(MapOut mo, int n_crops, int G, int K) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  const int total = n_crops * G * G;
  if (p >= total) return;
  const int c = p / (G * G);
  const int r = (p / G) % G;
  const int s = p % G;
  for (int l = 0; l < K; ++l) {
    const int f = 1 << (K - 1 - l);
    const int W = (G + f - 1) / f;
    const int i = r / f, j = s / f;
    const int rows = min(f, G - i * f), cols = min(f, G - j * f);
    const int off = c * G * G + i * f * G + rows * j * f;
    const int a = r - i * f, b = s - j * f;
    if (mo.mem[l]) mo.mem[l][off + a * cols + b] = p;
    if (mo.offs[l]) {
      if (a == 0 && b == 0) mo.offs[l][c * W * W + i * W + j] = off;
      if (p == 0) mo.offs[l][n_crops * W * W] = total;
    }
  }
}

template <int K, int VEC, typename Fmt>
void launch_pool(const davet_view_geom& g, const void* v, const LevelOut& lo,
                 hipStream_t s) {
  constexpr int F = 1 << (K - 1);
  const int Wc = (g.grid + F - 1) / F;
  dim3 grid(g.n_crops * Wc * Wc, (g.d / VEC + 255) / 256);
  hipLaunchKernelGGL((pool_views_kernel<K, VEC, Fmt>), grid, dim3(256), 0, s,
                     reinterpret_cast<const typename Fmt::st*>(v), lo,
                     g.n_crops, g.grid, g.d);
}

template <typename Fmt>
void launch_pool_k(const davet_view_geom& g, const void* v, const LevelOut& lo,
                   hipStream_t s) {
  switch (g.K) {
    case 2: launch_pool<2, 8, Fmt>(g, v, lo, s); break;
    case 3: launch_pool<3, 8, Fmt>(g, v, lo, s); break;
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
                     s, mo, g.n_crops, g.grid, g.K);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

}  // namespace davet

extern "C" int davet_view_sizes(const davet_view_geom* g, int32_t* n_tokens) {
  using namespace davet;
  DAVET_CHECK_ARG(g && n_tokens, DAVET_EINVAL, "davet_view_sizes: null argument");
  DAVET_CHECK_ARG(g->K >= 1 && g->K <= DAVET_MAX_LEVELS, DAVET_ESHAPE,
                  "davet_view_sizes: K out of range");
  DAVET_CHECK_ARG(g->grid >= 1 && g->n_crops >= 1, DAVET_ESHAPE,
                  "davet_view_sizes: grid and n_crops must be >= 1");
  for (int l = 0; l < g->K; ++l) {
    const int f = 1 << (g->K - 1 - l);
    const int W = (g->grid + f - 1) / f;
    n_tokens[l] = g->n_crops * W * W;
  }
  return DAVET_OK;
}

extern "C" int davet_build_views(const davet_view_geom* g, const void* v,
                                 void* const* levels,
                                 int32_t* const* idx_offsets,
                                 int32_t* const* idx_members,
                                 hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(g && v, DAVET_EINVAL, "davet_build_views: null geometry or v");
  DAVET_CHECK_ARG(g->K >= 1 && g->K <= DAVET_MAX_LEVELS, DAVET_ESHAPE,
                  "davet_build_views: K out of range [1, 4]");
  DAVET_CHECK_ARG(g->grid >= 1 && g->n_crops >= 1, DAVET_ESHAPE,
                  "davet_build_views: grid and n_crops must be >= 1");
  DAVET_CHECK_ARG(g->d >= 8 && g->d % 8 == 0, DAVET_ESHAPE,
                  "davet_build_views: d must be a positive multiple of 8");
  DAVET_CHECK_ARG(g->dtype == DAVET_F32 || g->dtype == DAVET_BF16 ||
                      g->dtype == DAVET_F16, DAVET_EDTYPE,
                  "davet_build_views: dtype must be DAVET_F32, BF16 or F16");
  DAVET_CHECK_ARG((long long)g->n_crops * g->grid * g->grid < (1ll << 31),
                  DAVET_ESHAPE, "davet_build_views: too many tokens");
  if (g->K > 1) {
    DAVET_CHECK_ARG(levels != nullptr, DAVET_EINVAL,
                    "davet_build_views: levels is null");
    for (int l = 0; l < g->K - 1; ++l)
      DAVET_CHECK_ARG(levels[l] != nullptr, DAVET_EINVAL,
                      "davet_build_views: null pooled level pointer");
  }
  int rc = launch_views(*g, v, levels, stream);
  if (rc != DAVET_OK) return rc;
  return launch_view_maps(*g, idx_offsets, idx_members, stream);
}
