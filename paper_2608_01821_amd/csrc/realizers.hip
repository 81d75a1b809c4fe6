// Pruning and merging evidence realizers (Sec. 4.3, "Compatible evidence
// realizers": pruning varies the retention ratio, merging the aggregation
// strength; the allocation policy is unchanged).  The paper gives neither
// criterion; the readings implemented here:
//   prune  token saliency = float64 L1 norm; per crop, level l keeps the n_l
//          most salient tokens (nested over levels), one member each;
//   merge  single linkage over the crop's 4-neighbour grid graph, edges
//          weighted by float64 cosine similarity, partition snapshotted when
//          n_l groups remain.
// n_l is the pooling pyramid's per-crop count, so every level costs the
// same as under pooling, and the levels go through the same CSR index maps.
//
// Three stages, each a kernel: keys (HBM-bound pass over v: one wavefront
// per token or grid edge, float64 accumulation), decisions (one 1024-thread
// workgroup per crop, everything in LDS: a rank per key, then for merge a
// single-lane union-find over the ranked edges, whose partition snapshots
// are labelled and scattered by all lanes), and the level rows (CSR means,
// float64 sums in member order, rounded once).

#include <mutex>
#include <string>

#include "common.h"

namespace davet {
namespace {

constexpr int RZ_NT = 1024;                                   // decision block
constexpr int RZ_MAXN = DAVET_MAX_REALIZER_GRID * DAVET_MAX_REALIZER_GRID;
constexpr int RZ_MAXE =
    2 * DAVET_MAX_REALIZER_GRID * (DAVET_MAX_REALIZER_GRID - 1);
constexpr int RZ_PER = RZ_MAXN / RZ_NT;                       // tokens/thread
static_assert(RZ_PER * RZ_NT == RZ_MAXN, "scan covers the largest crop");

struct LvlCnt { int n[DAVET_MAX_LEVELS]; };                   // per crop
struct MapPtrs {
  int32_t* offs[DAVET_MAX_LEVELS];
  int32_t* mem[DAVET_MAX_LEVELS];
};

// Eight consecutive features of one token as float64 (16-byte loads).
template <typename Fmt>
__device__ __forceinline__ void load8d(const typename Fmt::st* p, double* x) {
  if constexpr (sizeof(typename Fmt::st) == 2) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[2 * q] = (double)Fmt::load((uint16_t)(w[q] & 0xffffu));
      x[2 * q + 1] = (double)Fmt::load((uint16_t)(w[q] >> 16));
    }
  } else {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Ordered code of a key: larger key -> larger code; NaN as -inf, -0 as +0.
__device__ __forceinline__ uint64_t key_code(double x) {
  if (x != x) x = -__builtin_huge_val();
  if (x == 0.0) x = 0.0;
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}
// key a (index ia) is taken before key b (index ib)
__device__ __forceinline__ int before(uint64_t a, int ia, uint64_t b, int ib) {
  return (a > b || (a == b && ia < ib)) ? 1 : 0;
}

// Exclusive prefix sum of one int per thread over the block, in thread
// order; *total receives the block sum.  sh holds RZ_NT / 64 + 1 ints.
__device__ int block_scan_excl(int x, int* sh, int* total) {
  constexpr int NW = RZ_NT / 64;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  if (lane == 63) sh[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int i = 0; i < NW; ++i) {
      const int t = sh[i];
      sh[i] = acc;
      acc += t;
    }
    sh[NW] = acc;
  }
  __syncthreads();
  const int r = sh[w] + inc - x;
  *total = sh[NW];
  __syncthreads();
  return r;
}

// ------------------------------------------------------------------ keys --

// L1 norm of every token: one wavefront per token.
template <typename Fmt>
__global__ void __launch_bounds__(256)
prune_keys_kernel(const typename Fmt::st* __restrict__ v, int n_tok, int d,
                  double* __restrict__ keys) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= n_tok) return;
  const typename Fmt::st* row = v + (size_t)t * d;
  double acc = 0.0;
  for (int e0 = lane * 8; e0 < d; e0 += 512) {
    double x[8];
    load8d<Fmt>(row + e0, x);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc += fabs(x[k]);
  }
  acc = wave_sum_f64(acc);
  if (lane == 0) keys[t] = acc;
}

__device__ __forceinline__ void edge_ends(int e, int G, int& a, int& b) {
  const int H = G * (G - 1);
  if (e < H) {
    a = (e / (G - 1)) * G + e % (G - 1);
    b = a + 1;
  } else {
    a = e - H;
    b = a + G;
  }
}

// Cosine similarity of every grid edge: one wavefront per edge.
template <typename Fmt>
__global__ void __launch_bounds__(256)
merge_keys_kernel(const typename Fmt::st* __restrict__ v, int n_crops, int G,
                  int d, double* __restrict__ keys) {
  const int E = 2 * G * (G - 1);
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= n_crops * E) return;
  const int c = t / E;
  int a, b;
  edge_ends(t - c * E, G, a, b);
  const typename Fmt::st* ra = v + ((size_t)c * G * G + a) * d;
  const typename Fmt::st* rb = v + ((size_t)c * G * G + b) * d;
  double dot = 0.0, na = 0.0, nb = 0.0;
  for (int e0 = lane * 8; e0 < d; e0 += 512) {
    double x[8], y[8];
    load8d<Fmt>(ra + e0, x);
    load8d<Fmt>(rb + e0, y);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      dot += x[k] * y[k];
      na += x[k] * x[k];
      nb += y[k] * y[k];
    }
  }
  dot = wave_sum_f64(dot);
  na = wave_sum_f64(na);
  nb = wave_sum_f64(nb);
  if (lane == 0) keys[t] = (na == 0.0 || nb == 0.0) ? 0.0 : dot / sqrt(na * nb);
}

// ------------------------------------------------------------- decisions --

// Writes the identity map of the finest level (one crop per block).
__device__ void identity_map(const MapPtrs& mp, int K, int n_crops, int N) {
  const int c = blockIdx.x;
  for (int i = threadIdx.x; i < N; i += RZ_NT) {
    const int g = c * N + i;
    if (mp.mem[K - 1]) mp.mem[K - 1][g] = g;
    if (mp.offs[K - 1]) mp.offs[K - 1][g] = g;
  }
  if (c == 0 && threadIdx.x == 0 && mp.offs[K - 1])
    mp.offs[K - 1][n_crops * N] = n_crops * N;
}

// Prune: rank every token of the crop by its key, then per level keep the
// tokens ranked below n_l, compacted in index order by a block scan.
__global__ void __launch_bounds__(RZ_NT)
prune_maps_kernel(const double* __restrict__ keys, int n_crops, int G, int K,
                  LvlCnt cnt, MapPtrs mp) {
  __shared__ uint64_t code[RZ_MAXN];
  __shared__ int rank[RZ_MAXN];
  __shared__ int sh[RZ_NT / 64 + 1];
  const int N = G * G, c = blockIdx.x, tid = threadIdx.x;
  for (int i = tid; i < N; i += RZ_NT) code[i] = key_code(keys[(size_t)c * N + i]);
  __syncthreads();
  for (int i = tid; i < N; i += RZ_NT) {
    const uint64_t ki = code[i];
    int r = 0;
    for (int j = 0; j < N; ++j) r += before(code[j], j, ki, i);
    rank[i] = r;
  }
  __syncthreads();
  for (int l = 0; l < K - 1; ++l) {
    const int n = cnt.n[l];
    int kept[RZ_PER], local = 0;
#pragma unroll
    for (int q = 0; q < RZ_PER; ++q) {
      const int i = tid * RZ_PER + q;
      kept[q] = (i < N && rank[i] < n) ? 1 : 0;
      local += kept[q];
    }
    int total;
    int pos = block_scan_excl(local, sh, &total);
#pragma unroll
    for (int q = 0; q < RZ_PER; ++q) {
      if (!kept[q]) continue;
      const int slot = c * n + pos;
      if (mp.mem[l]) mp.mem[l][slot] = c * N + tid * RZ_PER + q;
      if (mp.offs[l]) mp.offs[l][slot] = slot;
      ++pos;
    }
    if (c == 0 && tid == 0 && mp.offs[l]) mp.offs[l][n_crops * n] = n_crops * n;
  }
  identity_map(mp, K, n_crops, N);
}

// root of x with path halving (single writer)
__device__ __forceinline__ int find_halve(int* parent, int x) {
  while (parent[x] != x) {
    const int gp = parent[parent[x]];
    parent[x] = gp;
    x = gp;
  }
  return x;
}

// Merge: rank the crop's edges by key; lane 0 of the block runs the
// union-find over the ranked edges (the larger root joins the smaller, so a
// root is its group's smallest member) until n_l groups remain; then all
// lanes label every token with its root, count group sizes, scan sizes and
// roots in index order (member start and group index), and scatter members.
__global__ void __launch_bounds__(RZ_NT)
merge_maps_kernel(const double* __restrict__ keys, int n_crops, int G, int K,
                  LvlCnt cnt, MapPtrs mp) {
  __shared__ uint64_t code[RZ_MAXE];
  __shared__ uint16_t order[RZ_MAXE];
  __shared__ int parent[RZ_MAXN];
  __shared__ int label[RZ_MAXN];
  __shared__ int aux[RZ_MAXN];          // group sizes, then member starts
  __shared__ int sh[RZ_NT / 64 + 1];
  __shared__ int s_groups, s_ptr;
  const int N = G * G, E = 2 * G * (G - 1), c = blockIdx.x, tid = threadIdx.x;
  for (int e = tid; e < E; e += RZ_NT) code[e] = key_code(keys[(size_t)c * E + e]);
  for (int i = tid; i < N; i += RZ_NT) parent[i] = i;
  __syncthreads();
  for (int e = tid; e < E; e += RZ_NT) {
    const uint64_t ke = code[e];
    int r = 0;
    for (int f = 0; f < E; ++f) r += before(code[f], f, ke, e);
    order[r] = (uint16_t)e;
  }
  if (tid == 0) { s_groups = N; s_ptr = 0; }
  __syncthreads();
  for (int l = K - 2; l >= 0; --l) {
    const int n = cnt.n[l];
    if (tid == 0) {
      int groups = s_groups, p = s_ptr;
      // the grid graph is connected, so groups reaches n before p reaches E
      while (groups > n && p < E) {
        int a, b;
        edge_ends(order[p++], G, a, b);
        const int ra = find_halve(parent, a), rb = find_halve(parent, b);
        if (ra != rb) {
          parent[max(ra, rb)] = min(ra, rb);
          --groups;
        }
      }
      s_groups = groups;
      s_ptr = p;
    }
    __syncthreads();
    for (int i = tid; i < N; i += RZ_NT) {
      int x = i;
      while (parent[x] != x) x = parent[x];
      label[i] = x;
      aux[i] = 0;
    }
    __syncthreads();
    for (int i = tid; i < N; i += RZ_NT) atomicAdd(&aux[label[i]], 1);
    __syncthreads();
    int sz[RZ_PER], rt[RZ_PER], lsz = 0, lrt = 0;
#pragma unroll
    for (int q = 0; q < RZ_PER; ++q) {
      const int i = tid * RZ_PER + q;
      sz[q] = i < N ? aux[i] : 0;
      rt[q] = (i < N && label[i] == i) ? 1 : 0;
      lsz += sz[q];
      lrt += rt[q];
    }
    int total;
    int start = block_scan_excl(lsz, sh, &total);
    int g = block_scan_excl(lrt, sh, &total);
#pragma unroll
    for (int q = 0; q < RZ_PER; ++q) {
      const int i = tid * RZ_PER + q;
      if (i >= N) continue;
      aux[i] = start;                     // this thread's own entries only
      if (rt[q]) {
        // g < n always (exactly n roots remain); the test keeps a broken
        // invariant from writing past the level's offsets
        if (mp.offs[l] && g < n) mp.offs[l][c * n + g] = c * N + start;
        ++g;
      }
      start += sz[q];
    }
    __syncthreads();
    if (mp.mem[l]) {
      for (int i = tid; i < N; i += RZ_NT) {
        const int r = label[i];
        int pos = 0;
        for (int j = r; j < i; ++j) pos += (label[j] == r) ? 1 : 0;
        mp.mem[l][c * N + aux[r] + pos] = c * N + i;
      }
    }
    if (c == 0 && tid == 0 && mp.offs[l]) mp.offs[l][n_crops * n] = n_crops * N;
    __syncthreads();
  }
  identity_map(mp, K, n_crops, N);
}

// ----------------------------------------------------------------- levels --

// Token t = float64 sum of rows mem[offs[t] .. offs[t+1]) of v in that
// order, divided by the member count, rounded once.  Eight features per
// thread; the rows of eight members are loaded together (independent loads
// in flight) and then added one member after another, so large merged
// groups are not bound by one load latency per member.
template <typename Fmt>
__global__ void __launch_bounds__(256)
pool_csr_kernel(const typename Fmt::st* __restrict__ v,
                const int32_t* __restrict__ offs,
                const int32_t* __restrict__ mem, int d,
                typename Fmt::st* __restrict__ out) {
  using T = typename Fmt::st;
  constexpr int B = 8;                            // members per batch
  constexpr int Q = sizeof(T) == 2 ? 1 : 2;       // 16-byte pieces per row
  const int t = blockIdx.x;
  const int e0 = (blockIdx.y * 256 + threadIdx.x) * 8;
  if (e0 >= d) return;
  const int b = offs[t], e = offs[t + 1];
  double acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) acc[k] = 0.0;
  for (int m0 = b; m0 < e; m0 += B) {
    const int nb = min(B, e - m0);
    u32x4 raw[B][Q];
#pragma unroll
    for (int k = 0; k < B; ++k) {
      if (k < nb) {
        const T* p = v + (size_t)mem[m0 + k] * d + e0;
#pragma unroll
        for (int q = 0; q < Q; ++q)
          raw[k][q] = *reinterpret_cast<const u32x4*>(p + q * (8 / Q));
      }
    }
#pragma unroll
    for (int k = 0; k < B; ++k) {
      if (k < nb) {
        if constexpr (sizeof(T) == 2) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            acc[2 * q] += (double)Fmt::load((uint16_t)(raw[k][0][q] & 0xffffu));
            acc[2 * q + 1] += (double)Fmt::load((uint16_t)(raw[k][0][q] >> 16));
          }
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j)
            acc[j] += (double)__uint_as_float(raw[k][j / 4][j % 4]);
        }
      }
    }
  }
  const double cnt = (double)(e - b);
  typename Fmt::st* dst = out + (size_t)t * d + e0;
  if constexpr (sizeof(typename Fmt::st) == 2) {
    u32x4 w;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      w[q] = (uint32_t)Fmt::from_f64(acc[2 * q] / cnt) |
             ((uint32_t)Fmt::from_f64(acc[2 * q + 1] / cnt) << 16);
    *reinterpret_cast<u32x4*>(dst) = w;
  } else {
    float4 a, bq;
    a.x = (float)(acc[0] / cnt); a.y = (float)(acc[1] / cnt);
    a.z = (float)(acc[2] / cnt); a.w = (float)(acc[3] / cnt);
    bq.x = (float)(acc[4] / cnt); bq.y = (float)(acc[5] / cnt);
    bq.z = (float)(acc[6] / cnt); bq.w = (float)(acc[7] / cnt);
    *reinterpret_cast<float4*>(dst) = a;
    *reinterpret_cast<float4*>(dst + 4) = bq;
  }
}

// ------------------------------------------------------------------ host --

bool is_realizer(const davet_view_geom& g) {
  return g.realizer == DAVET_REALIZER_PRUNE || g.realizer == DAVET_REALIZER_MERGE;
}

int key_count(const davet_view_geom& g) {
  if (g.realizer == DAVET_REALIZER_PRUNE) return g.n_crops * g.grid * g.grid;
  if (g.realizer == DAVET_REALIZER_MERGE)
    return g.n_crops * 2 * g.grid * (g.grid - 1);
  return 0;
}

LvlCnt level_counts(const davet_view_geom& g) {
  LvlCnt lc{};
  for (int l = 0; l < g.K; ++l) {
    const int f = 1 << (g.K - 1 - l);
    const int W = (g.grid + f - 1) / f;
    lc.n[l] = W * W;
  }
  return lc;
}

int check_realizer(const davet_view_geom* g, const void* v, const char* who) {
  int rc = check_view_geom(g, who);
  if (rc) return rc;
  DAVET_CHECK_ARG(is_realizer(*g), DAVET_EINVAL,
                  std::string(who) + ": the geometry's realizer is pooling, "
                  "which has no keys");
  DAVET_CHECK_ARG(g->d >= 8 && g->d % 8 == 0, DAVET_ESHAPE,
                  std::string(who) + ": d must be a positive multiple of 8");
  DAVET_CHECK_ARG(g->dtype == DAVET_F32 || g->dtype == DAVET_BF16 ||
                      g->dtype == DAVET_F16, DAVET_EDTYPE,
                  std::string(who) + ": dtype must be DAVET_F32, BF16 or F16");
  DAVET_CHECK_ARG(v == nullptr || ((uintptr_t)v & 15) == 0, DAVET_EINVAL,
                  std::string(who) + ": v must be 16-byte aligned");
  return DAVET_OK;
}

template <typename Fmt>
void launch_keys_t(const davet_view_geom& g, const void* v, double* keys,
                   hipStream_t s) {
  const auto* vv = reinterpret_cast<const typename Fmt::st*>(v);
  const int n = key_count(g);
  if (n == 0) return;
  if (g.realizer == DAVET_REALIZER_PRUNE)
    hipLaunchKernelGGL(prune_keys_kernel<Fmt>, dim3((n + 3) / 4), dim3(256), 0,
                       s, vv, n, g.d, keys);
  else
    hipLaunchKernelGGL(merge_keys_kernel<Fmt>, dim3((n + 3) / 4), dim3(256), 0,
                       s, vv, g.n_crops, g.grid, g.d, keys);
}

int launch_keys(const davet_view_geom& g, const void* v, double* keys,
                hipStream_t s) {
  ProfScope ps(KC_REALIZER_KEYS, s);
  if (g.dtype == DAVET_BF16) launch_keys_t<BF16S>(g, v, keys, s);
  else if (g.dtype == DAVET_F16) launch_keys_t<F16S>(g, v, keys, s);
  else launch_keys_t<F32S>(g, v, keys, s);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

int launch_maps(const davet_view_geom& g, const double* keys, const MapPtrs& mp,
                hipStream_t s) {
  bool any = false;
  for (int l = 0; l < g.K; ++l) any = any || mp.offs[l] || mp.mem[l];
  if (!any) return DAVET_OK;
  ProfScope ps(KC_REALIZER_MAPS, s);
  const LvlCnt lc = level_counts(g);
  if (g.realizer == DAVET_REALIZER_PRUNE)
    hipLaunchKernelGGL(prune_maps_kernel, dim3(g.n_crops), dim3(RZ_NT), 0, s,
                       keys, g.n_crops, g.grid, g.K, lc, mp);
  else
    hipLaunchKernelGGL(merge_maps_kernel, dim3(g.n_crops), dim3(RZ_NT), 0, s,
                       keys, g.n_crops, g.grid, g.K, lc, mp);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

template <typename Fmt>
void launch_pool_csr_t(const void* v, const int32_t* offs, const int32_t* mem,
                       int n_tok, int d, void* out, hipStream_t s) {
  dim3 grid(n_tok, (d / 8 + 255) / 256);
  hipLaunchKernelGGL(pool_csr_kernel<Fmt>, grid, dim3(256), 0, s,
                     reinterpret_cast<const typename Fmt::st*>(v), offs, mem, d,
                     reinterpret_cast<typename Fmt::st*>(out));
}

// Scratch layout: keys, then (offsets, members) of each level < K-1, each
// region 256-byte aligned.
struct RzLayout {
  size_t keys = 0, offs[DAVET_MAX_LEVELS] = {}, mem[DAVET_MAX_LEVELS] = {};
  size_t total = 0;
};

RzLayout rz_layout(const davet_view_geom& g) {
  RzLayout L;
  size_t o = 0;
  L.keys = o;
  o += align_up((size_t)key_count(g) * 8, 256);
  const LvlCnt lc = level_counts(g);
  for (int l = 0; l + 1 < g.K; ++l) {
    const size_t n = (size_t)g.n_crops * lc.n[l];
    const size_t m = g.realizer == DAVET_REALIZER_PRUNE
                         ? n : (size_t)g.n_crops * g.grid * g.grid;
    L.offs[l] = o;
    o += align_up((n + 1) * 4, 256);
    L.mem[l] = o;
    o += align_up(m * 4, 256);
  }
  L.total = o;
  return L;
}

}  // namespace

size_t realizer_scratch_bytes(const davet_view_geom& g) {
  return is_realizer(g) ? rz_layout(g).total : 0;
}

int build_views_realizer(const davet_view_geom& g, const void* v,
                         void* const* levels, int32_t* const* offs,
                         int32_t* const* mem, void* scratch,
                         size_t scratch_bytes, hipStream_t s) {
  const RzLayout L = rz_layout(g);
  DAVET_CHECK_ARG(scratch != nullptr && scratch_bytes >= L.total, DAVET_ENOMEM,
                  "davet_build_views: scratch smaller than "
                  "davet_views_scratch_bytes");
  DAVET_CHECK_ARG(((uintptr_t)scratch & 255) == 0, DAVET_EINVAL,
                  "davet_build_views: scratch must be 256-byte aligned");
  char* sc = static_cast<char*>(scratch);
  double* keys = reinterpret_cast<double*>(sc + L.keys);
  MapPtrs mp{};
  for (int l = 0; l < g.K; ++l) {
    const bool own = l + 1 < g.K;
    mp.offs[l] = offs && offs[l] ? offs[l]
                 : own ? reinterpret_cast<int32_t*>(sc + L.offs[l]) : nullptr;
    mp.mem[l] = mem && mem[l] ? mem[l]
                : own ? reinterpret_cast<int32_t*>(sc + L.mem[l]) : nullptr;
  }
  int rc = launch_keys(g, v, keys, s);
  if (rc) return rc;
  rc = launch_maps(g, keys, mp, s);
  if (rc) return rc;
  const LvlCnt lc = level_counts(g);
  ProfScope ps(KC_VIEWS, s);
  for (int l = 0; l + 1 < g.K; ++l) {
    const int n = g.n_crops * lc.n[l];
    if (g.dtype == DAVET_BF16)
      launch_pool_csr_t<BF16S>(v, mp.offs[l], mp.mem[l], n, g.d, levels[l], s);
    else if (g.dtype == DAVET_F16)
      launch_pool_csr_t<F16S>(v, mp.offs[l], mp.mem[l], n, g.d, levels[l], s);
    else
      launch_pool_csr_t<F32S>(v, mp.offs[l], mp.mem[l], n, g.d, levels[l], s);
  }
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

}  // namespace davet

extern "C" int davet_realizer_key_count(const davet_view_geom* g,
                                        int32_t* n_keys) {
  using namespace davet;
  DAVET_CHECK_ARG(g && n_keys, DAVET_EINVAL,
                  "davet_realizer_key_count: null argument");
  int rc = check_view_geom(g, "davet_realizer_key_count");
  if (rc) return rc;
  *n_keys = key_count(*g);
  return DAVET_OK;
}

extern "C" int davet_realizer_keys(const davet_view_geom* g, const void* v,
                                   double* keys, hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(g && v && keys, DAVET_EINVAL,
                  "davet_realizer_keys: null argument");
  int rc = check_realizer(g, v, "davet_realizer_keys");
  if (rc) return rc;
  DAVET_CHECK_ARG(((uintptr_t)keys & 7) == 0, DAVET_EINVAL,
                  "davet_realizer_keys: keys must be 8-byte aligned");
  return launch_keys(*g, v, keys, stream);
}

extern "C" int davet_realizer_maps(const davet_view_geom* g,
                                   const double* keys,
                                   int32_t* const* idx_offsets,
                                   int32_t* const* idx_members,
                                   hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(g, DAVET_EINVAL, "davet_realizer_maps: null geometry");
  int rc = check_realizer(g, nullptr, "davet_realizer_maps");
  if (rc) return rc;
  DAVET_CHECK_ARG(keys != nullptr || key_count(*g) == 0, DAVET_EINVAL,
                  "davet_realizer_maps: null keys");
  DAVET_CHECK_ARG(((uintptr_t)keys & 7) == 0, DAVET_EINVAL,
                  "davet_realizer_maps: keys must be 8-byte aligned");
  MapPtrs mp{};
  for (int l = 0; l < g->K; ++l) {
    mp.offs[l] = idx_offsets ? idx_offsets[l] : nullptr;
    mp.mem[l] = idx_members ? idx_members[l] : nullptr;
  }
  return launch_maps(*g, keys, mp, stream);
}

// ---------------------------------------------------------------------------
// davet_build_views_static: davet_build_views with the realizers' scratch
// (keys and the index maps of the pooled levels) in a file-scope device
// array instead of caller memory, for callers that cannot allocate.  Host
// code never passes the array's name to a kernel (in host code it is only a
// stand-in for the symbol): the device address is resolved once per device
// with hipGetSymbolAddress and kept.  Every call on a device shares that
// device's array; the keys and maps are written in full before they are
// read, so nothing needs clearing, and calls that overlap on one device race.

static __device__ __align__(256) char scratch[DAVET_STATIC_SCRATCH_BYTES];

namespace davet {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of `scratch` on the current device (resolved on the first
// call on that device).
int static_scratch(void** out) {
  int dev = -1;
  DAVET_HIP(hipGetDevice(&dev));
  DAVET_CHECK_ARG(dev >= 0 && dev < kMaxDevices, DAVET_EHIP,
                  "davet_build_views_static: device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    DAVET_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    DAVET_CHECK_ARG(p != nullptr && ((uintptr_t)p & 255) == 0, DAVET_EHIP,
                    "davet_build_views_static: scratch address unusable");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return DAVET_OK;
}

}  // namespace
}  // namespace davet

extern "C" int davet_build_views_static(const davet_view_geom* g,
                                        const void* v, void* const* levels,
                                        int32_t* const* idx_offsets,
                                        int32_t* const* idx_members,
                                        hipStream_t stream) {
  using namespace davet;
  DAVET_CHECK_ARG(g, DAVET_EINVAL, "davet_build_views_static: null geometry");
  int rc = check_view_geom(g, "davet_build_views_static");
  if (rc) return rc;
  const size_t need = realizer_scratch_bytes(*g);
  DAVET_CHECK_ARG(need <= DAVET_STATIC_SCRATCH_BYTES, DAVET_ENOMEM,
                  "davet_build_views_static: the geometry needs " +
                      std::to_string(need) + " bytes of scratch, more than "
                      "the static maximum of " +
                      std::to_string((size_t)DAVET_STATIC_SCRATCH_BYTES) +
                      " (use davet_build_views with caller scratch)");
  void* sc = nullptr;
  if (need) {
    rc = static_scratch(&sc);
    if (rc) return rc;
  }
  return davet_build_views(g, v, levels, idx_offsets, idx_members, sc,
                           need ? (size_t)DAVET_STATIC_SCRATCH_BYTES : 0,
                           stream);
}
