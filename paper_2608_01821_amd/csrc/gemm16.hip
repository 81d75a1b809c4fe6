// 16-bit (fp16 or bf16) matrix-core GEMMs of the denoiser: C[M,N] = A[M,K] B[N,K]^T
// with both operands K-contiguous (activations row-major, weights [out, in]).
//
// CDNA4 design.  A workgroup of 4, 8 or 16 wavefronts (a WM x WN grid, WN = 2
// or 4) owns a BM x BN tile; each wavefront accumulates (BM/WM) x (BN/WN)
// with v_mfma_f32_16x16x32 ops (fp32 accumulators).  K moves in slabs of BK (32
// or 64) through a STAGES-deep ring of LDS stages filled by direct
// global->LDS loads (global_load_lds_dwordx4: no VGPR staging), so up to
// STAGES - 1 slabs are in flight while one feeds the matrix cores; one
// barrier per slab.  Each LDS row holds BK 16-bit values in 16-byte chunks;
// chunk c of row r sits in slot c ^ ((r / rows-per-256-bytes) % chunks),
// which spreads the 16-byte fragment reads of 16 consecutive rows over
// distinct bank groups.  Workgroup ids are remapped so each XCD (ids
// congruent mod 8) walks a contiguous run of tiles, M fastest: a weight tile
// is fetched into one XCD's L2 and reused by every M tile.  The variants
// (tile, slab depth, ring depth, waves) and the plan that picks one per
// product shape are listed after the kernel.
//
// Split-K: with few output tiles (short sequences) the K range is cut into
// ksplit parts whose fp32 partial tiles land in a workspace; a row kernel
// sums them in a fixed order (deterministic) and applies the epilogue.
//
// Epilogues, fused:
//   EPI_STORE    16-bit C = acc, with the rotary embedding applied in fp32 to
//                the query/key columns (a lane owns dims i and i+64 of a head)
//   EPI_ADD_F32  fp32 C += acc (residual stream)
//   EPI_SWIGLU   B holds gate rows, B2 up rows; gate and up of one output
//                column sit in the same lane: 16-bit C = silu(gate) * up
//   EPI_HEAD     vocabulary slab reduction per row: (max, first argmax,
//                sum exp(l - max)) with [MASK] excluded
//   EPI_PARTIAL  fp32 partial tile of one K split

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "common.h"

namespace davet {
namespace {

constexpr int BK_MIN = 32;   // K must be a multiple of this

constexpr int EPI_HEAD = 3;

// Kernel variants: tile BM x BN, K slab BK (64-byte or 128-byte LDS rows),
// STAGES-deep LDS ring, WAVES wavefronts in a (WAVES / WN) x WN grid (WN = 2
// or 4 wave columns); IGLP >= 0 asks the compiler's scheduler for its
// matrix-op interleaving strategy of that number (__builtin_amdgcn_iglp_opt)
// on the slab body; SG = 1 gives it an explicit order instead (schedule
// groups: the first 32-deep step's fragment reads, then the second step's
// reads one per matrix op of the first step, then the remaining matrix ops).
template <int BM_, int BN_, int BK_, int STAGES_, int WAVES_, int IGLP_ = -1,
          int WN_ = 2, int SG_ = 0>
struct Var {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, STAGES = STAGES_,
                       WAVES = WAVES_, IGLP = IGLP_, WN = WN_, SG = SG_;
  static constexpr int LDS = STAGES * (BM + BN) * BK * 2;
  // workgroups per CU the register budget must allow (LDS is 160 KB per CU)
  static constexpr int MINB = LDS <= 80 * 1024 ? (LDS <= 53 * 1024 ? 3 : 2) : 1;
};
constexpr int EPI_PARTIAL = 4;

struct EpiArgs {
  void* C;
  int ldc;
  // rotary embedding (EPI_STORE): columns < rope_cols are rotated
  const int32_t* pos;
  const float2* cs;
  int rope_cols;
  // vocabulary head
  const int32_t* list;
  int vocab, mask_id, n_slabs;
  float* pmax;
  float* psum;
  int32_t* parg;
  float* logits_out;
  // split-K partials: part[ks][row][col], row stride part_ld
  float* part;
  int part_ld;
  int dual;              // B/B2 gate/up weights (SwiGLU), also for partials
  int ffn;
  // B is a tiled vocabulary head of 128 x 64 blocks (davet_pack_head), BN a
  // multiple of 128, BK 32 or 64: slab step kt reads BK columns of each of
  // its BN / 128 blocks in chunk kt * BK / 64, from column kt * BK % 64
  int b_tiled;
  // non-finite 16-bit values stored by EPI_STORE / EPI_SWIGLU (may be null)
  int32_t* overflow;
};

__device__ __forceinline__ int remap_xcd(int bid, int nwg) {
  const int full = nwg & ~7;
  if (bid >= full) return bid;
  const int per = full >> 3;
  return (bid & 7) * per + (bid >> 3);
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// s_waitcnt vmcnt(n) for a wave-uniform n in [LO, HI] known only at run time
// (the count is an instruction immediate): a binary tree of scalar branches.
template <int LO, int HI>
__device__ __forceinline__ void wait_vmcnt_rt(int n) {
  if constexpr (LO == HI) {
    wait_vmcnt<LO>();
  } else {
    constexpr int MID = (LO + HI) / 2;
    if (n <= MID) wait_vmcnt_rt<LO, MID>(n);
    else wait_vmcnt_rt<MID + 1, HI>(n);
  }
}

// Workgroup barrier without the memory fence __syncthreads() carries: the
// fence would wait for every outstanding global->LDS load (vmcnt(0)) and
// drain the pipeline.  Each wave has already waited for the slab it needs;
// the empty asm statements keep the compiler from moving LDS accesses across.
__device__ __forceinline__ void barrier_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

__device__ __forceinline__ void dma16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_ptr_t)lds, 16, 0, 0);
}

// Byte offset of chunk c (16 B) of row r inside a stage of BK-wide rows.
// Slot = c ^ f(r) with f chosen so 16 consecutive rows at the same chunk fall
// in 16 distinct 16-byte bank groups of a 256-byte bank line.
template <int BK>
__device__ __forceinline__ int swz(int r, int c) {
  constexpr int CPR = BK / 8;                 // 16-byte chunks per row
  constexpr int RPL = 16 / CPR;               // rows per 256-byte bank line
  return r * (BK * 2) + ((c ^ ((r / RPL) % CPR)) << 4);
}

template <typename Fmt, typename V, int EPI>
__global__ void __launch_bounds__(64 * V::WAVES, V::MINB)
gemm16_kernel(const uint16_t* __restrict__ A, const uint16_t* __restrict__ B,
              const uint16_t* __restrict__ B2, int M, int N, int K,
              int n_mtiles, int n_ntiles, int ksplit, EpiArgs ep) {
  using v8 = typename Fmt::v8;
  constexpr int BM = V::BM, BN = V::BN, BK = V::BK, STAGES = V::STAGES;
  constexpr int WAVES = V::WAVES;
  constexpr int WN = V::WN;              // wave grid WM x WN
  constexpr int WM = WAVES / WN;
  constexpr int WROWS = BM / WM;         // rows per wave
  constexpr int TM = WROWS / 32;         // 32-row sub-tiles per wave
  constexpr int TN = BN / 64;            // 64-column groups of the tile
  constexpr int CW = 64 / WN;            // a wave's columns in each group
  constexpr int QC = CW / 16;            // ... as 16-column blocks
  constexpr int NQ = 2 * QC;             // 16 x 16 accumulators per 32-row
                                         // sub-tile and column group
  static_assert(WN == 2 || WN == 4, "two or four wave columns");
  static_assert(EPI != EPI_HEAD || WN == 2, "the head reduction pairs two wave columns");
  constexpr int CPR = BK / 8;            // 16-byte chunks per LDS row
  constexpr int RPI = 64 / CPR;          // rows per load instruction
  constexpr int AI = BM / (RPI * WAVES); // A load instructions per wave/stage
  constexpr int BI = BN / (RPI * WAVES); // B load instructions per wave/stage
  static_assert(AI >= 1 && BI >= 1 && TM >= 1, "tile too small for the waves");
  constexpr int LPT = AI + BI;
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  constexpr int S_BYTES = A_BYTES + B_BYTES;
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * S_BYTES];

  const int nwg = gridDim.x;
  const int tile = remap_xcd(blockIdx.x, nwg);
  const int mb = tile % n_mtiles;
  const int rest = tile / n_mtiles;
  const int ks = rest % ksplit;
  const int nb = rest / ksplit;
  int m_live = M;
  if constexpr (EPI == EPI_HEAD) m_live = ep.list[0];
  const int n0 = nb * BN;
  // M tiles mb, mb + n_mtiles, ... (one tile unless the grid is narrower
  // than the rows: the vocabulary head sizes it for the live rows)
  for (int mt = mb; mt * BM < m_live; mt += n_mtiles) {
  const int m0 = mt * BM;
  if (mt != mb) __syncthreads();      // LDS of the previous tile retired
  const int nk_all = K / BK;
  const int chunk = (nk_all + ksplit - 1) / ksplit;
  const int kt0 = ks * chunk;
  const int nk = min(nk_all, kt0 + chunk) - kt0;

  const int t = threadIdx.x;
  const int lane = t & 63;
  // wave-uniform values live in scalar registers (branches on them are
  // scalar, not exec-masked)
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, hh = lane >> 5;
  const int l16 = lane & 15, k4 = lane >> 4;
  const bool dual = (EPI == EPI_SWIGLU) || (EPI == EPI_PARTIAL && ep.dual);

  // ---- per-lane sources of this wave's load instructions (fixed over K)
  const uint16_t* a_src[AI];
  const uint16_t* b_src[BI];
#pragma unroll
  for (int q = 0; q < AI; ++q) {
    const int r = (wave * AI + q) * RPI + lane / CPR;
    const int c = (lane % CPR) ^ ((r / (16 / CPR)) % CPR);
    const int gm = min(m0 + r, m_live - 1);
    a_src[q] = A + (size_t)gm * K + (size_t)kt0 * BK + c * 8;
  }
#pragma unroll
  for (int q = 0; q < BI; ++q) {
    const int r = (wave * BI + q) * RPI + lane / CPR;
    const int c = (lane % CPR) ^ ((r / (16 / CPR)) % CPR);
    const uint16_t* base = B;
    int gn;
    if (dual) {
      const int half = BN / 2;
      base = r < half ? B : B2;
      gn = nb * half + (r < half ? r : r - half);
    } else {
      gn = min(n0 + r, N - 1);
    }
    if (ep.b_tiled)
      b_src[q] = B + ((size_t)min(nb * (BN / 128) + (r >> 7), (N - 1) >> 7) * 128 +
                      (r & 127)) * 64 + c * 8;
    else
      b_src[q] = base + (size_t)gn * K + (size_t)kt0 * BK + c * 8;
  }
  const size_t b_kstride =
      ep.b_tiled ? (size_t)((N + 127) / 128) * 128 * 64 : (size_t)BK;

  // A load instructions of this wave holding at least one live row: rows
  // past the last live one are not fetched (their LDS rows feed only output
  // rows that are never stored).  The count is wave-uniform, so the per-slab
  // load count LPT_live of each wave is too.
  const int na = __builtin_amdgcn_readfirstlane(
      max(0, min(AI, (m_live - m0 - wave * AI * RPI + RPI - 1) / RPI)));
  const int lpt_live = na + BI;
  auto issue = [&](int stage, int kt) {
    char* sa = smem + stage * S_BYTES;
    char* sb = sa + A_BYTES;
#pragma unroll
    for (int q = 0; q < AI; ++q)
      if (q < na) dma16(a_src[q] + (size_t)kt * BK, sa + (wave * AI + q) * 1024);
    const int kel = (kt0 + kt) * BK;       // first K element of the slab
    const size_t boff = ep.b_tiled ? (size_t)(kel >> 6) * b_kstride + (kel & 63)
                                   : (size_t)kt * b_kstride;
#pragma unroll
    for (int q = 0; q < BI; ++q)
      dma16(b_src[q] + boff, sb + (wave * BI + q) * 1024);
  };

  // acc[i][j][q]: the 16 x 16 block (q / QC, q % QC) of the wave's
  // 32 x CW block (i, j), one v_mfma_f32_16x16x32 accumulator each
  f32x4 acc[TM][TN][NQ];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[i][j][q][e] = 0.f;

  // 32-row sub-tiles of this wave holding live rows: always a prefix, NL of
  // them.  The K loop is instantiated per NL, so its body has no branch
  // between the LDS fragment reads and the matrix ops.
  const int nl = max(0, min(TM, (m_live - m0 - wm * WROWS + 31) / 32));

#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) issue(s, s);

  auto k_loop = [&](auto nl_c) {
    constexpr int NL = decltype(nl_c)::value;
    for (int it = 0; it < nk; ++it) {
      // slab `it` must have landed; later slabs may still be in flight
      const int ahead = min(STAGES - 2, nk - 1 - it);
      static_assert((STAGES - 2) * LPT <= 63, "vmcnt range");
      wait_vmcnt_rt<0, (STAGES - 2) * LPT>(ahead * lpt_live);
      barrier_nofence();        // slab visible to all waves; slab it-1 retired
      if (it + STAGES - 1 < nk) issue((it + STAGES - 1) % STAGES, it + STAGES - 1);
      if constexpr (NL > 0) {
        const char* sa = smem + (it % STAGES) * S_BYTES;
        const char* sb = sa + A_BYTES;
        // 32-deep K steps of 16 x 16 x 32 matrix ops: lane l supplies row
        // (or column) l % 16 of a 16-row fragment and k = 8 (l / 16) .. +7,
        // i.e. 16-byte chunk 4 kk + l / 16 of that LDS row
        if constexpr (V::IGLP >= 0) __builtin_amdgcn_iglp_opt(V::IGLP);
#pragma unroll
        for (int kk = 0; kk < BK / 32; ++kk) {
          const int c = kk * 4 + k4;
          v8 af[NL][2], bfr[TN][QC];
#pragma unroll
          for (int i = 0; i < NL; ++i)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int r = wm * WROWS + i * 32 + h * 16 + l16;
              af[i][h] = *reinterpret_cast<const v8*>(sa + swz<BK>(r, c));
            }
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int h = 0; h < QC; ++h) {
              const int r = j * 64 + wn * CW + h * 16 + l16;
              bfr[j][h] = *reinterpret_cast<const v8*>(sb + swz<BK>(r, c));
            }
#pragma unroll
          for (int i = 0; i < NL; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
              for (int q = 0; q < NQ; ++q)
                acc[i][j][q] = Fmt::mfma16(af[i][q / QC], bfr[j][q % QC],
                                           acc[i][j][q]);
        }
        if constexpr (V::SG == 1) {
          static_assert(BK == 64 && V::IGLP < 0, "two 32-deep steps, no strategy");
          constexpr int DS_READ = 0x100, MATRIX = 0x008;   // group masks
          constexpr int R = NL * 2 + TN * QC;   // fragment reads per step
          constexpr int MO = NL * TN * NQ;      // matrix ops per step
          static_assert(MO >= R, "a read per matrix op");
          __builtin_amdgcn_sched_group_barrier(DS_READ, R, 0);
#pragma unroll
          for (int r = 0; r < R; ++r) {
            __builtin_amdgcn_sched_group_barrier(DS_READ, 1, 0);
            __builtin_amdgcn_sched_group_barrier(MATRIX, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(MATRIX, 2 * MO - R, 0);
        }
      }
    }
  };
  static_assert(TM <= 4, "live-prefix dispatch covers up to 4 sub-tiles");
  switch (nl) {
    case 0: k_loop(std::integral_constant<int, 0>{}); break;
    case 1: k_loop(std::integral_constant<int, 1>{}); break;
    case 2: k_loop(std::integral_constant<int, (TM >= 2 ? 2 : TM)>{}); break;
    case 3: k_loop(std::integral_constant<int, (TM >= 3 ? 3 : TM)>{}); break;
    default: k_loop(std::integral_constant<int, TM>{}); break;
  }

  // ---------------------------------------------------------------- epilogue
  // acc[i][j][q][u]: row = wm*WROWS + i*32 + (q/QC)*16 + (lane/16)*4 + u,
  //                  col = j*64 + wn*CW + (q%QC)*16 + lane%16   (tile-local)
  // so a lane's column in each 64-column group j is wn*CW + (q%QC)*16 + l16
  int nf = 0;     // non-finite 16-bit values stored by this lane
  const int rrow = k4 * 4;
  if constexpr (EPI == EPI_STORE) {
    uint16_t* C = reinterpret_cast<uint16_t*>(ep.C);
    const bool rope = ep.pos && n0 < ep.rope_cols;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int row = m0 + wm * WROWS + i * 32 + (q / QC) * 16 + rrow + u;
          if (row >= M) continue;
          const int cl = wn * CW + (q % QC) * 16 + l16;
          uint16_t* crow = C + (size_t)row * ep.ldc + n0 + cl;
          if (rope) {
            // j even / j+1: dims cl and cl+64 of the head starting at n0 + j*64
            const float2 c = ep.cs[(size_t)ep.pos[row] * 64 + cl];
#pragma unroll
            for (int j = 0; j < TN; j += 2) {
              const float x = acc[i][j][q][u], y = acc[i][j + 1][q][u];
              const uint16_t a = Fmt::store(x * c.x - y * c.y);
              const uint16_t b = Fmt::store(y * c.x + x * c.y);
              nf += Fmt::nonfinite(a) + Fmt::nonfinite(b);
              crow[j * 64] = a;
              crow[(j + 1) * 64] = b;
            }
          } else {
#pragma unroll
            for (int j = 0; j < TN; ++j) {
              const uint16_t a = Fmt::store(acc[i][j][q][u]);
              nf += Fmt::nonfinite(a);
              crow[j * 64] = a;
            }
          }
        }
  } else if constexpr (EPI == EPI_ADD_F32) {
    float* C = reinterpret_cast<float*>(ep.C);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int row = m0 + wm * WROWS + i * 32 + (q / QC) * 16 + rrow + u;
          if (row >= M) continue;
          float* crow = C + (size_t)row * ep.ldc + n0 + wn * CW + (q % QC) * 16 + l16;
#pragma unroll
          for (int j = 0; j < TN; ++j) crow[j * 64] += acc[i][j][q][u];
        }
  } else if constexpr (EPI == EPI_SWIGLU) {
    uint16_t* C = reinterpret_cast<uint16_t*>(ep.C);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int row = m0 + wm * WROWS + i * 32 + (q / QC) * 16 + rrow + u;
          if (row >= M) continue;
          uint16_t* crow = C + (size_t)row * ep.ldc + nb * (BN / 2) + wn * CW +
                           (q % QC) * 16 + l16;
#pragma unroll
          for (int j = 0; j < TN / 2; ++j) {
            const float g = acc[i][j][q][u], up = acc[i][j + TN / 2][q][u];
            const uint16_t h = Fmt::store(g / (1.0f + __expf(-g)) * up);
            nf += Fmt::nonfinite(h);
            crow[j * 64] = h;
          }
        }
  } else if constexpr (EPI == EPI_PARTIAL) {
    float* P = ep.part + (size_t)ks * M * ep.part_ld;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int row = m0 + wm * WROWS + i * 32 + (q / QC) * 16 + rrow + u;
          if (row >= M) continue;
          float* prow = P + (size_t)row * ep.part_ld;
          const int cl = wn * CW + (q % QC) * 16 + l16;
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            int col;
            if (ep.dual) {       // gate half -> [0, F), up half -> [F, 2F)
              const int jj = j % (TN / 2);
              col = (j < TN / 2 ? 0 : ep.ffn) + nb * (BN / 2) + jj * 64 + cl;
            } else {
              col = n0 + j * 64 + cl;
            }
            prow[col] = acc[i][j][q][u];
          }
        }
  } else {   // EPI_HEAD
    __shared__ float red_m[2][BM];
    __shared__ float red_s[2][BM];
    __shared__ int red_a[2][BM];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int qr = 0; qr < 2; ++qr) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int lrow = wm * WROWS + i * 32 + qr * 16 + rrow + u;
          const int row = m0 + lrow;
          float m = -INFINITY, s = 0.f;
          int a = 0x7fffffff;
          // this lane's columns of the row, ascending: j*64 + wn*32 +
          // qc*16 + l16 for j, then qc
#pragma unroll
          for (int j = 0; j < TN; ++j) {
#pragma unroll
            for (int qc = 0; qc < 2; ++qc) {
              const int col = n0 + j * 64 + wn * 32 + qc * 16 + l16;
              float v = acc[i][j][qr * 2 + qc][u];
              if (ep.logits_out && row < m_live && col < ep.vocab)
                ep.logits_out[(size_t)ep.list[1 + row] * ep.vocab + col] = v;
              if (col == ep.mask_id || col >= ep.vocab) v = -INFINITY;
              if (v > m) {              // columns ascend: keeps the first
                s = s * __expf(m - v) + 1.0f;
                m = v; a = col;
              } else if (v != -INFINITY) {
                s += __expf(v - m);
              }
            }
          }
          // the 16 lanes holding this row (same lane / 16)
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) {
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
          if (l16 == 0) {
            red_m[wn][lrow] = m;
            red_s[wn][lrow] = s;
            red_a[wn][lrow] = a;
          }
        }
      }
    }
    __syncthreads();
    for (int r = t; r < BM; r += 64 * WAVES) {
      const int row = m0 + r;
      if (row >= m_live) continue;
      const float m1 = red_m[0][r], m2 = red_m[1][r];
      const float mm = fmaxf(m1, m2);
      float s = 0.f;
      if (m1 != -INFINITY) s += red_s[0][r] * __expf(m1 - mm);
      if (m2 != -INFINITY) s += red_s[1][r] * __expf(m2 - mm);
      const int a1 = red_a[0][r], a2 = red_a[1][r];
      const int a = (m2 > m1 || (m2 == m1 && a2 < a1)) ? a2 : a1;
      const size_t o = (size_t)row * ep.n_slabs + nb;
      ep.pmax[o] = mm;
      ep.psum[o] = s;
      ep.parg[o] = a;
    }
  }
  if (nf && ep.overflow) atomicAdd(ep.overflow, nf);
  }  // M tiles
}

template <typename Fmt, typename V, int EPI>
int launch_tiles(const uint16_t* A, const uint16_t* B, const uint16_t* B2,
                 int M, int N, int K, int ksplit, const EpiArgs& ep,
                 hipStream_t s, int max_mtiles = 1 << 30) {
  const int mt = std::min((M + V::BM - 1) / V::BM, max_mtiles);
  const int nt = (N + V::BN - 1) / V::BN;
  const int nwg = mt * nt * ksplit;
  hipLaunchKernelGGL((gemm16_kernel<Fmt, V, EPI>), dim3(nwg),
                     dim3(64 * V::WAVES), 0, s, A, B, B2, M, N, K, mt, nt,
                     ksplit, ep);
  DAVET_HIP(hipGetLastError());
  return DAVET_OK;
}

// The kernel variants the planner can pick (index = GemmPlan::tile; the
// indices are those of the measurement tables, other tiles measured slower).
using V0 = Var<128, 128, 32, 4, 4>;    // 64 KB LDS, 2 workgroups per CU
// V6 with the scheduler's interleaving strategy 1: measured on MI355X
// (candidates interleaved launch by launch, cold weights) never slower on any
// table entry that uses it, median 5 % faster; the 256 x 256 and 8-wave
// 128 x 128 tiles gain nothing from it.  V14 with explicit schedule groups
// (SG = 1): 4-8 % faster than with strategy 0 on each of nine products at
// 300-2916 rows, on three parts
using V6 = Var<128, 128, 64, 2, 4, 1>; // 64 KB, 2 workgroups per CU
using V8 = Var<256, 256, 64, 2, 8>;    // 128 KB, deep slabs, large M
using V12 = Var<128, 128, 64, 2, 8>;   // 64 KB, 8 wavefronts, 2 WG/CU
using V13 = Var<256, 256, 64, 2, 16>;  // 128 KB, 16 wavefronts
// 192-row tiles: fewer padded rows and a fuller last wave of workgroups for
// sequences of ~700-3000 tokens (3 sub-tiles of 32 rows per wave)
using V14 = Var<192, 128, 64, 2, 4, -1, 2, 1>; // 80 KB, 2 workgroups per CU
using V15 = Var<128, 256, 32, 3, 8>;   // 72 KB: tiled vocabulary head
// V13's tile with the 16 wavefronts in a 4 x 4 grid (64 x 64 per wave
// instead of 32 x 128: a fifth fewer LDS fragment bytes per matrix op) and
// the scheduler's interleaving strategy 0; same accumulation order per
// output, so bit-identical to V13
using V16 = Var<256, 256, 64, 2, 16, 0, 4>;

int variant_bn(int tile) {
  switch (tile) {
    case 8: case 13: case 15: case 16: return 256;
    default: return 128;
  }
}
int variant_bm(int tile) {
  switch (tile) {
    case 14: return 192;
    case 8: case 13: case 16: return 256;
    default: return 128;
  }
}
int variant_bk(int tile) {
  return (tile == 0 || tile == 15) ? 32 : 64;
}
bool variant_known(int tile) {
  return tile == 0 || tile == 6 || tile == 8 || (tile >= 12 && tile <= 14) ||
         tile == 16;
}

template <typename Fmt, int EPI>
int launch_shape(const GemmPlan& p, const uint16_t* A, const uint16_t* B,
                 const uint16_t* B2, int M, int N, int K, const EpiArgs& ep,
                 hipStream_t s) {
#define LV(Vn) return launch_tiles<Fmt, Vn, EPI>(A, B, B2, M, N, K, p.ksplit, ep, s)
  switch (p.tile) {
    case 6: LV(V6);
    case 8: LV(V8);
    case 12: LV(V12);
    case 13: LV(V13);
    case 14: LV(V14);
    case 16: LV(V16);
    default: LV(V0);
  }
#undef LV
}

template <typename Fmt>
int gemm_dispatch(const GemmPlan& p, int epi, const uint16_t* A,
                  const uint16_t* B, const uint16_t* B2, int M, int N, int K,
                  const EpiArgs& ep, hipStream_t s) {
  if (p.ksplit > 1)
    return launch_shape<Fmt, EPI_PARTIAL>(p, A, B, B2, M, N, K, ep, s);
  switch (epi) {
    case EPI_STORE: return launch_shape<Fmt, EPI_STORE>(p, A, B, B2, M, N, K, ep, s);
    case EPI_ADD_F32: return launch_shape<Fmt, EPI_ADD_F32>(p, A, B, B2, M, N, K, ep, s);
    case EPI_SWIGLU: return launch_shape<Fmt, EPI_SWIGLU>(p, A, B, B2, M, N, K, ep, s);
  }
  return set_error(DAVET_EINVAL, "gemm16: unknown epilogue");
}

}  // namespace

// Kernel choice.  For the projections of a d = 4096, ffn = 12288 layer the
// plan is a table measured on MI355X with the weights and activations cold in
// the last-level cache (as inside a denoising step) at 26 token counts: the
// fastest (tile variant, K split) of a sweep over the variants 6, 8, 12, 13,
// 14 and splits {1, 2, 3, 4, 6, 8}, the split-K reduction included (a
// variant replaced the previous choice only when more than 3 % faster); a
// re-sweep on random data with 5-way splits added changed three entries that
// another plan beat by more than 5 % in both of two repetitions (a fourth,
// QKV at 209 rows with 5 splits, measured 1.2 % slower inside the step: its
// larger partials cost the reduction more than the sweep's cold-cache timing
// shows, and was left out).  After the move to 16 x 16 x 32 matrix ops a
// third sweep (variants 4, 6-9 and 12-14, splits 1-6 and 8, the split-K
// reduction or the following norm included) changed thirteen entries whose
// new plan was more than 4 % faster in each of three repetitions.  The
// 4 x 4-wave tile (V16) then replaced V13 wherever it was not slower, timed
// interleaved on every entry: median 5.8 % faster, bit-identical outputs.
// A last interleaved sweep over the current variants (6, 8, 12, 13, 14, 16
// with their scheduling hints, splits 1-6 and 8) moved 21 entries whose new
// plan was at least 3 % faster; a check of gate/up at 330-520 rows on two
// parts then moved three more (192 x 128 at 356, 4 x 4-wave 256 x 256 at 420
// and 480: 12 % and 6 % faster), and one at 150-250 rows (8-wave 128 x 128
// without a K split instead of 256 x 256 with two: 2-14 % faster).
// Because the number of row tiles and of waves of workgroups changes in
// steps, the best plan is jagged in M; a product of M rows takes the plan of
// the nearest sample point in log M, except in the ranges of kEdge.
constexpr int kPointM[] = {209, 300, 356, 420, 480, 565, 650, 750, 889,
                           960, 1100, 1300, 1500, 1700, 2048, 2300, 2600,
                           2916, 3092, 3300, 3645, 3965, 5000, 8000, 12000,
                           18020};
constexpr int kNP = 26;
struct TableShape { int N, K; GemmPlan plan[kNP]; };
constexpr TableShape kTable[] = {
    // QKV: N = 3d, K = d
    {12288, 4096, {{8, 5}, {16, 2}, {13, 2}, {16, 2}, {16, 2}, {12, 1}, {16, 3}, {14, 1}, {16, 1}, {16, 1}, {16, 1}, {14, 2}, {14, 2}, {12, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}}},
    // output projection: N = d, K = d
    {4096, 4096, {{6, 8}, {6, 5}, {6, 4}, {6, 4}, {12, 4}, {6, 3}, {6, 2}, {12, 2}, {16, 4}, {6, 2}, {16, 3}, {14, 2}, {14, 2}, {16, 2}, {6, 1}, {14, 1}, {14, 1}, {14, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}}},
    // gate + up: N = 2 ffn, K = d
    {24576, 4096, {{12, 1}, {14, 1}, {14, 1}, {16, 1}, {16, 1}, {12, 1}, {14, 1}, {14, 1}, {14, 1}, {14, 1}, {16, 1}, {14, 1}, {14, 1}, {16, 1}, {16, 1}, {14, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}}},
    // down projection: N = d, K = ffn
    {4096, 12288, {{12, 8}, {14, 8}, {16, 8}, {16, 8}, {8, 8}, {16, 5}, {16, 5}, {8, 5}, {16, 4}, {16, 4}, {16, 3}, {14, 2}, {14, 2}, {16, 2}, {16, 2}, {8, 3}, {14, 1}, {14, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 1}, {16, 2}, {16, 1}, {16, 1}, {16, 1}}},
};

// Row counts just past a multiple of a point's tile height, where the point's
// plan would add a nearly empty row tile the point itself does not have: the
// plan measured there instead (each range timed at one row count inside it,
// interleaved against the point's plan: 3-35 % faster; ranges where the next
// point's plan was not faster keep the point's own).
struct EdgeRange { int N, K, lo, hi; GemmPlan plan; };
constexpr EdgeRange kEdge[] = {
    {12288, 4096, 513, 520, {12, 1}},   {12288, 4096, 1537, 1596, {12, 1}},
    {4096, 4096, 513, 520, {6, 3}},     {4096, 4096, 1025, 1027, {16, 3}},
    {4096, 4096, 1537, 1596, {16, 2}},  {4096, 4096, 1793, 1865, {6, 1}},
    {4096, 4096, 2049, 2170, {14, 1}},
    {24576, 4096, 385, 386, {16, 1}},   {24576, 4096, 513, 520, {12, 1}},
    {24576, 4096, 961, 1027, {16, 1}},  {24576, 4096, 1537, 1596, {16, 1}},
    {24576, 4096, 2049, 2170, {14, 1}}, {24576, 4096, 2305, 2445, {16, 1}},
    {4096, 12288, 513, 520, {16, 5}},   {4096, 12288, 769, 816, {16, 4}},
    {4096, 12288, 1025, 1027, {16, 3}}, {4096, 12288, 1537, 1596, {16, 2}},
    {4096, 12288, 2049, 2170, {16, 3}}, {4096, 12288, 4097, 4352, {16, 2}},
};

// Point i serves the rows up to the geometric mean of points i and i+1.
static int point_index(int M) {
  int i = 0;
  while (i + 1 < kNP && (double)M * M > (double)kPointM[i] * kPointM[i + 1]) ++i;
  return i;
}
static int point_top(int i) {            // largest M served by point i
  if (i + 1 >= kNP) return 1 << 30;
  int m = (int)std::sqrt((double)kPointM[i] * kPointM[i + 1]);
  while ((double)(m + 1) * (m + 1) <= (double)kPointM[i] * kPointM[i + 1]) ++m;
  while ((double)m * m > (double)kPointM[i] * kPointM[i + 1]) --m;
  return m;
}

static const TableShape* table_shape(int N, int K) {
  for (const TableShape& t : kTable)
    if (t.N == N && t.K == K) return &t;
  return nullptr;
}

// Other shapes: 128 x 128 tiles with 128-byte slabs and two workgroups per CU
// up to ~2-3K rows, 256 x 256 tiles with 16 wavefronts (4 x 4) above; narrow-N
// products split K until the grid fills the 256 CUs (tiles * ksplit < 512).
static GemmPlan plan_generic(int M, int N, int K) {
  GemmPlan p{};
  const bool big = M >= (N >= 16384 ? 2048 : 3000);
  p.tile = (big && N % 256 == 0 && K % 64 == 0) ? 16 : (K % 64 == 0 ? 6 : 0);
  const int bm = variant_bm(p.tile), bn = variant_bn(p.tile);
  const int tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  const int nk = K / variant_bk(p.tile);
  p.ksplit = 1;
  if (N < 8192)
    while (tiles * p.ksplit < 256 && nk / (p.ksplit * 2) >= 16 && p.ksplit < 8)
      p.ksplit *= 2;
  return p;
}

GemmPlan plan_gemm16(int M, int N, int K) {
  if (const TableShape* t = table_shape(N, K)) {
    for (const EdgeRange& e : kEdge)
      if (e.N == N && e.K == K && M >= e.lo && M <= e.hi) return e.plan;
    return t->plan[point_index(M)];
  }
  return plan_generic(M, N, K);
}

// Largest split-K partial buffer (bytes) any M <= max_M needs.  Table shapes:
// within a run of rows that share one plan the size grows with M, so the
// bound is reached at the top of a point's range, of an edge range or of the
// rows below an edge range (or at max_M).  Other shapes: tiles * ksplit
// < 512 caps it at 512 tiles of at most 256 x 256.
size_t gemm16_partial_bound(int max_M, int N, int K) {
  size_t best = 0;
  auto at = [&](int m) {
    if (m < 1) return;
    const GemmPlan p = plan_gemm16(m, N, K);
    if (p.ksplit > 1) best = std::max(best, (size_t)p.ksplit * m * N * 4);
  };
  if (table_shape(N, K)) {
    for (int i = 0; i < kNP; ++i) at(std::min(max_M, point_top(i)));
    for (const EdgeRange& e : kEdge)
      if (e.N == N && e.K == K) {
        at(std::min(max_M, e.lo - 1));
        at(std::min(max_M, e.hi));
      }
    at(max_M);
    return best;
  }
  return (size_t)512 * 256 * 256 * 4;
}

int launch_gemm16(int dtype, int epi, const GemmPlan& plan, const uint16_t* A,
                  const uint16_t* B, const uint16_t* B2, void* C, int M, int N,
                  int K, int ldc, const int32_t* pos, const float* cs,
                  int rope_cols, float* partials, size_t partial_cap, int cls,
                  hipStream_t s, int32_t* overflow) {
  if (M <= 0) return DAVET_OK;
  if (plan.ksplit > 1 && (size_t)plan.ksplit * M * N * 4 > partial_cap)
    return set_error(DAVET_ENOMEM, "gemm16: split-K partials exceed the workspace");
  if (!variant_known(plan.tile))
    return set_error(DAVET_EINVAL, "gemm16: unknown tile variant");
  if (N % variant_bn(plan.tile) || K % variant_bk(plan.tile) ||
      (plan.ksplit > 1 && (K / variant_bk(plan.tile)) < plan.ksplit))
    return set_error(DAVET_ESHAPE, "gemm16: N or K not a multiple of the tile");
  if (plan.ksplit > 1 && !partials)
    return set_error(DAVET_EINVAL, "gemm16: split-K needs a partial buffer");
  ProfScope ps(cls, s);
  EpiArgs ep{};
  ep.C = C;
  ep.ldc = ldc;
  ep.pos = pos;
  ep.cs = reinterpret_cast<const float2*>(cs);
  ep.rope_cols = rope_cols;
  ep.part = partials;
  ep.part_ld = N;
  ep.dual = epi == EPI_SWIGLU;
  ep.ffn = N / 2;
  ep.overflow = overflow;
  return dtype == DAVET_F16
             ? gemm_dispatch<F16>(plan, epi, A, B, B2, M, N, K, ep, s)
             : gemm_dispatch<BF16>(plan, epi, A, B, B2, M, N, K, ep, s);
}

// The head kernel a launch runs, for a bound `live` on its live rows.  The
// tiled layout streams 256-column slabs: while at most 128 rows (or an odd
// number of 128-row tiles up to five) are live, 128 x 256 tiles with a
// 32-deep ring (V15: each activation tile re-read for half as many slabs as
// with 128-column slabs, one round of 494 workgroups; measured on MI355X at
// V = 126464, d = 4096: 188 -> 181 us at 2 live rows, 262 -> 232 at 128
// against 128 x 128 tiles); otherwise the head is bound by its matrix work
// and takes the 256 x 256 projection tile (V13; 192 rows 369 -> 295 us, 1024
// rows 1361 -> 1198, 2048 rows 2835 -> 2433), whose cost steps with every
// 256 rows where V15's steps with every 128.  Both read the same columns per
// lane, so logits and slab partials are the same bits whichever runs.  The
// row-major layout takes 128 x 128 tiles with 8 wavefronts.
static int head16_variant(int tiled, int live) {
  if (!tiled) return 12;
  const int n128 = (std::max(live, 1) + 127) / 128;
  return (n128 == 1 || (n128 % 2 == 1 && n128 <= 5)) ? 15 : 13;
}

int head16_slabs(int vocab, int tiled, int live_bound) {
  const int bn = variant_bn(head16_variant(tiled, live_bound));
  return (vocab + bn - 1) / bn;
}

int launch_head16(int dtype, const uint16_t* Hm, const uint16_t* W,
                  const int32_t* list, int max_rows, int vocab, int d,
                  int mask_id, float* pmax, float* psum, int32_t* parg,
                  float* logits_out, hipStream_t s, int tiled,
                  int live_bound) {
  // Row-major head: 8 wavefronts on the 128 x 128 tile (V12 over V6): the
  // matrix work of a slab is spread over twice the waves, so it hides behind
  // the other workgroup's stream (measured on MI355X: 201 -> 187 us at 2 live
  // rows, 214 -> 192 at 64)
  const int live = live_bound < 0 ? max_rows : std::min(max_rows, live_bound);
  const int variant = head16_variant(tiled, live);
  if (d % BK_MIN) return set_error(DAVET_ESHAPE, "head16: d % 32 != 0");
  ProfScope ps(KC_HEAD, s);
  EpiArgs ep{};
  ep.list = list;
  ep.vocab = vocab;
  ep.mask_id = mask_id;
  ep.n_slabs = head16_slabs(vocab, tiled, live);
  ep.pmax = pmax;
  ep.psum = psum;
  ep.parg = parg;
  ep.logits_out = logits_out;
  ep.b_tiled = tiled;
  if (tiled && d % 64)
    return set_error(DAVET_EINVAL, "head16: the tiled head needs d % 64 == 0");
  // m_slots M slots per vocabulary slab: a workgroup loops over the live row
  // tiles mb, mb + m_slots, ...  m_slots covers live_bound, a bound on the
  // live rows the caller knows on the host (the schedule loop's: at most
  // L - k(t-1) per sequence; a looser bound is still correct), so one slot
  // per live tile streams a slab's weights from HBM once (the tiles of a slab
  // sit on one XCD and share its L2), and late steps with few masked rows
  // launch no idle workgroups.
  const int bm = variant_bm(variant);
  const int m_slots = std::max(1, (live + bm - 1) / bm);
#define HV(Fmt, Vn) return launch_tiles<Fmt, Vn, EPI_HEAD>(Hm, W, nullptr, max_rows, vocab, d, 1, ep, s, m_slots)
#define HEAD_VARIANTS(Fmt)       \
  switch (variant) {             \
    case 12: HV(Fmt, V12);       \
    case 13: HV(Fmt, V13);       \
    case 15: HV(Fmt, V15);       \
  }
  if (dtype == DAVET_F16) {
    HEAD_VARIANTS(F16)
  } else {
    HEAD_VARIANTS(BF16)
  }
  return set_error(DAVET_EINVAL, "head16: no such head variant");
#undef HEAD_VARIANTS
#undef HV
}

}  // namespace davet
