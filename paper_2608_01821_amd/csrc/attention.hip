// Bidirectional (non-causal) attention over a packed batch of independent
// sequences (Sec. 1 and Sec. 3.1: dVLMs refine all answer positions in
// parallel through bidirectional attention).  Every query of a sequence sees
// every key of the same sequence; sequences never mix.
//
// 16-bit path (bf16 or fp16 operands), head_dim 128, CDNA4 matrix cores.  A
// workgroup owns 128 queries of one head and runs SPLIT (1 or 2) groups of 4
// wavefronts; group g takes the key tiles g, g + SPLIT, ... and each of its
// wavefronts owns 32 queries.  Keys stream in tiles of 64: global->LDS DMA
// moves each K and V tile row-major into LDS (16-byte chunks XOR-swizzled per
// row, so no padding is needed for conflict-free reads; the V^T fragments
// come from the CDNA4 transposing LDS read ds_read_b64_tr_b16).  With two
// groups each has two buffers, the next tile landing in one while the other
// feeds the matrix cores; with one group a single buffer lets three
// workgroups share a CU and overlap each other's loads.  Per tile a
// wavefront computes
// S^T = K Q^T (2 x 8 v_mfma_f32_32x32x16 ops), so every lane holds the scores
// of ONE query: the online-softmax rescale is a per-lane scalar and the
// probabilities, rounded to 16 bits, are already laid out as the B operand of
// O^T += V^T P^T (4 x 4 MFMAs) -- no LDS round trip for P.  Scores, running
// max and normaliser stay in fp32 (exp2 with log2(e) folded into the
// 1/sqrt(D) scale).  The groups' partial (max, normaliser, O) are merged
// through LDS at the end.  Ragged tails: keys past the sequence end score
// -inf; queries past it are computed on clamped rows and never stored.
// Workgroup ids are remapped so the full query tiles of a head share an XCD
// (and its L2 copy of that head's keys and values); the ragged last tile of
// each sequence (fewer than 128 queries) is dispatched after every full tile,
// so that when the grid is slightly larger than one wave of workgroups the
// work left for the second wave is the cheap part, and a wavefront whose 32
// queries all lie past the sequence end only moves K/V and meets the
// barriers.  The running maximum moves lazily: a lane adopts a new maximum
// only when a score exceeds the current one by more than 2^8 in probability
// (the probabilities, at most 2^8, stay well inside the 16-bit range and the
// normaliser is an fp32 sum), so the O rescale is rare after the first tiles.
//
// Key-range split: when the query tiles alone would leave CUs idle (short
// sequences), or leave a second round of workgroups for the ragged tiles,
// a query tile's keys are divided among S workgroups ("pieces", contiguous
// ranges of key tiles).  Each piece writes its (max, normaliser, unnormalised
// O) in fp32 to a partial slot, and attn_merge_kernel combines the S pieces
// in piece order (the result does not depend on which piece finishes first).

#include "common.h"

#include <algorithm>
#include <atomic>

namespace davet {
namespace {

constexpr int HD = 128;           // head dim of the matrix-core path
constexpr int QT = 128;           // queries per workgroup
constexpr int KT = 64;            // keys per tile
constexpr int TILE_U16 = KT * HD;            // one 64 x 128 K or V tile
constexpr int BUF_U16 = 2 * TILE_U16;        // K and V of one key tile

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s* lds_v4s_ptr;
typedef __attribute__((address_space(3))) void* lds_ptr;

__device__ __forceinline__ void dma16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_ptr)lds, 16, 0, 0);
}
// 16-byte chunk slot of chunk c of key row r.  K: XOR by r % 16, so the 16
// rows a fragment read touches at one chunk cover all 64 banks.  V: XOR by
// 4 (r % 4), moving whole 64-byte groups, so the 64-byte row pieces of four
// consecutive keys that a transposing read takes cover all banks.
__device__ __forceinline__ int k_slot(int r, int c) { return c ^ (r & 15); }
__device__ __forceinline__ int v_slot(int r, int c) { return c ^ ((r & 3) << 2); }

// x combined with the value of lane l ^ 32: v_permlane32_swap exchanges the
// upper half of one copy with the lower half of the other, so the two
// results hold, in every lane, x of that lane and of its partner
__device__ __forceinline__ float pair_max32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                                  __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                                  __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup barrier with no memory fence: each wave has waited for exactly
// the loads it needs; the empty asm statements keep LDS accesses in place.
__device__ __forceinline__ void sync_lds() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ int remap_xcd_attn(int bid, int nwg) {
  const int full = nwg & ~7;
  if (bid >= full) return bid;
  const int per = full >> 3;
  return (bid & 7) * per + (bid >> 3);
}

// Full query tile `tile` (in sequence order) -> sequence s and its tile qt.
__device__ __forceinline__ void locate_full(const SeqPack& sp, int tile,
                                            int qtile, int& s, int& qt) {
  s = 0;
  int acc = 0;
  for (;;) {
    const int nt = (sp.row0[s + 1] - sp.row0[s]) / qtile;
    if (tile < acc + nt || s + 1 >= sp.n_seqs) break;
    acc += nt;
    ++s;
  }
  qt = tile - acc;
}
// Ragged tile `r` -> the r-th sequence (in order) whose length is not a
// multiple of qtile, and its last tile.
__device__ __forceinline__ void locate_ragged(const SeqPack& sp, int r,
                                              int qtile, int& s, int& qt) {
  s = 0;
  for (;;) {
    const int n = sp.row0[s + 1] - sp.row0[s];
    if (n % qtile) {
      if (r == 0 || s + 1 >= sp.n_seqs) { qt = n / qtile; return; }
      --r;
    }
    ++s;
    if (s >= sp.n_seqs) { s = sp.n_seqs - 1; qt = 0; return; }
  }
}

// One key group (enough workgroups for the chip), fp16: a single K/V buffer
// per workgroup (32 KB) so three workgroups share a CU and hide each other's
// loads (bf16 rounding needs more registers than three waves per SIMD
// leave: it spills there, so it keeps two buffers at two per CU).  Two key
// groups (few workgroups): two buffers per group, the next tile landing
// during compute.
template <typename Fmt, int SPLIT>
constexpr int attn_bufs() {
  return SPLIT == 1 && Fmt::dtype == DAVET_F16 ? 1 : 2;
}
template <typename Fmt, int SPLIT>
constexpr int attn_minb() {
  return SPLIT == 2 ? 1 : attn_bufs<Fmt, SPLIT>() == 1 ? 3 : 2;
}

template <typename Fmt, int SPLIT>
__global__ void __launch_bounds__(256 * SPLIT, (attn_minb<Fmt, SPLIT>()))
attn16_kernel(const uint16_t* __restrict__ qkv, uint16_t* __restrict__ out,
              SeqPack sp, int n_heads, int n_full, int n_ragged,
              float scale_log2, int s_full, int s_rag,
              float* __restrict__ part) {
  using v8 = typename Fmt::v8;
  // SPLIT groups' double-buffered K/V tiles; after the loop the same bytes
  // hold the merge (O as [4 waves][4][16][64 lanes] floats, then max and
  // normaliser as [4][64] floats each)
  constexpr int BUFS = attn_bufs<Fmt, SPLIT>();
  constexpr int GROUP_LDS = BUFS * BUF_U16;
  constexpr int MERGE_U16 = SPLIT == 2 ? 2 * (QT * HD + 2 * 256) : 0;
  constexpr int LDS_U16 = SPLIT * GROUP_LDS > MERGE_U16 ? SPLIT * GROUP_LDS
                                                        : MERGE_U16;
  __shared__ __attribute__((aligned(1024))) uint16_t smem[LDS_U16];
  // blocks [0, n_heads * n_full * s_full): pieces of the full tiles,
  // head-major, XCD-remapped; then the pieces of the ragged tiles,
  // head-major.  Piece p of S takes key tiles [p*c, min(n_kt, (p+1)*c)),
  // c = ceil(n_kt / S); with S > 1 it writes partial slot `slot`.
  const int n_fb = n_heads * n_full * s_full;
  int h, s, qt, piece, S, slot;
  if ((int)blockIdx.x < n_fb) {
    const int logical = remap_xcd_attn(blockIdx.x, n_fb);
    const int tl = logical / s_full;
    piece = logical % s_full;
    S = s_full;
    slot = logical;
    h = tl / n_full;
    locate_full(sp, tl % n_full, QT, s, qt);
  } else {
    const int r = blockIdx.x - n_fb;
    const int nr = max(n_ragged, 1);
    const int tl = r / s_rag;
    piece = r % s_rag;
    S = s_rag;
    slot = (s_full > 1 ? n_fb : 0) + r;
    h = tl / nr;
    locate_ragged(sp, tl % nr, QT, s, qt);
  }
  const int d = n_heads * HD;
  const size_t ld = (size_t)3 * d;
  const int row0 = sp.row0[s];
  const int N = sp.row0[s + 1] - row0;
  const int t = threadIdx.x;
  const int grp = t >> 8;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane((t >> 6) & 3);
  const int l32 = lane & 31, hh = lane >> 5;
  const int q = qt * QT + wave * 32 + l32;
  const int qc = min(q, N - 1);
  // a wavefront whose queries all lie past the sequence end only moves K/V
  const bool live = qt * QT + wave * 32 < N;
  char* gbuf = reinterpret_cast<char*>(smem + grp * GROUP_LDS);

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
  // tile kb into buffer b: wave w moves rows 16w .. 16w+15 of K and of V, four
  // rows (1 KB) per load instruction; keys past the end repeat the last one
  auto issue = [&](int kb, int b) {
    char* kd = gbuf + b * (BUF_U16 * 2);
    char* vd = kd + TILE_U16 * 2;
    const int k0 = kb * KT;
#pragma unroll
    for (int qi = 0; qi < 4; ++qi) {
      const int r = (wave * 4 + qi) * 4 + (lane >> 4);
      const size_t go = (size_t)min(k0 + r, N - 1) * ld;
      dma16(kbase + go + k_slot(r, lane & 15) * 8, kd + (wave * 4 + qi) * 1024);
      dma16(vbase + go + v_slot(r, lane & 15) * 8, vd + (wave * 4 + qi) * 1024);
    }
  };
  const int n_kt = (N + KT - 1) / KT;
  const int chunk = (n_kt + S - 1) / S;
  const int kt0 = min(n_kt, piece * chunk);
  const int kt1 = min(n_kt, kt0 + chunk);
  const int n_it = (kt1 - kt0 + SPLIT - 1) / SPLIT;  // same for every group

  // the three parts of a key tile's work, on the K and V of one buffer
  auto qk_scores = [&](const char* Kb, f32x16 (&sc)[2]) {
    // ---- S^T = K Q^T for 64 keys x 32 queries (two 32-key halves)
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[mt][e] = 0.f;
      const int r = mt * 32 + l32;
#pragma unroll
      for (int ks = 0; ks < HD / 16; ++ks) {
        const v8 kf = *reinterpret_cast<const v8*>(
            Kb + r * 256 + (k_slot(r, ks * 2 + hh) << 4));
        sc[mt] = Fmt::mfma32(kf, qf[ks], sc[mt]);
      }
    }
  };
  auto softmax = [&](int k0, f32x16 (&sc)[2], uint32_t (&pw2)[4][4]) {
    // ---- online softmax for this lane's query over its 32 keys + partner's.
    // The running max is kept on raw scores (the scale is positive), so
    // each probability costs one fma and one exp2: 2^(s*scale - m*scale).
    if (k0 + KT > N) {                 // ragged last tile only
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = k0 + mt * 32 + (e >> 2) * 8 + hh * 4 + (e & 3);
          if (key >= N) sc[mt][e] = -INFINITY;
        }
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int e = 0; e < 16; ++e) tmax = fmaxf(tmax, sc[mt][e]);
    tmax = pair_max32(tmax);
    // lazy maximum: keep m_run unless a score exceeds it by more than
    // 8 / scale_log2 (probabilities up to 2^8); the first tile always moves
    const float m_new =
        (tmax - m_run) * scale_log2 > 8.0f ? tmax : m_run;
    const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * scale_log2);
    const float neg_m = -m_new * scale_log2;
    float psum = 0.f;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(sc[mt][e], scale_log2, neg_m));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(sc[mt][e + 1], scale_log2, neg_m));
        psum += p0;
        psum += p1;
        pw2[mt * 2 + (e >> 3)][(e & 7) >> 1] = Fmt::store2(p0, p1);
      }
    psum = pair_sum32(psum);
    l_run = l_run * alpha + psum;
    m_run = m_new;
    // rescale the accumulator unless no lane's maximum moved
    if (__any(alpha != 1.0f)) {
#pragma unroll
      for (int i = 0; i < HD / 32; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[i][e] *= alpha;
    }
  };
  auto pv_accumulate = [&](const char* Vb, const uint32_t (&pw2)[4][4]) {
    // ---- O^T += V^T P^T: k-step ps covers keys 16*ps .. 16*ps+15
#pragma unroll
    for (int ps = 0; ps < 4; ++ps) {
#pragma unroll
      for (int dt = 0; dt < HD / 32; ++dt) {
        // V^T fragment by transposing reads of the row-major tile: within
        // each 16-lane group, lane i receives element i % 4 of the 8-byte
        // piece addressed by group lane 4r + i / 4, for r = 0..3; group
        // lane j therefore addresses key ks + 4*(lane / 32) + j / 4 and dims
        // dt*32 + 16*((lane / 16) & 1) + 4*(j % 4), so lane l collects keys
        // ks + 4*(l / 32) + r of dim dt*32 + l % 32 (ks = ps*16, +8 for the
        // second half of the fragment); an 8-byte piece never crosses a
        // 16-byte chunk, so the swizzle moves it whole
        const int j = lane & 15;
        const int r = ps * 16 + hh * 4 + (j >> 2);
        const int dd = dt * 32 + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
        const char* vp = Vb + r * 256 + (v_slot(r, dd >> 3) << 4) + (dd & 7) * 2;
        const v4s t0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_ptr)vp);
        const v4s t1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_v4s_ptr)(vp + 8 * 256));
        const u32x2 v0 = __builtin_bit_cast(u32x2, t0);
        const u32x2 v1 = __builtin_bit_cast(u32x2, t1);
        u32x4 vv;
        vv[0] = v0[0]; vv[1] = v0[1]; vv[2] = v1[0]; vv[3] = v1[1];
        u32x4 pw;
#pragma unroll
        for (int u = 0; u < 4; ++u) pw[u] = pw2[ps][u];
        o[dt] = Fmt::mfma32(__builtin_bit_cast(v8, vv),
                            __builtin_bit_cast(v8, pw), o[dt]);
      }
    }
  };

  if constexpr (BUFS == 1) {
    // one buffer, refilled once every wave is done with it (the other
    // workgroups on the CU hide the load)
    if (kt0 < kt1) issue(kt0, 0);
    for (int kb = kt0; kb < kt1; ++kb) {
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
      sync_lds();
      if (live) {
        f32x16 sc[2];
        qk_scores(gbuf, sc);
        uint32_t pw2[4][4];
        softmax(kb * KT, sc, pw2);
        pv_accumulate(gbuf + TILE_U16 * 2, pw2);
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      sync_lds();
      if (kb + 1 < kt1) issue(kb + 1, 0);
    }
  } else {
    if (kt0 + grp < kt1) issue(kt0 + grp, 0);
    for (int it = 0; it < n_it; ++it) {
      const int kb = kt0 + it * SPLIT + grp;
      const bool have = kb < kt1 && live;
      // this wave's loads of tile kb have landed, and its reads of the other
      // buffer are done; after the barrier, so are every wave's
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
      sync_lds();
      if (kb + SPLIT < kt1) issue(kb + SPLIT, (it + 1) & 1);
      if (have) {
        const char* Kb = gbuf + (it & 1) * (BUF_U16 * 2);
        f32x16 sc[2];
        qk_scores(Kb, sc);
        uint32_t pw2[4][4];
        softmax(kb * KT, sc, pw2);
        pv_accumulate(Kb + TILE_U16 * 2, pw2);
      }
    }
  }

  // The lane's coordinates, derived again after the key loop so that they
  // need not stay live in registers across it (the asm keeps the compiler
  // from reusing the values computed before the loop).
  int lane_e;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\t"
               "v_mbcnt_hi_u32_b32 %0, -1, %0"
               : "=v"(lane_e));
  const int l32e = lane_e & 31, hhe = lane_e >> 5;
  const int qe = qt * QT + wave * 32 + l32e;

  if constexpr (SPLIT == 2) {
    // group 1 hands (max, normaliser, O) of each query to group 0, once both
    // groups are done with their tiles
    __syncthreads();
    float* mo = reinterpret_cast<float*>(smem);
    float* ml = mo + QT * HD;
    if (grp == 1) {
#pragma unroll
      for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          mo[((wave * 4 + dt) * 16 + e) * 64 + lane_e] = o[dt][e];
      ml[wave * 64 + lane_e] = m_run;
      ml[256 + wave * 64 + lane_e] = l_run;
    }
    __syncthreads();
    if (grp == 1) return;
    const float m1 = ml[wave * 64 + lane_e], l1 = ml[256 + wave * 64 + lane_e];
    const float mm = fmaxf(m_run, m1);
    const float a0 = exp2f((m_run - mm) * scale_log2);
    const float a1 = exp2f((m1 - mm) * scale_log2);
    l_run = l_run * a0 + l1 * a1;
#pragma unroll
    for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        o[dt][e] = o[dt][e] * a0 + mo[((wave * 4 + dt) * 16 + e) * 64 + lane_e] * a1;
  }

  if (S > 1) {
    // partial slot: O^T as [HD][QT] floats (lanes of a wave write 32
    // consecutive queries of one dim), then max and normaliser as [2][QT]
    if (qe < N) {
      float* po = part + (size_t)slot * ATT_SLOT_FLOATS;
      const int qr = wave * 32 + l32e;
#pragma unroll
      for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int dd = dt * 32 + (e >> 2) * 8 + hhe * 4 + (e & 3);
          po[dd * QT + qr] = o[dt][e];
        }
      if (hhe == 0) {
        po[HD * QT + qr] = m_run;
        po[HD * QT + QT + qr] = l_run;
      }
    }
    return;
  }
  if (qe < N) {
    const float inv = 1.0f / l_run;
    uint16_t* op = out + (size_t)(row0 + qe) * d + (size_t)h * HD;
#pragma unroll
    for (int dt = 0; dt < HD / 32; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int dd = dt * 32 + g * 8 + hhe * 4;
        u32x2 w;
        w[0] = (uint32_t)Fmt::store(o[dt][g * 4 + 0] * inv) |
               ((uint32_t)Fmt::store(o[dt][g * 4 + 1] * inv) << 16);
        w[1] = (uint32_t)Fmt::store(o[dt][g * 4 + 2] * inv) |
               ((uint32_t)Fmt::store(o[dt][g * 4 + 3] * inv) << 16);
        *reinterpret_cast<u32x2*>(op + dd) = w;
      }
  }
}

// Combines the S key-range pieces of each split query tile: with m the
// largest piece maximum and w_p = 2^((m_p - m) * scale_log2), the output is
// sum_p w_p O_p / sum_p w_p l_p, summed in piece order.  Eight workgroups per
// split tile (tiles of the full class first when s_full > 1, then of the
// ragged class); thread t of workgroup j takes query t % 128 and head dims
// 16 j + 8 (t / 128) .. +8, and issues all of its loads at once (the merge
// is latency-bound: a few MB over a few thousand threads).
template <typename Fmt>
__global__ void __launch_bounds__(256)
attn_merge_kernel(const float* __restrict__ part, uint16_t* __restrict__ out,
                  SeqPack sp, int n_heads, int n_full, int n_ragged,
                  float scale_log2, int s_full, int s_rag) {
  const int nfs = s_full > 1 ? n_heads * n_full : 0;
  const int b = blockIdx.x >> 3;
  int h, s, qt, S, slot0;
  if (b < nfs) {
    S = s_full;
    slot0 = b * s_full;
    h = b / n_full;
    locate_full(sp, b % n_full, QT, s, qt);
  } else {
    const int tl = b - nfs;
    const int nr = max(n_ragged, 1);
    S = s_rag;
    slot0 = (s_full > 1 ? n_heads * n_full * s_full : 0) + tl * s_rag;
    h = tl / nr;
    locate_ragged(sp, tl % nr, QT, s, qt);
  }
  const int row0 = sp.row0[s];
  const int N = sp.row0[s + 1] - row0;
  const int qr = threadIdx.x & (QT - 1);
  const int d0 = ((blockIdx.x & 7) * 2 + (threadIdx.x >> 7)) * 8;
  const int q = qt * QT + qr;
  if (q >= N) return;
  const float* base = part + (size_t)slot0 * ATT_SLOT_FLOATS;
  float mv[ATT_MAX_SPLIT], lv[ATT_MAX_SPLIT], ov[ATT_MAX_SPLIT][8];
#pragma unroll
  for (int p = 0; p < ATT_MAX_SPLIT; ++p) {
    if (p < S) {
      const float* ps = base + (size_t)p * ATT_SLOT_FLOATS;
      mv[p] = ps[HD * QT + qr];
      lv[p] = ps[HD * QT + QT + qr];
#pragma unroll
      for (int i = 0; i < 8; ++i) ov[p][i] = ps[(d0 + i) * QT + qr];
    }
  }
  float m = -INFINITY;
#pragma unroll
  for (int p = 0; p < ATT_MAX_SPLIT; ++p)
    if (p < S) m = fmaxf(m, mv[p]);
  float l = 0.f, acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int p = 0; p < ATT_MAX_SPLIT; ++p) {
    if (p < S) {
      const float w = mv[p] == -INFINITY ? 0.f : exp2f((mv[p] - m) * scale_log2);
      l += lv[p] * w;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] += ov[p][i] * w;
    }
  }
  const float inv = 1.0f / l;
  u32x4 v;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    v[i] = (uint32_t)Fmt::store(acc[2 * i] * inv) |
           ((uint32_t)Fmt::store(acc[2 * i + 1] * inv) << 16);
  *reinterpret_cast<u32x4*>(out + (size_t)(row0 + q) * (n_heads * HD) +
                            (size_t)h * HD + d0) = v;
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

// 0: automatic; 1: never split; 2..ATT_MAX_SPLIT: split every query tile
// that many ways (davet_set_attention_split)
static std::atomic<int> g_attn_split_mode{0};

size_t attention_part_bytes(int64_t tokens, int64_t seqs, int n_heads) {
  const int64_t tiles = (tokens + QT - 1) / QT + seqs;
  const int64_t slots =
      std::min<int64_t>(ATT_MAX_SLOTS, tiles * n_heads * ATT_MAX_SPLIT);
  return (size_t)slots * ATT_SLOT_FLOATS * sizeof(float);
}

// Key-range split factors (full tiles, ragged tiles) for a launch; depends
// on the sequence layout only.  Automatic: a query tile's workgroup sweeps
// every key, so when the ragged last tiles do not fit beside the last round
// of full tiles they form a second round as long as a whole sweep; their
// keys are then split (each piece at least four key tiles, 256 keys).
// Short sequences are not split: there the per-workgroup latencies (query
// load, first key tile, partial round trip) outweigh the idle CUs.
static void plan_split(const SeqPack& sp, int n_heads, int n_full,
                       int n_ragged, int slots, int& s_full, int& s_rag) {
  s_full = s_rag = 1;
  const int mode = g_attn_split_mode.load();
  const int full_wg = n_heads * n_full, rag_wg = n_heads * n_ragged;
  const int wg = full_wg + rag_wg;
  if (wg == 0 || mode == 1) return;
  if (mode >= 2) {
    const int S = std::min(mode, ATT_MAX_SLOTS / wg);
    if (S > 1) s_full = s_rag = S;
    return;
  }
  int kt_rag_min = 1 << 30;
  for (int i = 0; i < sp.n_seqs; ++i) {
    const int n = sp.row0[i + 1] - sp.row0[i];
    if (n % QT) kt_rag_min = std::min(kt_rag_min, (n + KT - 1) / KT);
  }
  if (rag_wg > 0 && wg > slots / 2 && rag_wg <= slots / 4 &&
      rag_wg > (slots - full_wg % slots) % slots) {
    int S = std::min({ATT_MAX_SPLIT, slots / rag_wg, kt_rag_min / 4});
    S = std::min(S, ATT_MAX_SLOTS / rag_wg);
    if (S > 1) s_rag = S;
  }
}

int launch_attention16(int dtype, const uint16_t* qkv, uint16_t* o,
                       const SeqPack& sp, int n_heads, int head_dim,
                       float* part, size_t part_bytes, hipStream_t s) {
  if (head_dim != HD)
    return set_error(DAVET_ESHAPE, "attention16: head_dim must be 128");
  int n_full = 0, n_ragged = 0;
  for (int i = 0; i < sp.n_seqs; ++i) {
    const int n = sp.row0[i + 1] - sp.row0[i];
    n_full += n / QT;
    n_ragged += n % QT != 0;
  }
  const int tiles = n_full + n_ragged;
  if (tiles == 0) return DAVET_OK;
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)head_dim);
  // Workgroup slots of the one-key-group kernel: three per CU with fp16
  // (single K/V buffer), two with bf16.
  const int slots = (dtype == DAVET_F16 ? 3 : 2) * 256;
  int s_full, s_rag;
  plan_split(sp, n_heads, n_full, n_ragged, slots, s_full, s_rag);
  const int split_slots = (s_full > 1 ? n_heads * n_full * s_full : 0) +
                          (s_rag > 1 ? n_heads * n_ragged * s_rag : 0);
  if (split_slots > 0 &&
      (!part || (size_t)split_slots * ATT_SLOT_FLOATS * sizeof(float) > part_bytes))
    s_full = s_rag = 1;                  // no room: the unsplit launch
  const bool pieces = s_full > 1 || s_rag > 1;
  const dim3 grid(n_heads * (n_full * s_full + n_ragged * s_rag));
  // Few workgroups and no split (short sequences with few key tiles): two
  // key groups per workgroup so each SIMD still holds two wavefronts.
  // Otherwise one key group each, three workgroups per CU (measured on
  // MI355X against two groups: 3805 tokens 477 -> 443 us, 18020 tokens 8.45
  // -> 7.61 ms; 889 tokens 36 vs 41 us the other way; one buffer at three
  // workgroups per CU against two at two: 3805 tokens 325 -> 313 us, 18020
  // 5.69 -> 5.42 ms).
  const bool two_groups = !pieces && tiles * n_heads < 512;
  {
    ProfScope ps(KC_ATTN, s);
#define ATTN(F)                                                                \
  if (two_groups)                                                              \
    hipLaunchKernelGGL((attn16_kernel<F, 2>), grid, dim3(512), 0, s, qkv, o,   \
                       sp, n_heads, n_full, n_ragged, scale_log2, s_full,      \
                       s_rag, part);                                           \
  else                                                                         \
    hipLaunchKernelGGL((attn16_kernel<F, 1>), grid, dim3(256), 0, s, qkv, o,   \
                       sp, n_heads, n_full, n_ragged, scale_log2, s_full,      \
                       s_rag, part)
    if (dtype == DAVET_F16) { ATTN(F16); } else { ATTN(BF16); }
#undef ATTN
    DAVET_HIP(hipGetLastError());
  }
  if (pieces) {
    ProfScope ps(KC_ATTN, s);
    const int mgrid = 8 * ((s_full > 1 ? n_heads * n_full : 0) +
                           (s_rag > 1 ? n_heads * n_ragged : 0));
    if (dtype == DAVET_F16)
      hipLaunchKernelGGL(attn_merge_kernel<F16>, dim3(mgrid), dim3(256), 0, s,
                         part, o, sp, n_heads, n_full, n_ragged, scale_log2,
                         s_full, s_rag);
    else
      hipLaunchKernelGGL(attn_merge_kernel<BF16>, dim3(mgrid), dim3(256), 0, s,
                         part, o, sp, n_heads, n_full, n_ragged, scale_log2,
                         s_full, s_rag);
    DAVET_HIP(hipGetLastError());
  }
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

extern "C" int davet_set_attention_split(int32_t mode) {
  using namespace davet;
  DAVET_CHECK_ARG(mode >= 0 && mode <= ATT_MAX_SPLIT, DAVET_EINVAL,
                  "davet_set_attention_split: mode must be in [0, 8]");
  g_attn_split_mode.store(mode);
  return DAVET_OK;
}
