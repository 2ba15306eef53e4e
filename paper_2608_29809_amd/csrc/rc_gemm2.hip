// bf16 matrix-core GEMM, second form: Y[M][N] = A[M][K] . W[N][K]^T over a
// ragged row count M with the epilogues of the step (see rc_internal.h).
//
// * Operands move global -> LDS with global_load_lds_dwordx4 (no VGPR
//   staging); every 128-byte K-row of a tile is stored with its eight
//   16-byte chunks XOR-swizzled by swz(row) = (row >> 1) & 7.  A 16-byte
//   fragment read (lane l reads row l%32, chunk 2kk + l/32) is served 16
//   lanes per pass over 64 four-byte banks: rows r..r+15 cover the two
//   128-byte bank halves by row parity and, within a parity, eight distinct
//   chunks, so no two lanes of a pass share a bank (an (row & 7) swizzle
//   gives rows r and r+8 the same banks: two-way conflicts).
// * STAGES-deep ring of LDS buffers, one barrier per 64-wide K step; loads
//   for step k+STAGES-1 are issued right after the barrier of step k.
// * A K group is 4 or 8 waves in a WGM x WGN grid, each wave a
//   (BM/WGM)x(BN/WGN) block of 32x32x16 MFMAs.
// * Split-K over grid.z: each split writes an fp32 partial tile and a
//   separate kernel sums the splits in a fixed order and applies the
//   epilogue, so results do not depend on scheduling.
// * Tiles are renumbered so that consecutive logical tiles (all row tiles of
//   one column panel of W) land on the same XCD (workgroups are dealt to the
//   eight XCDs round-robin) and share that XCD's L2.
#include "rc_common.h"
#include "rc_launch.h"
#include "rc_internal.h"

#include <cmath>

namespace rc {

constexpr int G2_BK = 64;  // bf16 elements per K step (128 bytes per row)

// 16-byte chunk swizzle of a tile row in LDS (see the file comment).
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier without the memory fence of __syncthreads(): the fence
// would make the compiler drain every in-flight global->LDS load before the
// barrier.  Each thread waits for its own loads of the stage being consumed
// (wait_vmcnt) before arriving; LDS reads of the previous stage have been
// consumed by MFMAs, so they are complete.  The clobber keeps the compiler
// from moving memory accesses across.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Store one output element through the epilogue.
template <int EPI>
__device__ __forceinline__ void epi_store(const GemmArgs &g, int m, int n, float v, float gate, int part, int hh,
                                          int dd) {
  if (EPI == EPI_STORE) {
    ((bf16 *)g.out)[(size_t)m * g.ldo + n] = (bf16)v;
  } else if (EPI == EPI_GELU || EPI == EPI_GELU_FOLD) {
    ((bf16 *)g.out)[(size_t)m * g.ldo + n] = (bf16)gelu_tanh(v);
  } else if (EPI == EPI_RESID) {
    float *xp = g.X + (size_t)m * g.ldx + n;
    const float x = *xp + gate * v;
    *xp = x;
    if (g.xt) ((bf16 *)g.xt)[(size_t)m * g.ldx + n] = (bf16)x;
    if (g.hrows) ((bf16 *)g.hrows)[(size_t)m * g.N + n] = (bf16)x;
    if (g.hslot) {
      const int pk = g.rows[m];
      ((bf16 *)g.hslot)[row_chain(pk) * g.chain_stride + (size_t)row_token(pk) * g.hidden + n] = (bf16)x;
    }
  } else if (EPI == EPI_QKV) {
    if (part == 0) {
      ((bf16 *)g.out)[(size_t)m * g.ldo + n] = (bf16)v;
    } else {
      const int pk = g.rows[m];
      const size_t cb = (size_t)row_chain(pk) * g.chain_stride;
      const int tok = row_token(pk);
      ((bf16 *)(part == 1 ? g.kslot : g.vslot))[cb + ((size_t)hh * g.tokens + tok) * kHeadDim + dd] = (bf16)v;
    }
  } else if (EPI == EPI_TEXTKV) {
    const int b = m / g.text_len, t = m - b * g.text_len;
    bf16 *base = (bf16 *)g.tkv + (size_t)b * g.tkv_chain_stride;
    const size_t half = (size_t)(g.hidden / kHeadDim) * g.text_pad * kHeadDim;
    if (part == 0)
      base[((size_t)hh * g.text_pad + t) * kHeadDim + dd] = (bf16)v;
    else
      base[half + ((size_t)hh * kHeadDim + dd) * g.text_pad + t] = (bf16)v;
  }
}

__device__ __forceinline__ void st4(bf16 *p, const float *v) {
  bf16x4 o;
  o[0] = (bf16)v[0]; o[1] = (bf16)v[1]; o[2] = (bf16)v[2]; o[3] = (bf16)v[3];
  *(bf16x4 *)p = o;
}

// X[m][n..n+3] += gate * v, with the E copies of the updated values; the
// updated values are returned in v.
__device__ __forceinline__ void resid4(const GemmArgs &g, int m, int n, float *v) {
  f32x4 gt = f32x4{1.0f, 1.0f, 1.0f, 1.0f};
  if (g.gate) {
    gt = *(const f32x4 *)(g.gate + n);
    if (g.gate2) {
      const f32x4 g2 = *(const f32x4 *)(g.gate2 + n);
#pragma unroll
      for (int q = 0; q < 4; ++q) gt[q] += g2[q];
    }
  }
  f32x4 *xp = (f32x4 *)(g.X + (size_t)m * g.ldx + n);
  f32x4 x = *xp;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    x[q] += gt[q] * v[q];
    v[q] = x[q];
  }
  *xp = x;
  if (g.xt) st4((bf16 *)g.xt + (size_t)m * g.ldx + n, v);
  if (g.hrows) st4((bf16 *)g.hrows + (size_t)m * g.N + n, v);
  if (g.hslot) {
    const int pk = g.rows[m];
    st4((bf16 *)g.hslot + row_chain(pk) * g.chain_stride + (size_t)row_token(pk) * g.hidden + n, v);
  }
}

// Four consecutive output columns n..n+3 of row m (n % 4 == 0; never the
// transposed text values, whose columns are handled one by one).
template <int EPI>
__device__ __forceinline__ void epi4(const GemmArgs &g, int m, int n, float *v, int part) {
  if (EPI == EPI_STORE) {
    st4((bf16 *)g.out + (size_t)m * g.ldo + n, v);
  } else if (EPI == EPI_GELU || EPI == EPI_GELU_FOLD) {
    float w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) w[q] = gelu_tanh(v[q]);
    st4((bf16 *)g.out + (size_t)m * g.ldo + n, w);
  } else if (EPI == EPI_RESID) {
    resid4(g, m, n, v);
  } else if (EPI == EPI_QKV) {
    if (part == 0) {
      st4((bf16 *)g.out + (size_t)m * g.ldo + n, v);
    } else {
      const int pk = g.rows[m];
      const int c = n - part * g.hidden, hh = c / kHeadDim, dd = c - hh * kHeadDim;
      st4((bf16 *)(part == 1 ? g.kslot : g.vslot) + (size_t)row_chain(pk) * g.chain_stride +
              ((size_t)hh * g.tokens + row_token(pk)) * kHeadDim + dd, v);
    }
  } else if (EPI == EPI_TEXTKV) {
    const int b = m / g.text_len, t = m - b * g.text_len;
    const int hh = n / kHeadDim, dd = n - hh * kHeadDim;
    st4((bf16 *)g.tkv + (size_t)b * g.tkv_chain_stride + ((size_t)hh * g.text_pad + t) * kHeadDim + dd, v);
  }
}

template <int EPI>
__device__ __forceinline__ void col_info(const GemmArgs &g, int n, float &bn, float &gate, int &part, int &hh,
                                         int &dd) {
  bn = g.bias ? g.bias[n] : 0.0f;
  gate = 1.0f;
  if (EPI == EPI_RESID && g.gate) gate = g.gate[n] + (g.gate2 ? g.gate2[n] : 0.0f);
  part = 0;
  hh = 0;
  dd = 0;
  if (EPI == EPI_QKV || EPI == EPI_TEXTKV) {
    part = n / g.hidden;
    const int c = n - part * g.hidden;
    hh = c / kHeadDim;
    dd = c - hh * kHeadDim;
  }
}

constexpr int pow2_ceil(int v) { return v <= 1 ? 1 : 2 * pow2_ceil((v + 1) / 2); }

// Sum over W = 2, 4, 8 or 16 consecutive lanes (aligned groups), in DPP;
// every lane of a group ends with the same value.
template <int W> __device__ __forceinline__ float lane_group_sum(float v) {
  static_assert(W == 2 || W == 4 || W == 8 || W == 16, "2 to 16 lanes");
  if (W == 16) return row16_sum(v);
  v += dpp_mov<0xB1>(v);                  // quad_perm [1,0,3,2]
  if (W >= 4) v += dpp_mov<0x4E>(v);      // quad_perm [2,3,0,1]
  if (W >= 8) v += dpp_mov<0x141>(v);     // row_half_mirror
  return v;
}

// Sum over W = 16 or 32 consecutive lanes (aligned groups): DPP within each
// row of 16, then a swizzle exchanging the two rows of a 32-lane half.
template <int W> __device__ __forceinline__ float group_sum(float v) {
  static_assert(W == 16 || W == 32, "16- or 32-lane groups");
  v = row16_sum(v);
  if (W == 32) v += __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x401F));  // lane ^ 16
  return v;
}

template <int BM, int BN, int STAGES, int KG, int WGM, int WGN, int EPI, bool SPLIT>
__global__ __launch_bounds__(64 * WGM * WGN * KG) void gemm2_kernel(GemmArgs g, float *partial, int k_per_split) {
  constexpr int NW = WGM * WGN;                       // waves per K group
  constexpr int WM = BM / WGM, WN = BN / WGN, FM = WM / 32, FN = WN / 32;
  constexpr int A_LD = BM * 8 / (64 * NW);            // direct loads per thread per stage (16 bytes each)
  constexpr int B_LD = BN * 8 / (64 * NW);
  static_assert(A_LD * 64 * NW == BM * 8 && B_LD * 64 * NW == BN * 8, "tile rows must split over the waves");
  constexpr int LPS = A_LD + B_LD;
  constexpr int STAGE_BYTES = (BM + BN) * 128;
  constexpr int GROUP_BYTES = STAGES * STAGE_BYTES;  // one K group's ring
  constexpr int CLD = BN + 4;                         // row of an fp32 output tile in LDS
  // the fp32 output tile is staged through the rings in PASSES row bands
  constexpr int PASSES = (BM * CLD * 4 <= GROUP_BYTES) ? 1 : 2;
  constexpr int HB = BM / PASSES;
  static_assert(HB * CLD * 4 <= GROUP_BYTES && HB % WM == 0, "an output band must fit a group's ring");
  // folded LayerNorm (EPI_GELU_FOLD): a tile's last four A rows are the
  // fold's (1 + scale) and shift rows, each as a bf16 pair (high part, then
  // the rounding remainder), so it covers TROWS rows of the output
  constexpr bool FOLD = EPI == EPI_GELU_FOLD;
  constexpr int TROWS = FOLD ? BM - 4 : BM;
  // after the rings: [BM] (mean, r) per row, [KG][2][BN] u and v partials;
  // the producer's statistics of the tile's rows [TROWS][fold_nt] get a
  // region of their own where that keeps the workgroups per CU (merged after
  // the K loop, their loads land during it), else they pass through the
  // first ring's last stage, which the prologue leaves empty (merged before
  // the K loop)
  constexpr int FOLD_OFF = KG * GROUP_BYTES + 256;
  constexpr int LDS_BASE = FOLD_OFF + (FOLD ? BM * 8 + KG * 2 * BN * 4 : 0);
  constexpr int ST_BYTES = TROWS * kFoldMaxTiles * 8;
  constexpr bool ST_OWN = FOLD && kLdsBytes / (LDS_BASE + ST_BYTES) == kLdsBytes / LDS_BASE;
  constexpr int FOLD_ST_OFF = ST_OWN ? LDS_BASE : (STAGES - 1) * STAGE_BYTES;
  static_assert(!FOLD || ST_OWN || ST_BYTES <= STAGE_BYTES, "the statistics must fit a stage");
  __shared__ __attribute__((aligned(1024))) char lds[LDS_BASE + (ST_OWN ? ST_BYTES : 0)];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kgrp = wave / NW, w4 = wave % NW;
  const int wm = w4 / WGN, wn = w4 % WGN;

  // XCD-aware tile order: logical tile L walks the row tiles of one column
  // panel before moving to the next panel; physical id p runs on XCD p % 8.
  // Logical order per split: groups of up to 16 row tiles, and within a
  // group row tiles fastest, then column panels.  Consecutive logical tiles
  // run on one XCD, so the ~64 tiles in flight there share <= 16 row panels
  // of A and a few column panels of W in that XCD's L2.
  const int tiles_m = gridDim.y, tiles_n = gridDim.x, TT = tiles_m * tiles_n, T = TT * gridDim.z;
  const int p = blockIdx.x + tiles_n * (blockIdx.y + tiles_m * blockIdx.z);
  const int L = xcd_logical_id(p, T);
  const int kz = L / TT, r = L - kz * TT;
  constexpr int GM = 16;
  const int grp = r / (GM * tiles_n), gm = min(GM, tiles_m - grp * GM), idx = r - grp * GM * tiles_n;
  const int tm = grp * GM + idx % gm, tn = idx / gm;
  const int m0 = tm * TROWS, n0 = tn * BN;
  // K group kgrp covers its own contiguous share of this split's K range
  if (wave == 0) warm_lines(g.warm, g.warm_lines, p, T, lds + KG * GROUP_BYTES);
  const int kps_g = k_per_split / KG;
  const int kbeg = kz * k_per_split + kgrp * kps_g;
  const int nk = kps_g / G2_BK;
  char *ring = lds + kgrp * GROUP_BYTES;

  const bf16 *A = (const bf16 *)g.A;
  const bf16 *W = (const bf16 *)g.W;

  auto issue = [&](int stage, int k0) {
    char *sa = ring + stage * STAGE_BYTES;
    char *sb = sa + BM * 128;
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int ch = (i * NW + w4) * 64 + lane;
      const int r = ch >> 3, c = (ch & 7) ^ swz(r);
      const int gr = min(m0 + r, g.M - 1);
      const bf16 *src = A + (size_t)gr * g.lda + k0 + c * 8;
      if (FOLD && r >= TROWS) src = (const bf16 *)g.fold_extra + (size_t)(r - TROWS) * g.K + k0 + c * 8;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)src,
                                       (__attribute__((address_space(3))) void *)(sa + (i * NW + w4) * 1024), 16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int ch = (i * NW + w4) * 64 + lane;
      const int r = ch >> 3, c = (ch & 7) ^ swz(r);
      const bf16 *src = W + (size_t)(n0 + r) * g.K + k0 + c * 8;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)src,
                                       (__attribute__((address_space(3))) void *)(sb + (i * NW + w4) * 1024), 16, 0, 0);
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  // the fold's per-row partial statistics of the tile's rows (contiguous:
  // TROWS x fold_nt pairs) go to LDS by direct loads issued before the first
  // stages; each wave loads and merges the statistics of its own FRW rows,
  // so it waits for its own loads only (they are older than its stage
  // loads) and needs no barrier
  constexpr int NTH = 64 * NW * KG, NWAVES = NW * KG;
  constexpr int FRW = pow2_ceil((TROWS + NWAVES - 1) / NWAVES);  // rows per wave
  constexpr int FLR = 64 / FRW;                                  // lanes per row
  static_assert(!FOLD || (FLR >= 2 && FLR <= 16), "2 to 16 lanes per row");
  const float2 *sts = (const float2 *)(lds + FOLD_ST_OFF);
  float2 *fold_rs = (float2 *)(lds + FOLD_OFF);        // [BM] (mean, r)
  float *fold_uv = (float *)(lds + FOLD_OFF + BM * 8);  // [KG][2][BN]
  const int frow0 = wave * FRW;  // the wave's first row (FRW and m0 even: 16-byte aligned)
  if (FOLD && frow0 < TROWS) {
    const int nt = g.fold_nt, nch = min(FRW, TROWS - frow0) * nt / 2;
    const int first = (m0 + frow0) * nt / 2, last = (g.M * nt + 1) / 2 - 1;
    for (int c0 = 0; c0 < nch; c0 += 64) {
      if (c0 + lane < nch) {
        const char *src = (const char *)g.fold_stats + (size_t)min(first + c0 + lane, last) * 16;
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)src,
                                         (__attribute__((address_space(3))) void *)(lds + FOLD_ST_OFF + (frow0 * nt / 2 + c0) * 16),
                                         16, 0, 0);
      }
    }
  }

#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) issue(s, kbeg + s * G2_BK);
  // FLR lanes per row merge the row's equal-size partials (strided over the
  // lanes, then summed across them: a fixed order)
  auto fold_merge = [&]() {
    const int nt = g.fold_nt, row = frow0 + lane / FLR, j0 = lane % FLR;
    const float2 *st = sts + min(row, TROWS - 1) * nt;
    constexpr int PER = (kFoldMaxTiles + FLR - 1) / FLR;
    float2 p[PER];  // (unpredicated reads: no branch between them)
#pragma unroll
    for (int i = 0; i < PER; ++i) p[i] = st[min(j0 + i * FLR, nt - 1)];
    float sm = 0.0f;
#pragma unroll
    for (int i = 0; i < PER; ++i) sm += j0 + i * FLR < nt ? p[i].x : 0.0f;
    const float mu = lane_group_sum<FLR>(sm) / (float)nt;
    const float cnt = (float)(g.K / nt);
    float m2 = 0.0f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const float d = p[i].x - mu;
      m2 += j0 + i * FLR < nt ? p[i].y + cnt * d * d : 0.0f;
    }
    m2 = lane_group_sum<FLR>(m2);
    if (j0 == 0 && row < TROWS) fold_rs[row] = make_float2(mu, rsqrtf(m2 / (float)g.K + g.fold_eps));
  };
  if (FOLD && !ST_OWN && frow0 < TROWS) {
    // the wave's own statistics are older than its stage loads
    if (nk >= STAGES - 1) wait_vmcnt<(STAGES - 1) * LPS>();
    else wait_vmcnt<0>();
    fold_merge();
  }

  const int g32 = lane >> 5, r32 = lane & 31;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + STAGES - 2 < nk) wait_vmcnt<(STAGES - 2) * LPS>();
    else wait_vmcnt<0>();
    lds_barrier();
    if (kt + STAGES - 1 < nk) issue((kt + STAGES - 1) % STAGES, kbeg + (kt + STAGES - 1) * G2_BK);
    const char *sa = ring + (kt % STAGES) * STAGE_BYTES;
    const char *sb = sa + BM * 128;
    // fragments of sub-step kk+1 are read while the MFMAs of kk run
    bf16x8 a[2][FM], b[2][FN];
    auto frags = [&](int buf, int kk) {
      const int c = kk * 2 + g32;
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int r = wm * WM + i * 32 + r32;
        a[buf][i] = *(const bf16x8 *)(sa + r * 128 + ((c ^ swz(r)) << 4));
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int r = wn * WN + j * 32 + r32;
        b[buf][j] = *(const bf16x8 *)(sb + r * 128 + ((c ^ swz(r)) << 4));
      }
    };
    frags(0, 0);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      if (kk < 3) frags((kk + 1) & 1, kk + 1);
      // keep the reads of kk+1 ahead of the MFMAs of kk (the scheduler would
      // otherwise sink them and reuse one register set)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk & 1][i], b[kk & 1][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // Each K group's tile goes to LDS (the rings are free: every load has been
  // consumed), one band of HB rows at a time; the groups' tiles are summed in
  // group order while the band is written back with 16-byte row-contiguous
  // accesses.  Tiles of transposed text values are walked column-major
  // instead so that consecutive threads write consecutive tokens.
  if (FOLD) {
    if (ST_OWN && frow0 < TROWS) {  // (every load has completed: the loop's last wait)
      wait_vmcnt<0>();
      fold_merge();
    }
    // rows BM-4 .. BM-1 (u as two parts, then v): local rows 28 to 31 of
    // the last 32-row block, accumulators 12 to 15 of the upper half-wave
    if (wm == WGM - 1 && g32 == 1) {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = wn * WN + j * 32 + r32;
        fold_uv[(kgrp * 2) * BN + col] = acc[FM - 1][j][12] + acc[FM - 1][j][13];
        fold_uv[(kgrp * 2 + 1) * BN + col] = acc[FM - 1][j][14] + acc[FM - 1][j][15];
      }
    }
  }
  float *ct = (float *)ring;
  auto tile_at = [&](int row, int col) {
    float v = 0.0f;
#pragma unroll
    for (int q = 0; q < KG; ++q) v += ((const float *)(lds + q * GROUP_BYTES))[row * CLD + col];
    return v;
  };
  constexpr int NT = NTH;
  const int tile_part = (EPI == EPI_QKV || EPI == EPI_TEXTKV) ? n0 / g.hidden : 0;
  const bool transposed = EPI == EPI_TEXTKV && tile_part == 1;
#pragma unroll
  for (int pass = 0; pass < PASSES; ++pass) {
    const int rb = pass * HB;  // first tile row of the band
    __syncthreads();
    if (wm * WM >= rb && wm * WM < rb + HB) {
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            ct[(wm * WM - rb + i * 32 + (e >> 2) * 8 + g32 * 4 + (e & 3)) * CLD + wn * WN + j * 32 + r32] =
                acc[i][j][e];
    }
    __syncthreads();
    if (SPLIT) {
      float *P = partial + (size_t)kz * g.M * g.N;
      for (int idx = tid; idx < HB * BN / 4; idx += NT) {
        const int row = idx / (BN / 4), c4 = (idx % (BN / 4)) * 4;
        const int m = m0 + rb + row;
        if (m >= g.M) continue;
        f32x4 v;
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = tile_at(row, c4 + q);
        *(f32x4 *)(P + (size_t)m * g.N + n0 + c4) = v;
      }
    } else if (!transposed) {
      // a thread keeps one group of 4 columns over the band's rows: column
      // data is loaded once, and every row-dependent load (residual, packed
      // row id) is issued before the first store so their latencies overlap
      static_assert(NT % (BN / 4) == 0, "a thread keeps its columns over the band");
      constexpr int RPI = NT / (BN / 4), IT = (HB + RPI - 1) / RPI;
      const int c4 = (tid % (BN / 4)) * 4, row0 = tid / (BN / 4);
      const int n = n0 + c4;
      const f32x4 bb = g.bias ? *(const f32x4 *)(g.bias + n) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      constexpr bool NEED_X = EPI == EPI_RESID;
      const bool need_rows = (EPI == EPI_RESID && g.hslot) || (EPI == EPI_QKV && tile_part > 0);
      // column loads land in registers with their defaults and are combined
      // only after the row loads below are issued (a use inside a branch
      // would make the row loads wait for them)
      f32x4 ga = f32x4{1.0f, 1.0f, 1.0f, 1.0f}, gb = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      if (EPI == EPI_RESID && g.gate) ga = *(const f32x4 *)(g.gate + n);
      if (EPI == EPI_RESID && g.gate && g.gate2) gb = *(const f32x4 *)(g.gate2 + n);
      // fold consumer: u and v of the tile's columns, summed over the K groups
      f32x4 fu = f32x4{0.0f, 0.0f, 0.0f, 0.0f}, fw = fu;
      if (FOLD) {
#pragma unroll
        for (int k = 0; k < KG; ++k) {
          fu += *(const f32x4 *)(fold_uv + (k * 2) * BN + c4);
          fw += *(const f32x4 *)(fold_uv + (k * 2 + 1) * BN + c4);
        }
      }
      // fold producer: the next LayerNorm's (1 + scale), and the consumer's
      // four extra rows (1 + scale and shift, each split into a bf16 high
      // part and its remainder so that u and v carry ~16 bits: a rounding of
      // these per-column factors would be the same for every row)
      // (unconditional loads, from X's first row without the fold: a branch
      // here would take the add of 1 into it, and the wait with it)
      const bool fold_out = EPI == EPI_RESID && g.fold_stats;
      const bool fold_rows = fold_out && tm == 0 && row0 == 0;  // writes the consumer's extra rows
      f32x4 fa = f32x4{0.0f, 0.0f, 0.0f, 0.0f}, fb = fa, fc = fa, fd = fa;
      if (EPI == EPI_RESID) {
        fa = *(const f32x4 *)((fold_out ? g.fold_scale[0] : g.X) + n);
        fb = *(const f32x4 *)((fold_out ? g.fold_scale[1] : g.X) + n);
        fc = *(const f32x4 *)((fold_rows ? g.fold_shift[0] : g.X) + n);
        fd = *(const f32x4 *)((fold_rows ? g.fold_shift[1] : g.X) + n);
      }
      f32x4 xo[NEED_X ? IT : 1];
      int pk[IT];
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int m = min(m0 + rb + min(row0 + it * RPI, HB - 1), g.M - 1);
        if (NEED_X) xo[it] = *(const f32x4 *)(g.X + (size_t)m * g.ldx + n);
        pk[it] = need_rows ? g.rows[m] : 0;
      }
      const f32x4 gt = ga + gb, fsc = 1.0f + fa + fb;
#pragma unroll
      for (int it = 0; it < IT; ++it) {
        const int row = row0 + it * RPI;
        const int m = m0 + rb + row;
        if ((IT * RPI != HB && row >= HB) || m >= g.M || (FOLD && rb + row >= TROWS)) continue;
        float v[4];
        if (FOLD) {  // h W^T + b = r (x~ W^T - mean u) + v + b
          const float2 st = fold_rs[rb + row];
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = st.y * (tile_at(row, c4 + q) - st.x * fu[q]) + fw[q] + bb[q];
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = tile_at(row, c4 + q) + bb[q];
        }
        if (EPI == EPI_RESID) {
          f32x4 x;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            x[q] = xo[NEED_X ? it : 0][q] + gt[q] * v[q];
            v[q] = x[q];
          }
          *(f32x4 *)(g.X + (size_t)m * g.ldx + n) = x;
          if (fold_out) {
            // the next LayerNorm's statistics of this row over the tile's
            // BN columns (every lane of the row's group takes part), and x~
            const float mean = group_sum<BN / 4>((v[0] + v[1]) + (v[2] + v[3])) / BN;
            float d2 = 0.0f;
#pragma unroll
            for (int q = 0; q < 4; ++q) d2 += (v[q] - mean) * (v[q] - mean);
            d2 = group_sum<BN / 4>(d2);
            if (c4 == 0) g.fold_stats[(size_t)m * g.fold_nt + n0 / BN] = make_float2(mean, d2);
            const float xs[4] = {v[0] * fsc[0], v[1] * fsc[1], v[2] * fsc[2], v[3] * fsc[3]};
            st4((bf16 *)g.xt + (size_t)m * g.ldx + n, xs);
          } else if (g.xt) {
            st4((bf16 *)g.xt + (size_t)m * g.ldx + n, v);
          }
          if (g.hrows) st4((bf16 *)g.hrows + (size_t)m * g.N + n, v);
          if (g.hslot)
            st4((bf16 *)g.hslot + row_chain(pk[it]) * g.chain_stride + (size_t)row_token(pk[it]) * g.hidden + n, v);
        } else if (EPI == EPI_QKV && tile_part > 0) {
          const int c = n - tile_part * g.hidden, hh = c / kHeadDim, dd = c - hh * kHeadDim;
          st4((bf16 *)(tile_part == 1 ? g.kslot : g.vslot) + (size_t)row_chain(pk[it]) * g.chain_stride +
                  ((size_t)hh * g.tokens + row_token(pk[it])) * kHeadDim + dd, v);
        } else {
          epi4<EPI>(g, m, n, v, tile_part);
        }
      }
      // (after the rows: a branch between the loads above and their use
      // would make the residual loads wait for the scale loads)
      if (fold_rows && pass == 0) {
        const f32x4 fsh = fc + fd;
        float part[4][4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          part[0][q] = (float)(bf16)fsc[q];
          part[1][q] = fsc[q] - part[0][q];
          part[2][q] = (float)(bf16)fsh[q];
          part[3][q] = fsh[q] - part[2][q];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) st4((bf16 *)g.fold_extra + (size_t)e * g.N + n, part[e]);
      }
    } else {
      // a wave walks one column, lanes on consecutive rows: each store covers
      // consecutive text tokens of one transposed-V row
      static_assert(NT % HB == 0, "a pass must cover whole columns");
      for (int idx = tid; idx < HB * BN; idx += NT) {
        const int col = idx / HB, row = idx - col * HB;
        const int m = m0 + rb + row;
        if (m >= g.M) continue;
        const int n = n0 + col;
        const float bn = g.bias ? g.bias[n] : 0.0f;
        const int c = n - tile_part * g.hidden, hh = c / kHeadDim, dd = c - hh * kHeadDim;
        epi_store<EPI>(g, m, n, tile_at(row, col) + bn, 1.0f, tile_part, hh, dd);
      }
    }
  }
}

// Sum of the split partials in split order, then the epilogue.  One thread
// per output element; consecutive threads walk n.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs g, const float *partial, int splits) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)g.M * g.N) return;
  const int m = idx / g.N, n = idx - (long)m * g.N;
  float v = 0.0f;
  for (int s = 0; s < splits; ++s) v += partial[(size_t)s * g.M * g.N + idx];
  float bn, gate;
  int part, hh, dd;
  col_info<EPI>(g, n, bn, gate, part, hh, dd);
  epi_store<EPI>(g, m, n, v + bn, gate, part, hh, dd);
}

// Split reduction of a residual GEMM fused with the next block's LayerNorm:
// one 256-thread workgroup per row sums the splits in order, adds bias,
// applies gate and residual (with the E copies), then normalises the
// finished row and writes the modulated E row for the next GEMM.
template <int S>
__global__ __launch_bounds__(256) void splitk_finish_ln_kernel(GemmArgs g, const float *partial, LnNext ln) {
  __shared__ float red[4];
  const int m = blockIdx.x, t = threadIdx.x;
  constexpr int MAXV = 2;  // N <= 4 * 256 * MAXV
  const int N4 = g.N >> 2;
  const float *sh = ln.sst + (size_t)ln.shift_row * g.N, *sc = sh + g.N;
  const float *tsh = ln.t0 + (size_t)ln.shift_row * g.N, *tsc = tsh + g.N;
  // every load first (partials, bias, gate, residual, modulation), then the
  // stores: the compiler may not move a load above a store to X
  f32x4 p[MAXV], xo[MAXV], gt[MAXV], shift[MAXV], scale[MAXV];
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int n4 = t + 256 * i;
    p[i] = xo[i] = shift[i] = scale[i] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    gt[i] = f32x4{1.0f, 1.0f, 1.0f, 1.0f};
    if (n4 < N4) {
      const int n = 4 * n4;
      shift[i] = *(const f32x4 *)(sh + n) + *(const f32x4 *)(tsh + n);
      scale[i] = *(const f32x4 *)(sc + n) + *(const f32x4 *)(tsc + n);
#pragma unroll
      for (int sp = 0; sp < S; ++sp) p[i] += *(const f32x4 *)(partial + ((size_t)sp * g.M + m) * g.N + n);
      if (g.bias) p[i] += *(const f32x4 *)(g.bias + n);
      if (g.gate) {
        gt[i] = *(const f32x4 *)(g.gate + n);
        if (g.gate2) gt[i] += *(const f32x4 *)(g.gate2 + n);
      }
      xo[i] = *(const f32x4 *)(g.X + (size_t)m * g.ldx + n);
    }
  }
  float x[MAXV][4];
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int n4 = t + 256 * i;
#pragma unroll
    for (int q = 0; q < 4; ++q) x[i][q] = xo[i][q] + gt[i][q] * p[i][q];
    if (n4 < N4) {
      const int n = 4 * n4;
      *(f32x4 *)(g.X + (size_t)m * g.ldx + n) = f32x4{x[i][0], x[i][1], x[i][2], x[i][3]};
      if (g.xt) st4((bf16 *)g.xt + (size_t)m * g.ldx + n, x[i]);
      if (g.hrows) st4((bf16 *)g.hrows + (size_t)m * g.N + n, x[i]);
      if (g.hslot) {
        const int pk = g.rows[m];
        st4((bf16 *)g.hslot + row_chain(pk) * g.chain_stride + (size_t)row_token(pk) * g.hidden + n, x[i]);
      }
      sum += (x[i][0] + x[i][1]) + (x[i][2] + x[i][3]);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) x[i][q] = 0.0f;
    }
  }
  const float mean = block4_sum(sum, red) / g.N;
  float sq = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i)
    if (t + 256 * i < N4)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float d = x[i][q] - mean;
        sq += d * d;
      }
  const float rstd = rsqrtf(block4_sum(sq, red) / g.N + ln.eps);
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int n4 = t + 256 * i;
    if (n4 < N4) {
      float y[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) y[q] = (x[i][q] - mean) * rstd * (1.0f + scale[i][q]) + shift[i][q];
      st4((bf16 *)ln.out + (size_t)m * g.N + 4 * n4, y);
    }
  }
}

template <int BM, int BN, int STAGES, int KG, int WGM, int WGN, bool SPLIT>
static void launch_g2(const GemmArgs &a, int epi, int splits, float *partial, hipStream_t s) {
  const int trows = epi == EPI_GELU_FOLD ? BM - 4 : BM;
  dim3 grid(a.N / BN, (a.M + trows - 1) / trows, splits);
  const int kps = a.K / splits;
#define RC_G2(E)                                                                                       \
  rc_launch(gemm2_kernel<BM, BN, STAGES, KG, WGM, WGN, E, SPLIT>, grid, dim3(64 * WGM * WGN * KG), 0, s, \
                     a, partial, kps)
  switch (epi) {
    case EPI_STORE: RC_G2(EPI_STORE); break;
    case EPI_GELU: RC_G2(EPI_GELU); break;
    case EPI_GELU_FOLD:
      if constexpr (!SPLIT) RC_G2(EPI_GELU_FOLD);
      break;
    case EPI_RESID: RC_G2(EPI_RESID); break;
    case EPI_QKV: RC_G2(EPI_QKV); break;
    case EPI_TEXTKV: RC_G2(EPI_TEXTKV); break;
  }
#undef RC_G2
}

static void launch_reduce(const GemmArgs &a, int epi, int splits, const float *partial, hipStream_t s) {
  const long n = (long)a.M * a.N;
  dim3 grid((n + 255) / 256);
#define RC_RD(E) rc_launch(splitk_reduce_kernel<E>, grid, dim3(256), 0, s, a, partial, splits)
  switch (epi) {
    case EPI_STORE: RC_RD(EPI_STORE); break;
    case EPI_GELU: RC_RD(EPI_GELU); break;
    case EPI_RESID: RC_RD(EPI_RESID); break;
    case EPI_QKV: RC_RD(EPI_QKV); break;
    case EPI_TEXTKV: RC_RD(EPI_TEXTKV); break;
  }
#undef RC_RD
}

// Choice of tile, wave layout, K groups and split count for a shape, from
// sweeps on the step's shapes with the activations in cache and the weights
// cold (410 to 4096 rows; N in {1152, 3456, 4608}; K in {1152, 4608}).  The
// operand traffic into a CU (L2 -> LDS, ~64 bytes per clock) bounds small
// tiles, and a workgroup's time is set by its K steps: a grid that fits the
// 256 CUs in one wave of workgroups takes the largest tile that still fills
// them, with eight waves (32x32 or 32x64 / 64x32 per wave) where the tile
// allows it; grids of one to two waves of 64-row tiles keep 64x128 with two
// workgroups per CU.  Split-K over the grid pays only for K = 4608, in two
// halves up to ~2700 rows (the halves as 128-row tiles while they fit one
// wave of workgroups); three splits measured slower in the step at 4096 rows.
// Narrow outputs (N = 1152, K = 1152) at a few hundred to ~900 rows take
// 64x64 tiles with two K groups of 2x2 waves (216 workgroups at 723 rows:
// 9.1 against 10.9 us for 32x128 tiles, weights cold), and below ~450 rows
// 32x64 tiles with two K groups of two waves (8.3 against 10.6 us at 154
// rows).  The wide outputs below ~250 rows take the 64x64 two-group tiles
// too (QKV at 154 rows: 9.6 against 13.2 us), and the MLP-down at a few
// hundred rows four K quarters (12.4 against 18.8 us at 154 rows).  A
// four-deep ring gains ~3 % over three for the 64x64 tiles and for the
// 4x2-wave 128x128 QKV tiles (16.3 against 16.8 us), nothing for the
// 2x4-wave MLP-up tiles.  Two K groups of 2x2 waves beat one group of 2x4
// for 64x128 tiles at ~400 rows (13.3 against 13.6 us).
GemmPlan plan_gemm2(int M, int N, int K, size_t partial_cap_floats) {
  GemmPlan p{64, 128, 1, 1, 2, 2, 2};
  const int nk = K / G2_BK;
  const long tn = N / 128;
  const long t32 = (long)((M + 31) / 32) * tn, t64 = (long)((M + 63) / 64) * tn, t128 = (long)((M + 127) / 128) * tn;
  const long t64x64 = (long)((M + 63) / 64) * (N / 64), t32x64 = (long)((M + 31) / 32) * (N / 64);
  auto set = [&](int bm, int kg, int stages, int wgm, int wgn) {
    p.bm = bm; p.kg = kg; p.stages = stages; p.wgm = wgm; p.wgn = wgn;
  };
  if (K >= 2048) {
    const bool room2 = (size_t)2 * M * N <= partial_cap_floats, room4 = (size_t)4 * M * N <= partial_cap_floats;
    if (t32 * 4 <= 256 && nk % 8 == 0 && room4) {
      p.splits = 4;  // a few hundred rows: four K quarters keep ~180 workgroups busy
      set(32, 2, 3, 1, 4);
    } else if (t64 < 160 && nk % 4 == 0 && room2) {
      p.splits = 2;
      if (t32 * 2 <= 256) set(32, 2, 3, 1, 4);
      else set(64, 2, 3, 2, 2);
    } else if (t64 < 384 && nk % 2 == 0 && room2) {
      p.splits = 2;
      if (t128 * 2 <= 256) set(128, 1, 3, 2, 4);
      else set(64, 1, 2, 2, 2);
    }
    return p;
  }
  if (N >= 3072) {
    if (nk % 2 == 0 && N % 64 == 0 && t64x64 <= 256) {  // ~250 rows and fewer
      set(64, 2, 4, 2, 2);
      p.bn = 64;
    } else if (nk % 2 == 0 && t64 <= 256) set(64, 2, 3, 2, 2);
    else if (t64 <= 256) set(64, 1, 3, 2, 4);
    else if (t128 <= 256 && N % 512) set(128, 1, 4, 4, 2);
    else if (t128 <= 256) set(128, 1, 3, 2, 4);
    else set(128, 1, 2, 4, 2);  // eight waves: 8-10 % faster than four from 3072 to 16384 rows
    return p;
  }
  if (nk % 2 == 0 && N % 64 == 0 && t32x64 <= 256) {  // up to ~450 rows at N = 1152
    set(32, 2, 3, 1, 2);
    p.bn = 64;
  } else if (nk % 2 == 0 && M > 256 && N % 64 == 0 && t64x64 <= 256) {
    set(64, 2, 4, 2, 2);
    p.bn = 64;
  } else if (nk % 2 == 0 && t32 <= 256) set(32, 2, 3, 1, 4);
  else if (nk % 2 == 0 && t64 <= 256) set(64, 2, 3, 2, 2);
  else if (t64 <= 512) set(64, 1, 3, 2, 4);
  return p;
}

hipError_t launch_gemm2(const GemmArgs &a, int epi, const GemmPlan &pl, float *partial, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if ((pl.bn != 128 && pl.bn != 64) || a.N % pl.bn || a.K % (G2_BK * pl.splits * pl.kg)) return hipErrorInvalidValue;
  const bool split = pl.splits > 1;
  // the folded LayerNorm needs the whole K range in one launch and the
  // producer's per-tile statistics (equal column counts, at most kFoldMaxTiles)
  if (epi == EPI_GELU_FOLD &&
      (split || a.fold_nt <= 0 || a.fold_nt > kFoldMaxTiles || a.K % a.fold_nt || !a.fold_stats || !a.fold_extra))
    return hipErrorInvalidValue;
  // the fold's producer writes its statistics from the one-pass row epilogue
  if (epi == EPI_RESID && a.fold_stats && (split || a.fold_nt != a.N / pl.bn || !a.xt || !a.fold_extra))
    return hipErrorInvalidValue;
  // 4-wave K groups: 128 rows = 2x2 waves of 64x64, 64 rows = 2x2 of 32x64,
  // 32 rows = 1x4 of 32x32, 64x64 tiles = 2x2 of 32x32; 8-wave: 128 rows =
  // 4x2 of 32x64 or 2x4 of 64x32, 64 rows = 2x4 of 32x32
#define RC_G2(BMV, BNV, KGV, STG, WM_, WN_)                                                   \
  {                                                                                          \
    if (split) launch_g2<BMV, BNV, STG, KGV, WM_, WN_, true>(a, epi, pl.splits, partial, s); \
    else launch_g2<BMV, BNV, STG, KGV, WM_, WN_, false>(a, epi, 1, nullptr, s);              \
  }
  const long cfg = pl.bn * 10000000L + pl.bm * 10000 + pl.kg * 1000 + pl.stages * 100 + pl.wgm * 10 + pl.wgn;
  switch (cfg) {
    case 1280641222: RC_G2(64, 128, 1, 2, 2, 2) break;
    case 1280642322: RC_G2(64, 128, 2, 3, 2, 2) break;
    case 1280641324: RC_G2(64, 128, 1, 3, 2, 4) break;
    case 1280321314: RC_G2(32, 128, 1, 3, 1, 4) break;
    case 1280322314: RC_G2(32, 128, 2, 3, 1, 4) break;
    case 1280323214: RC_G2(32, 128, 3, 2, 1, 4) break;
    case 1281281222: RC_G2(128, 128, 1, 2, 2, 2) break;
    case 1281281242: RC_G2(128, 128, 1, 2, 4, 2) break;
    case 1281281342: RC_G2(128, 128, 1, 3, 4, 2) break;
    case 1281281324: RC_G2(128, 128, 1, 3, 2, 4) break;
    case 640642422: RC_G2(64, 64, 2, 4, 2, 2) break;
    case 640322312: RC_G2(32, 64, 2, 3, 1, 2) break;
    case 1281281442: RC_G2(128, 128, 1, 4, 4, 2) break;
    default: return hipErrorInvalidValue;
  }
#undef RC_G2
  return hipGetLastError();
}

hipError_t launch_gemm2_finish(const GemmArgs &a, int epi, const GemmPlan &pl, const float *partial, hipStream_t s,
                               const LnNext *ln, bool *ln_done) {
  if (ln_done) *ln_done = false;
  if (a.M <= 0 || pl.splits <= 1) return hipSuccess;
  if (ln && epi == EPI_RESID && a.N % 4 == 0 && a.N <= 4 * 256 * 2 && pl.splits <= 4) {
    const dim3 grid(a.M), block(256);
    const float *pp = partial;
    if (pl.splits == 2) rc_launch(splitk_finish_ln_kernel<2>, grid, block, 0, s, a, pp, *ln);
    else if (pl.splits == 3) rc_launch(splitk_finish_ln_kernel<3>, grid, block, 0, s, a, pp, *ln);
    else rc_launch(splitk_finish_ln_kernel<4>, grid, block, 0, s, a, pp, *ln);
    if (ln_done) *ln_done = true;
  } else {
    launch_reduce(a, epi, pl.splits, partial, s);
  }
  return hipGetLastError();
}

}  // namespace rc
