// bf16 cross-attention of the active rows to the text tokens (head dim 72),
// with the query projection fused in and the delta-column probabilities of
// the localisation maps (Sec. 3.2).  The text values are stored transposed
// ([72][keys] per head).
//
// Operand layouts shared with the self-attention (rc_attn3.hip): scores are
// formed transposed (S^T = K Q^T) so each lane owns one query, and the
// probabilities are reused in registers as the B operand of O^T = V^T P^T.
// * Key order inside a 32-key sub-tile: the K row that lane m supplies is
//   key pi(m) = ((m>>4)&1)*16 + ((m>>2)&1)*8 + ((m>>3)&1)*4 + (m&3).  Then the
//   16 accumulators of lane group g are keys c*16 + g*8 + k (c = 0,1; k = 0..7)
//   in order, so each PV instruction reads 8 contiguous keys of V^T (one
//   16-byte LDS read), and the eight lanes of every 16-byte read phase of the
//   K tile (row stride 144 bytes) touch eight disjoint bank groups.
// * V^T tile rows are 128 bytes with their 16-byte chunks XOR-swizzled by
//   (row & 7), conflict-free for the 32-row operand reads.
// * Softmax in the exp2 domain on raw scores: p = exp2(s*c - m*c) (one FMA +
//   v_exp); a row of bf16 ones as row 72 of the V^T operand makes output row
//   72 the denominator, with the same rounded probabilities as the numerator.
#include "rc_common.h"
#include "rc_launch.h"
#include "rc_internal.h"

namespace rc {

constexpr int A2_BK = 64;  // keys per text tile

__device__ __forceinline__ int key_perm2(int m) {
  return ((m >> 4) & 1) * 16 + ((m >> 2) & 1) * 8 + ((m >> 3) & 1) * 4 + (m & 3);
}

__device__ __forceinline__ void lds_barrier2() { asm volatile("s_barrier" ::: "memory"); }
__device__ __forceinline__ void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// ---------------------------------------------------------------------------
// Cross-attention with its query projection fused in (launch_attention2q).
//
// One workgroup = 64 active rows of one (chain, head), eight waves, one
// workgroup per CU (12 x 16 = 192 workgroups at 723 rows).
//
// Phase 1 projects the 64 x 72 query tile Q = Xq . Wq_h^T + bq_h.  The rows
// of Xq and the head's 72 rows of Wq stream through LDS in 128-wide K chunks
// (16 KB + 18 KB per stage, three stages, coalesced direct-to-LDS copies; the
// 16-byte pieces of each 256-byte row are XOR-swizzled by row & 15, so the
// fragment reads of 16 consecutive rows are conflict-free).  Few, large
// chunks matter here: each chunk costs one wait, one barrier, the copy issue
// and the LDS read latency in series.  Wave w = 4 rh + kq takes rows
// 32 rh .. 32 rh + 31 and the 32-wide K quarter kq of every chunk: per 16 k,
// one Xq fragment and three Wq fragments feed three 32x32x16 MFMAs (operand
// A = Wq rows d = 32 t + r32, rows past 71 reading row 71 and never stored;
// operand B = the query rows).  The four K-quarter partials are summed in
// the order kq = 0..3, plus the bias, into the bf16 query tile (the GEMM's
// rounding of Q).
//
// Phase 2 attends to the text: wave w = 2 kt + qh takes queries 32 qh .. and
// key sub-tile kt (keys 32 kt .. 32 kt + 31 of the at most 128 text keys),
// forms its scores S^T = K Q^T, its own maximum, probabilities and P.V with
// the denominator row (the operand layouts above); the four partial
// softmaxes of a query merge in LDS with weights exp2(m_kt - M) in the order
// kt = 0..3.  The text key/value tiles and the first two weight chunks are
// copied at entry, before the row offsets are read.
constexpr int AQ_ROWS = 64, AQ_KC = 128;

__device__ __forceinline__ int aq_swz(int row) { return row & 15; }

template <int NCH, bool WARM>
__global__ __launch_bounds__(512, 1) void attn2q_kernel(AttnArgs a) {
  constexpr int D = kHeadDim;
  constexpr int KT_BYTES = A2_BK * D * 2, VT_BYTES = D * A2_BK * 2, STAGE = KT_BYTES + VT_BYTES;
  constexpr int K_CH = KT_BYTES / 16;
  constexpr int QS_LD = 88;  // bf16 row stride of the query tile (176 bytes: conflict-free 16-byte reads)
  constexpr int RROW = AQ_KC * 2;  // 256-byte ring rows
  constexpr int RX = AQ_ROWS * RROW, RW = D * RROW, RSTAGE = RX + RW, RSTAGES = 3;
  constexpr int REG = 2 * STAGE;                            // after the key/value tiles
  constexpr int PART_OFF = REG;                             // [4][64][72] fp32 projection partials,
                                                            // then [8][32][72] fp32 P.V partials
  constexpr int QS_OFF = PART_OFF + 4 * AQ_ROWS * D * 4;    // [64][88] bf16 query tile
  constexpr int ML_OFF = QS_OFF + AQ_ROWS * QS_LD * 2;      // [2][8][32] log2-domain maxima, denominators
  constexpr int SD_OFF = ML_OFF + 2 * 8 * 32 * 4;           // [8][64] raw scores of the delta columns
  constexpr int REG_END = SD_OFF + 8 * AQ_ROWS * 4;
  constexpr int RING_END = REG + RSTAGES * RSTAGE;
  // the ring overlaps everything of the region: it is dead once the last
  // chunk's fragments are read, before any partial is written
  constexpr int ONES_OFF = RING_END > REG_END ? RING_END : REG_END;
  constexpr int WARM_OFF = ONES_OFF + 128;
  static_assert(WARM_OFF + 256 <= 160 * 1024, "LDS of one CU");
  __shared__ __attribute__((aligned(1024))) char lds[WARM_OFF + (WARM ? 256 : 0)];
  char *ones_row = lds + ONES_OFF;
  if (threadIdx.x < 8) *(V16 *)(ones_row + threadIdx.x * 16) = V16{{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u}};

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, r32 = lane & 31;
  const int C = a.hidden;
  // XCD-aware order with the query tiles of one (chain, head) consecutive:
  // they share that head's projection weights through one XCD's L2
  const int G = gridDim.x, Y = gridDim.y, T = G * Y * gridDim.z;
  const int p = blockIdx.x + G * (blockIdx.y + Y * blockIdx.z);
  const int L = xcd_logical_id(p, T);
  const int qt = L % G, h = (L / G) % Y, b = L / (G * Y);
  const int n_tiles = a.n_keys / A2_BK;
  const bf16 *Kg = (const bf16 *)a.K + b * a.chain_stride + h * a.head_stride;
  const bf16 *Vg = (const bf16 *)a.V + b * a.chain_stride + h * a.head_stride;  // transposed [72][n_keys]
  if (WARM && wave == 0) warm_lines(a.warm, a.warm_lines, p, T, lds + WARM_OFF);
  // operands of later phases, fetched now so their latency hides under
  // phase 1: this thread's bias columns c0 + 8j of the query tile
  // reduction, and the chain's valid key count
  float qb[D / 8];
#pragma unroll
  for (int j = 0; j < D / 8; ++j) qb[j] = a.q_b[h * D + (tid & 7) + 8 * j];
  const int nv = a.text_valid ? min(max(a.text_valid[b], 1), a.n_valid) : a.n_valid;

  // copies that depend only on (chain, head) go first, in flight while the
  // row offsets are fetched: every text key/value tile, then the first two
  // weight chunks
  for (int tile = 0; tile < n_tiles; ++tile) {
    char *ks = lds + tile * STAGE, *vs = ks + KT_BYTES;
    const char *kt = (const char *)(Kg + (size_t)tile * A2_BK * D);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int base = i * 512 + wave * 64;
      if (base < K_CH) lds_dma16(kt + (base + lane) * 16, ks + base * 16);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int base = i * 512 + wave * 64;
      if (base < K_CH) {
        const int ch = base + lane, d = ch >> 3, lc = (ch & 7) ^ (d & 7);
        lds_dma16(Vg + (size_t)d * a.n_keys + tile * A2_BK + lc * 8, vs + base * 16);
      }
    }
  }
  const bf16 *wq = (const bf16 *)a.q_w + (size_t)h * D * C;
  auto issue_w = [&](int stage, int chunk) {  // 3 copies on waves 0 and 1, 2 on the others
    char *sw = lds + REG + stage * RSTAGE + RX;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const int base = i * 512 + wave * 64;
      if (base < D * 16) {
        const int pc = base + lane, row = pc >> 4, lc = (pc & 15) ^ aq_swz(row);
        lds_dma16(wq + (size_t)row * C + chunk * AQ_KC + lc * 8, sw + base * 16);
      }
    }
  };
  issue_w(0, 0);
  issue_w(1, 1);

  const int2 rr = chain_rows(a, b);
  const int r0 = rr.x, r1 = rr.y;
  const int q0 = r0 + qt * AQ_ROWS;
  if (q0 >= r1) {  // uniform across the workgroup; every copy lands before exit
    wait_vm0();
    return;
  }

  // phase 1: the projection.  The two pieces of Xq this lane copies per
  // chunk: rows xr (rows past the chain's last are clamped to it and never
  // stored).
  const bf16 *xsrc[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int pc = i * 512 + wave * 64 + lane, xr = pc >> 4;
    xsrc[i] = (const bf16 *)a.q_x + (size_t)min(q0 + xr, r1 - 1) * C + (((pc & 15) ^ aq_swz(xr)) << 3);
  }
  auto issue_x = [&](int stage, int chunk) {  // 2 copies per wave
    char *sx = lds + REG + stage * RSTAGE;
#pragma unroll
    for (int i = 0; i < 2; ++i) lds_dma16(xsrc[i] + chunk * AQ_KC, sx + (i * 512 + wave * 64) * 16);
  };
  issue_x(0, 0);
  issue_x(1, 1);
  const int rh = wave >> 2, kq = wave & 3;
  int xo[2], wo[2][3];
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2) {
    const int lc = kq * 4 + s2 * 2 + g;  // 16-byte piece of k = 32 kq + 16 s2 + 8 g
    const int xrow = rh * 32 + r32;
    xo[s2] = xrow * RROW + ((lc ^ aq_swz(xrow)) << 4);
#pragma unroll
    for (int t = 0; t < 3; ++t) {
      const int row = min(t * 32 + r32, D - 1);
      wo[s2][t] = RX + row * RROW + ((lc ^ aq_swz(row)) << 4);
    }
  }
  f32x16 acc[3];
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[t][e] = 0.0f;
  for (int ch = 0; ch < NCH; ++ch) {
    // copies retire in order.  Chunk ch has landed once at most the copies
    // issued after it are outstanding: the first wait leaves chunk 1's two
    // Xq copies, later ones chunk ch+1's (Wq then Xq: 5 on waves 0 and 1,
    // 4 on the others).
    if (ch == 0) wait_vm<2>();
    else if (ch + 1 < NCH) {
      if (wave < 2) wait_vm<5>();
      else wait_vm<4>();
    } else {
      wait_vm0();
    }
    lds_barrier2();  // chunk ch is visible to all waves; stage (ch + 2) % 3 is free
    if (ch + 2 < NCH) {
      issue_w((ch + 2) % RSTAGES, ch + 2);
      issue_x((ch + 2) % RSTAGES, ch + 2);
    }
    const char *st = lds + REG + (ch % RSTAGES) * RSTAGE;
    bf16x8 xf[2], wf[2][3];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      xf[s2] = *(const bf16x8 *)(st + xo[s2]);
#pragma unroll
      for (int t = 0; t < 3; ++t) wf[s2][t] = *(const bf16x8 *)(st + wo[s2][t]);
    }
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int t = 0; t < 3; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[s2][t], xf[s2], acc[t], 0, 0, 0);
  }
  lds_barrier2();  // every wave is done with the ring, which the partials overlap
  // block t of Q^T: lane (r32, g) holds query 32 rh + r32 and columns
  // d = 32 t + 8 (e / 4) + 4 g + e % 4, four consecutive per e / 4
  float *part = (float *)(lds + PART_OFF);
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int a4 = 0; a4 < 4; ++a4) {
      const int d = t * 32 + a4 * 8 + g * 4;
      if (d < D)
        *(f32x4 *)(part + (kq * AQ_ROWS + rh * 32 + r32) * D + d) =
            f32x4{acc[t][a4 * 4], acc[t][a4 * 4 + 1], acc[t][a4 * 4 + 2], acc[t][a4 * 4 + 3]};
    }
  __syncthreads();
  // the four partials summed in the order kq = 0..3, plus the bias: the bf16
  // query tile.  Thread t: query t / 8, columns t % 8 + 8 j.
  bf16 *qs = (bf16 *)(lds + QS_OFF);
  {
    const int q = tid >> 3, c0 = tid & 7;
#pragma unroll
    for (int j = 0; j < D / 8; ++j) {
      const int d = c0 + 8 * j;
      const float v = ((part[q * D + d] + part[(AQ_ROWS + q) * D + d]) + part[(2 * AQ_ROWS + q) * D + d]) +
                      part[(3 * AQ_ROWS + q) * D + d];
      qs[q * QS_LD + d] = (bf16)(v + qb[j]);
    }
    qs[q * QS_LD + D + c0] = (bf16)0.0f;  // columns 72..79
  }
  wait_vm0();  // this wave's key/value copies have landed
  __syncthreads();

  // phase 2: queries 32 qh .., key sub-tile kt
  const int qh = wave & 1, kt = wave >> 1;
  const float c2 = a.scale_log2;
  float *ml = (float *)(lds + ML_OFF);
  float *sd = (float *)(lds + SD_OFF);
  f32x16 o[3];
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.0f;
  float mc = -INFINITY, l_w = 0.0f;
  if (kt * 32 < a.n_keys) {
    const int tile = kt >> 1, st = kt & 1;
    const char *ks = lds + tile * STAGE, *vs = ks + KT_BYTES;
    bf16x8 qf[5], kf[5];
    const char *krow = ks + (st * 32 + key_perm2(r32)) * (D * 2);
#pragma unroll
    for (int c = 0; c < 5; ++c) {
      qf[c] = *(const bf16x8 *)(qs + (qh * 32 + r32) * QS_LD + c * 16 + g * 8);
      kf[c] = *(const bf16x8 *)(krow + (c * 16 + g * 8) * 2);
    }
    // d0 = 72 of the upper half-wave reads into the next row; zeroed
    kf[4] = (g == 0) ? kf[4] : Mfma<bf16>::zero();
    f32x16 sc;
#pragma unroll
    for (int c = 0; c < 5; ++c)
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[c], qf[c], c == 0 ? f32x16{} : sc, 0, 0, 0);
    // lane (r32 = query, g): accumulator e <-> key 32 kt + (e >> 3) * 16 + g * 8 + (e & 7)
    float tmax = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = kt * 32 + (e >> 3) * 16 + g * 8 + (e & 7);
      if (key >= nv) sc[e] = -INFINITY;
      tmax = fmaxf(tmax, sc[e]);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j < a.n_delta) {
        const int rel = a.delta[j] - kt * 32;
        if (rel >= 0 && rel < 32 && ((rel >> 3) & 1) == g) {
          const int e = ((rel >> 4) & 1) * 8 + (rel & 7);
          float v = 0.0f;
#pragma unroll
          for (int ee = 0; ee < 16; ++ee)
            if (ee == e) v = sc[ee];
          sd[j * AQ_ROWS + qh * 32 + r32] = v;
        }
      }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    mc = (tmax == -INFINITY) ? -INFINITY : tmax * c2;
    const float msub = (tmax == -INFINITY) ? 0.0f : mc;
    bf16x8 pf[2];
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int k = 0; k < 8; ++k) pf[c][k] = (bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(sc[c * 8 + k], c2, -msub));
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int lc = st * 4 + c * 2 + g;  // logical 16-byte chunk of the 64-key row
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const int d = min(t * 32 + r32, D - 1);
        const char *va = vs + d * 128 + ((lc ^ (d & 7)) << 4);
        if (t == 2 && r32 == 8) va = ones_row + (lc << 4);
        const bf16x8 vf = *(const bf16x8 *)va;
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[c], o[t], 0, 0, 0);
      }
    }
    l_w = __shfl(o[2][4], r32, 64);  // output row 72: the denominator
  }
  // P.V partials over the projection partials (all read before the last
  // barrier); accumulators 4a..4a+3 of block t are 4 consecutive columns
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int a4 = 0; a4 < 4; ++a4) {
      const int d = t * 32 + a4 * 8 + g * 4;
      if (d < D)
        *(f32x4 *)(part + (wave * 32 + r32) * D + d) =
            f32x4{o[t][a4 * 4], o[t][a4 * 4 + 1], o[t][a4 * 4 + 2], o[t][a4 * 4 + 3]};
    }
  if (g == 0) {
    ml[wave * 32 + r32] = mc;
    ml[8 * 32 + wave * 32 + r32] = l_w;
  }
  __syncthreads();

  // merge of the four key sub-tiles of each query, in the order kt = 0..3:
  // thread t takes query t / 8 and columns t % 8 + 8 j
  {
    const int q = tid >> 3, c0 = tid & 7, ql = q & 31, wq0 = q >> 5;  // waves 2 kt + (q >> 5)
    float mx = -INFINITY;
#pragma unroll
    for (int k4 = 0; k4 < 4; ++k4) mx = fmaxf(mx, ml[(2 * k4 + wq0) * 32 + ql]);
    float al[4], den = 0.0f;
#pragma unroll
    for (int k4 = 0; k4 < 4; ++k4) {
      const float m = ml[(2 * k4 + wq0) * 32 + ql];
      al[k4] = (m == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m - mx);
      den += al[k4] * ml[8 * 32 + (2 * k4 + wq0) * 32 + ql];
    }
    const float inv = 1.0f / den;
    if (q0 + q < r1) {
      bf16 *orow = (bf16 *)a.O + (size_t)(q0 + q) * C + h * D;
#pragma unroll
      for (int j = 0; j < D / 8; ++j) {
        const int d = c0 + 8 * j;
        float num = 0.0f;
#pragma unroll
        for (int k4 = 0; k4 < 4; ++k4) num += al[k4] * part[((2 * k4 + wq0) * 32 + ql) * D + d];
        orow[d] = (bf16)(num * inv);
      }
      if (a.pmaps && c0 < a.n_delta)
        a.pmaps[((size_t)h * a.total_rows + q0 + q) * a.n_delta + c0] =
            __builtin_amdgcn_exp2f(__builtin_fmaf(sd[c0 * AQ_ROWS + q], c2, -mx)) * inv;
    }
  }
}

hipError_t launch_attention2q(const AttnArgs &a, int n_chains, int max_rows, hipStream_t s) {
  if (max_rows <= 0) return hipSuccess;
  if (a.n_keys % A2_BK != 0 || a.n_keys > 2 * A2_BK || a.splits != 1 || a.v_rowmajor || !a.q_x || !a.q_w ||
      !a.q_b || a.n_delta < 0 || a.n_delta > 8)
    return hipErrorInvalidValue;
  dim3 grid((max_rows + AQ_ROWS - 1) / AQ_ROWS, a.hidden / kHeadDim, n_chains);
  const bool warm = a.warm && a.warm_lines > 0;
  if (a.hidden == 9 * AQ_KC) {
    if (warm) rc_launch(attn2q_kernel<9, true>, grid, dim3(512), 0, s, a);
    else rc_launch(attn2q_kernel<9, false>, grid, dim3(512), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace rc
