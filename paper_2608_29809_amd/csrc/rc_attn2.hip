// bf16 cross-attention of the active rows to the text tokens (head dim 72),
// with the delta-column probabilities of the localisation maps (Sec. 3.2).
// The text values are stored transposed ([72][keys] per head).  (The self-
// attention over the cache, rc_attn3.hip, descends from this kernel.)
//
// Same decomposition as rc_attn.hip -- one workgroup = 4 waves = 128 queries
// of one (chain, head, key range), each wave 32 queries, scores formed
// transposed (S^T = K Q^T) so each lane owns one query, probabilities reused
// in registers as the B operand of O^T = V^T P^T -- with these changes:
//
// * K and V^T tiles (64 keys) move global -> LDS with global_load_lds_dwordx4
//   into a two-stage ring, one barrier per tile.
// * Key order inside a 32-key sub-tile: the K row that lane m supplies is
//   key pi(m) = ((m>>4)&1)*16 + ((m>>2)&1)*8 + ((m>>3)&1)*4 + (m&3).  Then the
//   16 accumulators of lane group g are keys c*16 + g*8 + k (c = 0,1; k = 0..7)
//   in order, so each PV instruction reads 8 contiguous keys of V^T (one
//   16-byte LDS read), and the eight lanes of every 16-byte read phase of the
//   K tile (row stride 144 bytes) touch eight disjoint bank groups.
// * V^T tile rows are 128 bytes with their 16-byte chunks XOR-swizzled by
//   (row & 7), conflict-free for the 32-row operand reads.
// * Softmax in the exp2 domain on raw scores: p = exp2(s*c - m*c) (one FMA +
//   v_exp), running max on raw scores, and the output rescale is skipped when
//   no query of the wave raised its maximum.
// * Key ranges split unevenly over grid.y so the grid fills the chip; the
//   deterministic combine is rc_attn.hip's.
#include "rc_common.h"
#include "rc_launch.h"
#include "rc_internal.h"

namespace rc {

constexpr int A2_BQ = 128, A2_BK = 64;

__device__ __forceinline__ int key_perm2(int m) {
  return ((m >> 4) & 1) * 16 + ((m >> 2) & 1) * 8 + ((m >> 3) & 1) * 4 + (m & 3);
}

__device__ __forceinline__ void lds_barrier2() { asm volatile("s_barrier" ::: "memory"); }
__device__ __forceinline__ void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// WARM: also warm a.warm into the memory-side cache (a separate instantiation).
template <bool CROSS, int STAGES, bool WARM>
__global__ __launch_bounds__(256, 2) void attn2_kernel(AttnArgs a) {
  constexpr int D = kHeadDim;
  constexpr int KT_BYTES = A2_BK * D * 2;      // 9216: K tile [64][72]
  constexpr int VT_BYTES = D * A2_BK * 2;      // 9216: V^T tile [72][64]
  constexpr int STAGE = KT_BYTES + VT_BYTES;
  constexpr int K_CH = KT_BYTES / 16;          // 576 chunks
  __shared__ __attribute__((aligned(1024))) char lds[STAGES * STAGE + 128 + (WARM ? 256 : 0)];
  // a row of 64 bf16 ones: row 72 of the V^T operand, so that output row 72
  // of O^T accumulates sum_k P[k] -- the softmax denominator, with the same
  // rounded probabilities as the numerator
  char *ones_row = lds + STAGES * STAGE;
  if (threadIdx.x < 8) *(V16 *)(ones_row + threadIdx.x * 16) = V16{{0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u}};

  // the wave index is uniform across the wave; telling the compiler so keeps
  // the per-wave load choices on scalar branches
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, r32 = lane & 31;
  const int heads = a.hidden / D;
  // XCD-aware order: workgroups are dealt to the eight XCDs round-robin, so
  // consecutive logical ids are packed onto one XCD; the query tiles of one
  // (chain, head, key range) are consecutive and read their keys and values
  // through that XCD's L2 instead of each fetching them from HBM.
  const int G = gridDim.x, Y = gridDim.y, T = G * Y * gridDim.z;
  const int p = blockIdx.x + G * (blockIdx.y + Y * blockIdx.z);
  const int L = xcd_logical_id(p, T);
  const int qt = L % G, hy = (L / G) % Y, b = L / (G * Y);
  const int h = hy % heads, split = hy / heads;
  const int n_tiles = a.n_keys / A2_BK;
  const int t_beg = (int)((long)split * n_tiles / a.splits), t_end = (int)((long)(split + 1) * n_tiles / a.splits);
  const bf16 *Kg = (const bf16 *)a.K + b * a.chain_stride + h * a.head_stride;
  const bf16 *Vg = (const bf16 *)a.V + b * a.chain_stride + h * a.head_stride;  // transposed [72][n_keys]
  if (WARM && wave == 0) warm_lines(a.warm, a.warm_lines, p, T, lds + STAGES * STAGE + 128);

  auto issue = [&](int stage, int tile) {
    char *ks = lds + stage * STAGE, *vs = ks + KT_BYTES;
    const int key0 = tile * A2_BK;
    const char *kt = (const char *)(Kg + (size_t)key0 * D);
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const int base = i * 256 + wave * 64;
      if (base < K_CH)
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)(kt + (base + lane) * 16),
                                         (__attribute__((address_space(3))) void *)(ks + base * 16), 16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const int base = i * 256 + wave * 64;
      if (base < K_CH) {
        const int ch = base + lane, d = ch >> 3, lc = (ch & 7) ^ (d & 7);
        const bf16 *src = Vg + (size_t)d * a.n_keys + key0 + lc * 8;
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)src,
                                         (__attribute__((address_space(3))) void *)(vs + base * 16), 16, 0, 0);
      }
    }
  };

  // the first key tiles depend only on (chain, head, key range): they are in
  // flight while the row offsets and the queries are fetched
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (t_beg + s < t_end) issue(s, t_beg + s);

  const int r0 = a.offsets[b], r1 = a.offsets[b + 1];
  const int q0 = r0 + qt * A2_BQ;
  if (q0 >= r1) {  // uniform across the workgroup; no LDS write may land after exit
    wait_vm0();
    return;
  }
  const int my_q = q0 + wave * 32 + r32;
  const bool q_ok = my_q < r1;
  // keys of this chain that are valid (prompt padding masked)
  const int nv = a.text_valid ? min(max(a.text_valid[b], 1), a.n_valid) : a.n_valid;

  bf16x8 qf[5];
  {
    const bf16 *qrow = (const bf16 *)a.Q + (size_t)(q_ok ? my_q : q0) * a.hidden + h * D;
#pragma unroll
    for (int c = 0; c < 5; ++c) {
      const int d0 = c * 16 + g * 8;
      qf[c] = Mfma<bf16>::zero();
      if (q_ok && d0 < D) qf[c] = *(const bf16x8 *)(qrow + d0);
    }
  }

  f32x16 o[3];
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.0f;
  float m_run = -INFINITY;
  float sd[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) sd[j] = -INFINITY;
  const float c2 = a.scale_log2;

  // ring of STAGES tiles: tiles t+1 .. t+STAGES-1 are in flight while tile t
  // is consumed.  Wave 0 issues 6 loads per tile (the 576-chunk K and V
  // tiles leave 64 chunks each over), the other waves 4.
  for (int tile = t_beg; tile < t_end; ++tile) {
    const int stage = (tile - t_beg) % STAGES;
    if (tile + STAGES - 2 < t_end) {
      if (wave == 0) wait_vm<(STAGES - 2) * 6>();
      else wait_vm<(STAGES - 2) * 4>();
    } else {
      wait_vm0();
    }
    lds_barrier2();
    if (tile + STAGES - 1 < t_end) issue((tile - t_beg + STAGES - 1) % STAGES, tile + STAGES - 1);
    const char *ks = lds + stage * STAGE, *vs = ks + KT_BYTES;
    const int key0 = tile * A2_BK;

    // all ten K fragments of the tile are read before the first MFMA
    bf16x8 kf[2][5];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const char *krow = ks + (st * 32 + key_perm2(r32)) * (D * 2);
#pragma unroll
      for (int c = 0; c < 5; ++c) kf[st][c] = *(const bf16x8 *)(krow + (c * 16 + g * 8) * 2);
      // d0 = 72 (c = 4, upper half-wave) lies past the row; it reads the next
      // row, which meets zero queries, and is then zeroed without a branch
      // so that no non-finite neighbour can leak
      kf[st][4] = (g == 0) ? kf[st][4] : Mfma<bf16>::zero();
    }
    f32x16 s[2];
#pragma unroll
    for (int c = 0; c < 5; ++c)
#pragma unroll
      for (int st = 0; st < 2; ++st)
        s[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st][c], qf[c], c == 0 ? f32x16{} : s[st], 0, 0, 0);

    // lane group g, sub-tile st, accumulator e = c*8 + k  <->  key st*32 + c*16 + g*8 + k
    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        if (CROSS) {
          const int key = key0 + st * 32 + (e >> 3) * 16 + g * 8 + (e & 7);
          if (key >= nv) s[st][e] = -INFINITY;
        }
        tmax = fmaxf(tmax, s[st][e]);
      }
    if (CROSS) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (j < a.n_delta) {
          const int rel = a.delta[j] - key0;
          if (rel >= 0 && rel < A2_BK && ((rel >> 3) & 1) == g) {
            const int st = rel >> 5, e = ((rel >> 4) & 1) * 8 + (rel & 7);
#pragma unroll
            for (int ee = 0; ee < 16; ++ee)
              if (ee == e) sd[j] = st ? s[1][ee] : s[0][ee];
          }
        }
      }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    // Lazy rescaling: the reference maximum m_run only moves when some query
    // of the wave gained more than 2^8 over it, so probabilities stay below
    // 256 and the output rescale is rare.  The result is unchanged: every
    // probability and the denominator share the reference.
    const float m_new = fmaxf(m_run, tmax);
    if (__any((m_new - m_run) * c2 > 8.0f)) {
      const float alpha = (m_run == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f((m_run - m_new) * c2);
#pragma unroll
      for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[t][e] *= alpha;
      m_run = m_new;
    }
    const float mc = (m_run == -INFINITY) ? 0.0f : m_run * c2;
    bf16x8 pf[2][2];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int k = 0; k < 8; ++k)
          pf[st][c][k] = (bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[st][c * 8 + k], c2, -mc));

#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int lc = st * 4 + c * 2 + g;  // logical 16-byte chunk of the 64-key row
#pragma unroll
        for (int t = 0; t < 3; ++t) {
          // rows d >= 72 of the V^T operand only feed output rows that are
          // never stored, so their lanes read a clamped in-bounds row
          const int d = min(t * 32 + r32, D - 1);
          const char *va = vs + d * 128 + ((lc ^ (d & 7)) << 4);
          if (t == 2 && r32 == 8) va = ones_row + (lc << 4);
          const bf16x8 vf = *(const bf16x8 *)va;
          o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[st][c], o[t], 0, 0, 0);
        }
      }
  }

  // denominator: output row 72 = accumulator 4 of o[2] in the lower half-wave
  const float l_tot = __shfl(o[2][4], r32, 64);
  if (CROSS && a.pmaps) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j < a.n_delta) {
        const int owner = (a.delta[j] >> 3) & 1;
        float p = (g == owner && m_run != -INFINITY) ? __builtin_amdgcn_exp2f((sd[j] - m_run) * c2) / l_tot : 0.0f;
        p += __shfl_xor(p, 32, 64);
        if (g == 0 && q_ok) a.pmaps[((size_t)h * a.total_rows + my_q) * a.n_delta + j] = p;
      }
    }
  }
  if (!q_ok) return;
  if (a.splits == 1) {
    const float inv = 1.0f / l_tot;
    bf16 *orow = (bf16 *)a.O + (size_t)my_q * a.hidden + h * D;
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = t * 32 + i * 8 + g * 4;
        if (d < D) {
          bf16x4 v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = (bf16)(o[t][i * 4 + j] * inv);
          *(bf16x4 *)(orow + d) = v;
        }
      }
  } else {
    float *orow = a.Opart + ((size_t)split * a.total_rows + my_q) * a.hidden + h * D;
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = t * 32 + i * 8 + g * 4;
        if (d < D) *(f32x4 *)(orow + d) = f32x4{o[t][i * 4], o[t][i * 4 + 1], o[t][i * 4 + 2], o[t][i * 4 + 3]};
      }
    if (g == 0) {
      float *ml = a.ML + (((size_t)split * a.total_rows + my_q) * heads + h) * 2;
      ml[0] = m_run * c2;  // log2-domain maximum, as the combine expects
      ml[1] = l_tot;
    }
  }
}

hipError_t launch_attention2(const AttnArgs &a, int n_chains, int max_rows, hipStream_t s) {
  if (max_rows <= 0) return hipSuccess;
  if (a.n_keys % A2_BK != 0 || a.splits < 1 || a.splits > a.n_keys / A2_BK || a.v_rowmajor) return hipErrorInvalidValue;
  dim3 grid((max_rows + A2_BQ - 1) / A2_BQ, (a.hidden / kHeadDim) * a.splits, n_chains);
  if (a.warm && a.warm_lines > 0) rc_launch(attn2_kernel<true, 2, true>, grid, dim3(256), 0, s, a);
  else rc_launch(attn2_kernel<true, 2, false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace rc
