// bf16 self-attention, third form: a software pipeline over the key tiles in
// which the matrix core works on the scores of tile t+1 and the PV product of
// tile t-1 while the vector ALUs exponentiate tile t, within the same wave.
//
// Operand layouts are those of the cross-attention (rc_attn2.hip): S^T =
// K Q^T with the permuted key rows; O^T = V^T P^T with the swizzled V^T tile
// and the ones row that accumulates the softmax denominator.  128 queries of
// one (chain, head, key range) per workgroup, 32 per wave; exp2 online
// softmax in which the reference maximum only moves when some query of the
// wave gained more than 2^8 over it (so the output rescale is rare and the
// result unchanged); uneven key splits and the deterministic combine.  On
// top of that:
//
// * a four-slot ring: while tile t-1's values and tile t+1's keys are read,
//   tile t+2 streams in; one barrier per tile;
// * the loop carries the scores of the next tile and the probabilities of
//   the previous tile in registers; a rescale of the reference maximum is
//   applied after the previous tile's PV product has been added, so the
//   accumulator sees the same operations in the same order as a
//   tile-by-tile loop;
// * values are stored token-major like the keys ([n_keys][72] per head), so
//   a tile is one contiguous 9216-byte copy; the V^T operand fragments are
//   assembled by LDS transpose reads (ds_read_b64_tr_b16: within a 16-lane
//   group, lane i's k-th element is element i%4 of the 4-element chunk whose
//   address lane 4k + i/4 supplied), two per fragment;
// * tile copies go through lds_dma16 (explicit waits), so the fragment reads
//   of resident tiles do not wait for the copy just issued.
#include "rc_common.h"
#include "rc_launch.h"
#include "rc_internal.h"

#include <type_traits>

namespace rc {

constexpr int A3_BQ = 128, A3_BK = 64, A3_STAGES = 4;

__device__ __forceinline__ int key_perm3(int m) {
  return ((m >> 4) & 1) * 16 + ((m >> 2) & 1) * 8 + ((m >> 3) & 1) * 4 + (m & 3);
}
__device__ __forceinline__ void lds_barrier3() { asm volatile("s_barrier" ::: "memory"); }
__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// WARM: also warm a.warm into the memory-side cache (a separate instantiation,
// so that the kernel without it carries none of its code or LDS).
template <bool WARM>
__global__ __launch_bounds__(256, 2) void attn3_kernel(AttnArgs a) {
  constexpr int D = kHeadDim;
  constexpr int KT_BYTES = A3_BK * D * 2;  // K tile [64][72]
  constexpr int VT_BYTES = A3_BK * D * 2;  // V tile [64][72]
  constexpr int STAGE = KT_BYTES + VT_BYTES;
  constexpr int K_CH = KT_BYTES / 16;      // 576 16-byte chunks per operand tile
  __shared__ __attribute__((aligned(1024))) char lds[A3_STAGES * STAGE + 16 + (WARM ? 256 : 0)];
  // two 4-element chunks read in place of value dims >= 72: (1, 0, 0, 0), so
  // that output row 72 of O^T accumulates sum_k P[k] -- the softmax
  // denominator, with the same rounded probabilities as the numerator -- and
  // zeros for the rows that are never stored
  char *ones_chunk = lds + A3_STAGES * STAGE, *zero_chunk = ones_chunk + 8;
  if (threadIdx.x == 0) *(V16 *)ones_chunk = V16{{0x00003F80u, 0u, 0u, 0u}};

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, r32 = lane & 31;
  const int heads = a.hidden / D;
  // XCD-aware order (query tiles of one (chain, head, key range) share an XCD)
  const int G = gridDim.x, Y = gridDim.y, T = G * Y * gridDim.z;
  const int p = blockIdx.x + G * (blockIdx.y + Y * blockIdx.z);
  const int L = xcd_logical_id(p, T);
  const int qt = L % G, hy = (L / G) % Y, b = L / (G * Y);
  const int h = hy % heads, split = hy / heads;
  const int n_tiles = a.n_keys / A3_BK;
  const int t_beg = (int)((long)split * n_tiles / a.splits), t_end = (int)((long)(split + 1) * n_tiles / a.splits);
  const bf16 *Kg = (const bf16 *)a.K + b * a.chain_stride + h * a.head_stride;
  const bf16 *Vg = (const bf16 *)a.V + b * a.chain_stride + h * a.head_stride;  // [n_keys][72]
  if (WARM && wave == 0) warm_lines(a.warm, a.warm_lines, p, T, lds + A3_STAGES * STAGE + 16);

  auto issue = [&](int stage, int tile) {
    char *ks = lds + stage * STAGE, *vs = ks + KT_BYTES;
    const int key0 = tile * A3_BK;
    const char *kt = (const char *)(Kg + (size_t)key0 * D);
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const int base = i * 256 + wave * 64;
      if (base < K_CH) lds_dma16(kt + (base + lane) * 16, ks + base * 16);
    }
    const char *vt = (const char *)(Vg + (size_t)key0 * D);
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const int base = i * 256 + wave * 64;
      if (base < K_CH) lds_dma16(vt + (base + lane) * 16, vs + base * 16);
    }
  };
  // the first two key tiles depend only on (chain, head, key range): they
  // are in flight while the row offsets and the queries are fetched
  issue(0, t_beg);
  if (t_beg + 1 < t_end) issue(1, t_beg + 1);

  const int r0 = a.offsets[b], r1 = a.offsets[b + 1];
  const int q0 = r0 + qt * A3_BQ;
  if (q0 >= r1) {  // uniform across the workgroup; no LDS write may land after exit
    wait_vm_all();
    return;
  }
  const int my_q = q0 + wave * 32 + r32;
  const bool q_ok = my_q < r1;

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

  const f32x16 zero16 = {};  // C operand of a tile's first score MFMA, kept live
  // S^T of one tile: lane group g, sub-tile st, accumulator e = c*8 + k  <->
  // key st*32 + c*16 + g*8 + k.  For c = 4 the g = 1 lanes read dims 72..79,
  // i.e. the first dims of the next key row (or of value row 0): finite
  // values multiplied by the zero query dims 72..79, adding exact zeros.
  auto scores = [&](int stage, f32x16 *s) {
    const char *ks = lds + stage * STAGE;
    bf16x8 kf[2][5];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const char *krow = ks + (st * 32 + key_perm3(r32)) * (D * 2);
#pragma unroll
      for (int c = 0; c < 5; ++c) kf[st][c] = *(const bf16x8 *)(krow + (c * 16 + g * 8) * 2);
    }
#pragma unroll
    for (int c = 0; c < 5; ++c)
#pragma unroll
      for (int st = 0; st < 2; ++st)
        s[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st][c], qf[c], c == 0 ? zero16 : s[st], 0, 0, 0);
  };

  f32x16 o[3];
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.0f;
  float m_run = -INFINITY;
  const float c2 = a.scale_log2;

  // Transpose reads of the V tile: the fragment of dims 32t + (lane%32) and
  // keys kb..kb+7 (kb = st*32 + c*16 + g*8) is two reads; in the first this
  // lane supplies the 4 dims from d0 of key kb_w + j/4, in the second of key
  // kb_w + 4 + j/4 (16-lane group w = lane/16, j = lane%16).
  const int tw = lane >> 4, tj = lane & 15;
  int v_off[3];  // byte offset of the supplied chunk within a key row block, per dim block t
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    const int d0 = 32 * t + 16 * (tw & 1) + 4 * (tj & 3);
    v_off[t] = ((tj >> 2) * D + d0) * 2;
  }
  const int d0_2 = 64 + 16 * (tw & 1) + 4 * (tj & 3);  // dims of the last block: real below 72
  auto vfrag = [&](const char *vs, int kb, int t) {
    typedef short v4s __attribute__((ext_vector_type(4)));
    typedef short v8s __attribute__((ext_vector_type(8)));
    const char *p0 = vs + kb * (D * 2) + v_off[t];
    const char *p1 = p0 + 4 * D * 2;
    if (t == 2 && d0_2 >= D) p0 = p1 = (d0_2 == D) ? ones_chunk : zero_chunk;
    const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s *)p0);
    const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s *)p1);
    const v8s both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, both);
  };

  // prologue: wait for tile t_beg (every load issued after its last one --
  // tile t_beg+1, the queries -- may still be in flight), scores of t_beg
  if (t_beg + 1 < t_end) {
    if (wave == 0) asm volatile("s_waitcnt vmcnt(6)" ::: "memory");  // wave 0 issues 6 loads per tile, others 4
    else asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  } else {
    wait_vm_all();
  }
  lds_barrier3();
  f32x16 s_cur[2];
  scores(0, s_cur);

  // One key tile i (tile = t_beg + i): wait for tile i+1 and recycle the slot
  // of tile i-2 for tile i+2, update the running maximum with tile i's
  // scores, then a run of MFMA groups: the score MFMAs of tile i+1, then the
  // PV MFMAs of tile i-1 (probabilities from the previous step, values still
  // in their ring slot), one MFMA per group, each group also taking its
  // share of tile i's exponentials (and, under the score MFMAs, the value
  // fragment reads), so that the vector ALU works while the matrix core
  // runs.  Group boundaries are scheduling barriers, and each exponential's
  // operand and result pass through an empty asm so that the compiler keeps
  // it inside its group instead of batching all of them before or after the
  // MFMAs.  A rescale of the reference maximum is applied to o after the
  // groups, once the PV contribution of tile i-1 (relative to the old
  // maximum) is in; every output element sees the same operations in the
  // same order as a tile-by-tile loop.
  auto step = [&](int i, auto has_next_c, auto has_prev_c, f32x16 *s_in, f32x16 *s_out, bf16x8 (*p_in)[2],
                  bf16x8 (*p_out)[2]) {
    constexpr bool HAS_NEXT = decltype(has_next_c)::value;
    constexpr bool HAS_PREV = decltype(has_prev_c)::value;
    constexpr int NS = HAS_NEXT ? 10 : 0, NP = HAS_PREV ? 12 : 0, NG = NS + NP;
    const int tile = t_beg + i;
    wait_vm_all();
    lds_barrier3();
    if (tile + 2 < t_end) issue((i + 2) % A3_STAGES, tile + 2);
    bf16x8 kf[2][5];  // key fragments of tile i+1, consumed in (c, st) order
    if (HAS_NEXT) {
      const char *ks = lds + ((i + 1) % A3_STAGES) * STAGE;
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const char *krow = ks + (st * 32 + key_perm3(r32)) * (D * 2);
#pragma unroll
        for (int c = 0; c < 5; ++c) kf[st][c] = *(const bf16x8 *)(krow + (c * 16 + g * 8) * 2);
      }
    }
    const char *vs = lds + ((i + A3_STAGES - 1) % A3_STAGES) * STAGE + KT_BYTES;
    bf16x8 vf[12];  // value fragment k = (st, c, t) = (k / 6, k / 3 % 2, k % 3) of tile i-1
    auto vread = [&](int k) { vf[k] = vfrag(vs, (k / 6) * 32 + ((k / 3) % 2) * 16 + (tw >> 1) * 8, k % 3); };
    if (HAS_PREV && !HAS_NEXT) {
#pragma unroll
      for (int k = 0; k < 12; ++k) vread(k);
    }

    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) tmax = fmaxf(tmax, s_in[st][e]);
    tmax = half_swap_max(tmax);
    const float m_new = fmaxf(m_run, tmax);
    const bool resc = __any((m_new - m_run) * c2 > 8.0f);
    const float alpha = (m_run == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f((m_run - m_new) * c2);
    m_run = resc ? m_new : m_run;
    const float mc = (m_run == -INFINITY) ? 0.0f : m_run * c2;
    __builtin_amdgcn_sched_barrier(0);

    float pe[32];  // exponentials of tile i, element st*16 + c*8 + k
    // the wave in its MFMA groups takes issue priority over the other wave
    // of its SIMD (in its barrier wait or conversion tail)
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int j = 0; j < NG; ++j) {
      if (j < NS) {
        const int c = j / 2, st = j % 2;
        s_out[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st][c], qf[c], c == 0 ? zero16 : s_out[st], 0, 0, 0);
        if (HAS_PREV) vread(j);
      } else {
        const int k = j - NS;
        o[k % 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[k], p_in[k / 6][(k / 3) % 2], o[k % 3], 0, 0, 0);
        if (HAS_NEXT && j < 12) vread(j);
      }
      const int e0 = 32 * j / NG, e1 = 32 * (j + 1) / NG;
#pragma unroll
      for (int e = e0; e < e1; ++e) {
        float x = __builtin_fmaf(s_in[e / 16][e % 16], c2, -mc);
        asm volatile("" : "+v"(x));
        pe[e] = __builtin_amdgcn_exp2f(x);
        asm volatile("" : "+v"(pe[e]));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_setprio(0);
    if (NG == 0) {
#pragma unroll
      for (int e = 0; e < 32; ++e) pe[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s_in[e / 16][e % 16], c2, -mc));
    }
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int k = 0; k < 8; ++k) p_out[st][c][k] = (bf16)pe[st * 16 + c * 8 + k];
    if (resc) {
#pragma unroll
      for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[t][e] *= alpha;
    }
  };
  // PV of the last tile (its probabilities are in p_last)
  auto drain = [&](int i, bf16x8 (*p_last)[2]) {
    const char *vs = lds + (i % A3_STAGES) * STAGE + KT_BYTES;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int t = 0; t < 3; ++t)
          o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag(vs, st * 32 + c * 16 + (tw >> 1) * 8, t),
                                                         p_last[st][c], o[t], 0, 0, 0);
  };
  f32x16 s_alt[2];
  bf16x8 pA[2][2], pB[2][2];
  const int n = t_end - t_beg;
  std::true_type T_;
  std::false_type F_;
  if (n > 1) step(0, T_, F_, s_cur, s_alt, pB, pA);
  else step(0, F_, F_, s_cur, s_alt, pB, pA);
  int i = 1;
  for (; i + 2 < n; i += 2) {
    step(i, T_, T_, s_alt, s_cur, pA, pB);
    step(i + 1, T_, T_, s_cur, s_alt, pB, pA);
  }
  if (i + 1 < n) {
    step(i, T_, T_, s_alt, s_cur, pA, pB);
    step(i + 1, F_, T_, s_cur, s_alt, pB, pA);
    drain(i + 1, pA);
  } else if (i < n) {
    step(i, F_, T_, s_alt, s_cur, pA, pB);
    drain(i, pB);
  } else {
    drain(0, pA);
  }

  const float l_tot = __shfl(o[2][4], r32, 64);  // output row 72: the denominator
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
    // a split stores its own normalised output (a convex combination of
    // value rows, so bf16 keeps its relative precision) with its log2-domain
    // maximum and denominator; the combine re-weights the splits
    const float inv = 1.0f / l_tot;
    bf16 *orow = (bf16 *)a.Opart + ((size_t)split * a.total_rows + my_q) * a.hidden + h * D;
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
    if (g == 0) {
      float *ml = a.ML + (((size_t)split * a.total_rows + my_q) * heads + h) * 2;
      ml[0] = m_run * c2;
      ml[1] = l_tot;
    }
  }
}

// Combine of normalised bf16 split outputs: O = sum_s w_s O_s / sum_s w_s with
// w_s = 2^(m_s - max m) l_s, in split order.  One thread per (row, head,
// 8 dims); all loads are issued before use.
__global__ __launch_bounds__(256) void attn_combine_norm_kernel(const bf16 *Opart, const float *ML, bf16 *O, int R,
                                                                int heads, int splits) {
  constexpr int G = kHeadDim / 8;
  const int C = heads * kHeadDim;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)R * heads * G) return;
  const int r = idx / (heads * G);
  const int rem = idx - (long)r * heads * G;
  const int h = rem / G, d = (rem - h * G) * 8;
  constexpr int SMAX = 16;
  float2 ml[SMAX];
  bf16x8 p[SMAX];
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < splits) {
      ml[s] = *(const float2 *)(ML + (((size_t)s * R + r) * heads + h) * 2);
      p[s] = *(const bf16x8 *)(Opart + ((size_t)s * R + r) * C + h * kHeadDim + d);
    }
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < splits) M = fmaxf(M, ml[s].x);
  float num[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f}, den = 0.0f;
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < splits) {
      const float w = exp2f(ml[s].x - M) * ml[s].y;
#pragma unroll
      for (int k = 0; k < 8; ++k) num[k] += w * (float)p[s][k];
      den += w;
    }
  const float inv = 1.0f / den;
  bf16x8 v;
#pragma unroll
  for (int k = 0; k < 8; ++k) v[k] = (bf16)(num[k] * inv);
  *(bf16x8 *)(O + (size_t)r * C + h * kHeadDim + d) = v;
}

hipError_t launch_attn_combine_norm(const void *Opart, const float *ML, void *O, int R, int heads, int splits,
                                    hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (splits < 1 || splits > 16) return hipErrorInvalidValue;
  const long n = (long)R * heads * (kHeadDim / 8);
  rc_launch(attn_combine_norm_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (const bf16 *)Opart, ML, (bf16 *)O, R,
            heads, splits);
  return hipGetLastError();
}

hipError_t launch_attention3(const AttnArgs &a, int n_chains, int max_rows, hipStream_t s) {
  if (max_rows <= 0) return hipSuccess;
  if (a.n_keys % A3_BK != 0 || a.splits < 1 || a.splits > a.n_keys / A3_BK || !a.v_rowmajor)
    return hipErrorInvalidValue;
  dim3 grid((max_rows + A3_BQ - 1) / A3_BQ, (a.hidden / kHeadDim) * a.splits, n_chains);
  if (a.warm && a.warm_lines > 0) rc_launch(attn3_kernel<true>, grid, dim3(256), 0, s, a);
  else rc_launch(attn3_kernel<false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace rc
