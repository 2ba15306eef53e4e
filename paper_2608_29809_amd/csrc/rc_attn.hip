// Variable-query-length flash-style attention for head dim 72 on matrix cores.
//
// Region-level sparse attention (Sec. 3.3): queries are only the active rows
// of each chain (compact, chains concatenated), while keys and values span
// every token of the chain's cache slot -- fresh rows for active tokens
// (written by the QKV epilogue just before) and cached rows for the rest.
// The same kernel serves cross-attention to the padded text keys and then
// also emits, per head, the probability of each delta text column: the
// cross-attention map of Sec. 3.2.
//
// Work split: one workgroup = 4 waves = 128 queries of one (chain, head,
// key-split); each wave owns 32 queries.  Key/value tiles of 64 keys are
// staged in LDS and shared by the four waves.  Scores are formed transposed
// (S^T = K Q^T) so that each lane holds one query and 16 keys; those
// accumulators, converted to the storage type, are exactly the B operand of
// O^T = V^T P^T, so probabilities never leave registers.  K rows are loaded
// into the A operand in a permuted order that makes each lane's 16 keys
// contiguous, which lets the transposed-V operand be read as contiguous
// LDS vectors.  Values are cached transposed ([72][N] per head) for the
// same reason.  Softmax runs in the exp2 domain with the 1/sqrt(72) scale
// folded into one multiply.
#include "rc_common.h"
#include "rc_launch.h"
#include "rc_internal.h"

namespace rc {

constexpr int ATT_BQ = 128;   // queries per workgroup
constexpr int ATT_BK = 64;    // keys per tile

// A-operand row m of a 32-key sub-tile is loaded from key pi(m) so that
// accumulator element e of lane group g corresponds to key g*16 + e.
__device__ __forceinline__ int key_perm(int m) { return ((m >> 2) & 1) * 16 + (m >> 3) * 4 + (m & 3); }

template <typename T, bool EMIT>
__global__ __launch_bounds__(256) void attn_kernel(AttnArgs a) {
  typedef Mfma<T> MF;
  typedef typename MF::frag frag;
  constexpr int KS = MF::KS;
  constexpr int D = kHeadDim;
  constexpr int DC = (D + 2 * KS - 1) / (2 * KS);     // k-chunks over the head dim
  constexpr int VE = 16 / sizeof(T);
  constexpr int VT_LD = ATT_BK + VE;                   // padded row of the V^T tile
  constexpr int K_CH = ATT_BK * D * sizeof(T) / 16;    // 16-byte chunks of a K tile
  constexpr int V_CPR = ATT_BK * sizeof(T) / 16;       // chunks per V^T row
  constexpr int V_CH = D * V_CPR;
  constexpr int K_IT = (K_CH + 255) / 256;
  constexpr int V_IT = (V_CH + 255) / 256;
  constexpr int PCH = 32 / (2 * KS);                   // PV instructions per 32-key sub-tile

  __shared__ __attribute__((aligned(16))) T Ks[ATT_BK * D];
  __shared__ __attribute__((aligned(16))) T Vs[D * VT_LD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5;
  const int heads = a.hidden / D;
  const int b = blockIdx.z;
  const int h = blockIdx.y % heads, split = blockIdx.y / heads;
  const int r0 = a.offsets[b], r1 = a.offsets[b + 1];
  const int q0 = r0 + blockIdx.x * ATT_BQ;
  if (q0 >= r1) return;  // uniform across the workgroup
  const int my_q = q0 + wave * 32 + (lane & 31);
  const bool q_ok = my_q < r1;
  // keys of this chain that are valid (prompt padding masked)
  const int nv = a.text_valid ? min(max(a.text_valid[b], 1), a.n_valid) : a.n_valid;

  const int keys_per_split = a.n_keys / a.splits;
  const int kbeg = split * keys_per_split, kend = kbeg + keys_per_split;
  const T *Kg = (const T *)a.K + b * a.chain_stride + h * a.head_stride;
  const T *Vg = (const T *)a.V + b * a.chain_stride + h * a.head_stride;

  // queries as the B operand of S^T = K Q^T
  frag qf[DC];
  {
    const T *qrow = (const T *)a.Q + (size_t)my_q * a.hidden + h * D;
#pragma unroll
    for (int c = 0; c < DC; ++c) {
      const int d0 = c * 2 * KS + g * KS;
      qf[c] = (q_ok && d0 < D) ? *(const frag *)(qrow + d0) : MF::zero();
    }
  }

  V16 rk[K_IT], rv[V_IT];
  auto load = [&](int key0) {
    const T *kt = Kg + (size_t)key0 * D;
#pragma unroll
    for (int i = 0; i < K_IT; ++i) {
      const int ch = tid + i * 256;
      if (ch < K_CH) rk[i] = *(const V16 *)(kt + ch * VE);
    }
#pragma unroll
    for (int i = 0; i < V_IT; ++i) {
      const int ch = tid + i * 256;
      if (ch < V_CH) {
        if (a.v_rowmajor) {  // chunk = VE consecutive dims of one key
          const int key = ch / (D / VE), c = ch % (D / VE);
          rv[i] = *(const V16 *)(Vg + (size_t)(key0 + key) * D + c * VE);
        } else {             // chunk = VE consecutive keys of one dim
          const int d = ch / V_CPR, c = ch % V_CPR;
          rv[i] = *(const V16 *)(Vg + (size_t)d * a.n_keys + key0 + c * VE);
        }
      }
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < K_IT; ++i) {
      const int ch = tid + i * 256;
      if (ch < K_CH) *(V16 *)(Ks + ch * VE) = rk[i];
    }
#pragma unroll
    for (int i = 0; i < V_IT; ++i) {
      const int ch = tid + i * 256;
      if (ch < V_CH) {
        if (a.v_rowmajor) {  // transpose the chunk into the V^T tile
          const int key = ch / (D / VE), c = ch % (D / VE);
          const T *e = (const T *)&rv[i];
#pragma unroll
          for (int q = 0; q < VE; ++q) Vs[(c * VE + q) * VT_LD + key] = e[q];
        } else {
          const int d = ch / V_CPR, c = ch % V_CPR;
          *(V16 *)(Vs + d * VT_LD + c * VE) = rv[i];
        }
      }
    }
  };

  f32x16 o[3];
#pragma unroll
  for (int t = 0; t < 3; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;
  float sd[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) sd[j] = -INFINITY;

  load(kbeg);
  store();
  __syncthreads();
  for (int key0 = kbeg; key0 < kend; key0 += ATT_BK) {
    if (key0 + ATT_BK < kend) load(key0 + ATT_BK);

    f32x16 s[2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[st][e] = 0.0f;
      const T *krow = Ks + (st * 32 + key_perm(lane & 31)) * D;
#pragma unroll
      for (int c = 0; c < DC; ++c) {
        const int d0 = c * 2 * KS + g * KS;
        const frag kf = (d0 < D) ? *(const frag *)(krow + d0) : MF::zero();
        s[st] = MF::mma(kf, qf[c], s[st]);
      }
    }

    // scale into the log2 domain, mask padded keys, tile max per query
    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = key0 + st * 32 + g * 16 + e;
        float x = s[st][e] * a.scale_log2;
        if (key >= nv) x = -INFINITY;
        s[st][e] = x;
        tmax = fmaxf(tmax, x);
      }
    }
    if (EMIT) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (j < a.n_delta) {
          const int rel = a.delta[j] - key0;
          if (rel >= 0 && rel < ATT_BK && ((rel >> 4) & 1) == g) {
            const int st = rel >> 5, e = rel & 15;
#pragma unroll
            for (int ee = 0; ee < 16; ++ee)
              if (ee == e) sd[j] = st ? s[1][ee] : s[0][ee];
          }
        }
      }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    const float base = (m_new == -INFINITY) ? 0.0f : m_new;
    const float alpha = exp2f(m_run - base);
    m_run = m_new;
    float psum = 0.0f;
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = exp2f(s[st][e] - base);
        s[st][e] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[t][e] *= alpha;

    // O^T += V^T P^T
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int c = 0; c < PCH; ++c) {
        frag pf;
        if constexpr (KS == 1) {
          pf = s[st][c];
        } else {
#pragma unroll
          for (int k = 0; k < KS; ++k) pf[k] = from_f<T>(s[st][c * KS + k]);
        }
        const int kcol = st * 32 + g * 16 + c * KS;
#pragma unroll
        for (int t = 0; t < 3; ++t) {
          const int d = t * 32 + (lane & 31);
          const frag vf = (d < D) ? *(const frag *)(Vs + d * VT_LD + kcol) : MF::zero();
          o[t] = MF::mma(vf, pf, o[t]);
        }
      }
    }

    __syncthreads();
    if (key0 + ATT_BK < kend) {
      store();
      __syncthreads();
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (EMIT) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j < a.n_delta) {
        const int owner = ((a.delta[j] - kbeg) >> 4) & 1;
        float p = (g == owner) ? exp2f(sd[j] - m_run) / l_tot : 0.0f;
        p += __shfl_xor(p, 32, 64);
        if (g == 0 && q_ok) a.pmaps[((size_t)h * a.total_rows + my_q) * a.n_delta + j] = p;
      }
    }
  }
  if (!q_ok) return;
  if (a.splits == 1) {
    const float inv = 1.0f / l_tot;
    T *orow = (T *)a.O + (size_t)my_q * a.hidden + h * D;
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int d = t * 32 + (e >> 2) * 8 + g * 4 + (e & 3);
        if (d < D) orow[d] = from_f<T>(o[t][e] * inv);
      }
  } else {
    float *orow = a.Opart + ((size_t)split * a.total_rows + my_q) * a.hidden + h * D;
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int d = t * 32 + (e >> 2) * 8 + g * 4 + (e & 3);
        if (d < D) orow[d] = o[t][e];
      }
    if (g == 0) {
      float *ml = a.ML + (((size_t)split * a.total_rows + my_q) * heads + h) * 2;
      ml[0] = m_run;
      ml[1] = l_tot;
    }
  }
}

// Deterministic combine of key-split partials: O = sum_s 2^(m_s-M) o_s / sum_s
// 2^(m_s-M) l_s, in split order.  One thread per (row, head, 4 dims).
template <typename T> __device__ __forceinline__ void put4(T *p, const float *v);
template <> __device__ __forceinline__ void put4<float>(float *p, const float *v) {
  *(f32x4 *)p = f32x4{v[0], v[1], v[2], v[3]};
}
template <> __device__ __forceinline__ void put4<bf16>(bf16 *p, const float *v) {
  bf16x4 o;
  o[0] = (bf16)v[0]; o[1] = (bf16)v[1]; o[2] = (bf16)v[2]; o[3] = (bf16)v[3];
  *(bf16x4 *)p = o;
}

template <typename T>
__global__ void attn_combine_kernel(const float *Opart, const float *ML, T *O, int R, int heads, int splits) {
  constexpr int G = kHeadDim / 4;
  const int C = heads * kHeadDim;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)R * heads * G) return;
  const int r = idx / (heads * G);
  const int rem = idx - (long)r * heads * G;
  const int h = rem / G, d = (rem - h * G) * 4;
  // all loads are issued before any use (the split loops are unrolled to the
  // largest split count and predicated), so a thread waits on memory once
  constexpr int SMAX = 16;
  float2 ml[SMAX];
  f32x4 p[SMAX];
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < splits) {
      ml[s] = *(const float2 *)(ML + (((size_t)s * R + r) * heads + h) * 2);
      p[s] = *(const f32x4 *)(Opart + ((size_t)s * R + r) * C + h * kHeadDim + d);
    }
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < splits) M = fmaxf(M, ml[s].x);
  float num[4] = {0.0f, 0.0f, 0.0f, 0.0f}, den = 0.0f;
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
    if (s < splits) {
      const float w = exp2f(ml[s].x - M);
#pragma unroll
      for (int k = 0; k < 4; ++k) num[k] += w * p[s][k];
      den += w * ml[s].y;
    }
  const float inv = 1.0f / den;
  float v[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) v[k] = num[k] * inv;
  put4<T>(O + (size_t)r * C + h * kHeadDim + d, v);
}

// maps[chain][token][j] += sum over heads (fixed order) of the per-head
// probabilities of the delta columns.
__global__ void maps_reduce_kernel(const float *pmaps, const int *rows, float *maps, int R, int heads,
                                   int n_delta, int tokens) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= R * n_delta) return;
  const int r = idx / n_delta, j = idx - r * n_delta;
  float s = 0.0f;
  for (int h = 0; h < heads; ++h) s += pmaps[((size_t)h * R + r) * n_delta + j];
  const int pk = rows[r];
  maps[((size_t)row_chain(pk) * tokens + row_token(pk)) * n_delta + j] += s;
}

template <typename T>
hipError_t launch_attention(const AttnArgs &a, int n_chains, int max_rows, bool emit_maps, hipStream_t s) {
  if (max_rows <= 0) return hipSuccess;
  if (a.n_keys % ATT_BK != 0 || (a.n_keys / a.splits) % ATT_BK != 0) return hipErrorInvalidValue;
  dim3 grid((max_rows + ATT_BQ - 1) / ATT_BQ, (a.hidden / kHeadDim) * a.splits, n_chains);
  if (emit_maps)
    rc_launch(attn_kernel<T, true>, grid, dim3(256), 0, s, a);
  else
    rc_launch(attn_kernel<T, false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template hipError_t launch_attention<bf16>(const AttnArgs &, int, int, bool, hipStream_t);
template hipError_t launch_attention<float>(const AttnArgs &, int, int, bool, hipStream_t);

hipError_t launch_attn_combine(const float *Opart, const float *ML, void *O, bool bf16_out, int R,
                               int heads, int splits, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (splits < 1 || splits > 16) return hipErrorInvalidValue;
  const long n = (long)R * heads * (kHeadDim / 4);
  dim3 grid((n + 255) / 256);
  if (bf16_out)
    rc_launch(attn_combine_kernel<bf16>, grid, dim3(256), 0, s, Opart, ML, (bf16 *)O, R, heads, splits);
  else
    rc_launch(attn_combine_kernel<float>, grid, dim3(256), 0, s, Opart, ML, (float *)O, R, heads, splits);
  return hipGetLastError();
}

hipError_t launch_maps_reduce(const float *pmaps, const int *rows, float *maps, int R, int heads,
                              int n_delta, int tokens, hipStream_t s) {
  if (R <= 0 || n_delta <= 0) return hipSuccess;
  dim3 grid((R * n_delta + 255) / 256);
  rc_launch(maps_reduce_kernel, grid, dim3(256), 0, s, pmaps, rows, maps, R, heads, n_delta, tokens);
  return hipGetLastError();
}

}  // namespace rc
