// Row-wise and elementwise kernels of the step: active-row bookkeeping,
// token gather + patch embedding, adaLN LayerNorm-modulate, timestep
// conditioning GEMVs, the final layer fused with the DDIM update, and the
// cache copies of the reuse path.
#include "rc_common.h"
#include "rc_launch.h"
#include "rc_elem.h"

namespace rc {

// rows[r] = (chain << 16) | token for r in [0, R); idx == null means the
// dense identity set (token = r - offsets[chain]).
__global__ void build_rows_kernel(const int *offsets, const int *idx, int B, int R, int *rows) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= R) return;
  int b = 0;
  while (b + 1 < B && offsets[b + 1] <= r) ++b;
  const int tok = idx ? idx[r] : r - offsets[b];
  rows[r] = (b << 16) | tok;
}

hipError_t launch_build_rows(const int *offsets, const int *idx, int B, int R, int *rows, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  rc_launch(build_rows_kernel, dim3((R + 255) / 256), dim3(256), 0, s, offsets, idx, B, R, rows);
  return hipGetLastError();
}

// Dense-step offsets: offsets[b] = b*N for b = 0..B (B+1 entries, any B).
__global__ void dense_offsets_kernel(int *offsets, int B, int N) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b <= B) offsets[b] = b * N;
}

hipError_t launch_dense_offsets(int *offsets, int B, int N, hipStream_t s) {
  rc_launch(dense_offsets_kernel, dim3((B + 1 + 255) / 256), dim3(256), 0, s, offsets, B, N);
  return hipGetLastError();
}

// X[r][:] = patch(token) . W_pe^T + b_pe + pos(token), or in token mode the
// gathered hidden row.  One workgroup per row.
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs a) {
  const int r = blockIdx.x;
  const int pk = a.rows[r];
  const int b = row_chain(pk), tok = row_token(pk);
  float *xrow = a.X + (size_t)r * a.C;
  if (a.tokens_in) {
    const T *src = (const T *)a.tokens_in + ((size_t)b * a.N + tok) * a.C;
    for (int n = threadIdx.x; n < a.C; n += 256) xrow[n] = to_f<T>(src[n]);
    return;
  }
  __shared__ float patch[16];
  const int y = tok / a.gw, x = tok - (tok / a.gw) * a.gw;
  if (threadIdx.x < 16) {
    const int c = threadIdx.x >> 2, pi = (threadIdx.x >> 1) & 1, qi = threadIdx.x & 1;
    const int Hl = a.gh * 2, Wl = a.gw * 2;
    patch[threadIdx.x] = a.latent[(((size_t)b * 4 + c) * Hl + 2 * y + pi) * Wl + 2 * x + qi];
  }
  __syncthreads();
  const T *W = (const T *)a.pe_w;
  const int half = a.C / 2, quarter = a.C / 4;
  const float log2_10000 = 13.287712379549449f;
  for (int n = threadIdx.x; n < a.C; n += 256) {
    float acc = a.pe_b[n];
#pragma unroll
    for (int k = 0; k < 16; ++k) acc += to_f<T>(W[n * 16 + k]) * patch[k];
    const int coord = n < half ? x : y;
    const int kk = n % half;
    const int f = kk % quarter;
    const float w = exp2f(-(float)f / (float)quarter * log2_10000);
    const float arg = (float)coord * w;
    acc += kk < quarter ? sinf(arg) : cosf(arg);
    xrow[n] = acc;
  }
}

template <typename T> hipError_t launch_embed(const EmbedArgs &a, int R, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  rc_launch(embed_kernel<T>, dim3(R), dim3(256), 0, s, a);
  return hipGetLastError();
}
template hipError_t launch_embed<bf16>(const EmbedArgs &, int, hipStream_t);
template hipError_t launch_embed<float>(const EmbedArgs &, int, hipStream_t);

// out[r][:] = E( LN(X[r]) * (1 + scale) + shift ), scale/shift = table row + t0
// row.  One wave per row, 16-byte accesses; statistics in fp32 with a
// two-pass variance over the values held in registers.
template <typename T> __device__ __forceinline__ void store4(T *p, float a, float b, float c, float d);
template <> __device__ __forceinline__ void store4<float>(float *p, float a, float b, float c, float d) {
  *(f32x4 *)p = f32x4{a, b, c, d};
}
template <> __device__ __forceinline__ void store4<bf16>(bf16 *p, float a, float b, float c, float d) {
  bf16x4 v;
  v[0] = (bf16)a; v[1] = (bf16)b; v[2] = (bf16)c; v[3] = (bf16)d;
  *(bf16x4 *)p = v;
}

template <typename T>
__global__ __launch_bounds__(256) void ln_mod_kernel(const float *X, int R, int C, const float *table,
                                                     const float *t0, int shift_row, float eps, T *out) {
  __shared__ float red[4];
  const int r = blockIdx.x, t = threadIdx.x;  // one 256-thread workgroup per row
  constexpr int MAXV = 2;                      // C <= 4 * 256 * MAXV
  const int C4 = C >> 2;
  const f32x4 *x = (const f32x4 *)(X + (size_t)r * C);
  const f32x4 *sh = (const f32x4 *)(table + (size_t)shift_row * C), *sc = (const f32x4 *)(table + (size_t)(shift_row + 1) * C);
  const f32x4 *tsh = (const f32x4 *)(t0 + (size_t)shift_row * C), *tsc = (const f32x4 *)(t0 + (size_t)(shift_row + 1) * C);
  // the row and its modulation rows are loaded together (one memory round trip)
  f32x4 v[MAXV], shift[MAXV], scale[MAXV];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int n = t + i * 256;
    const f32x4 z = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    v[i] = n < C4 ? x[n] : z;
    shift[i] = n < C4 ? sh[n] + tsh[n] : z;
    scale[i] = n < C4 ? sc[n] + tsc[n] : z;
    s += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
  }
  const float mean = block4_sum(s, red) / C;
  float q = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int n = t + i * 256;
    if (n < C4)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float d = v[i][k] - mean;
        q += d * d;
      }
  }
  const float rstd = rsqrtf(block4_sum(q, red) / C + eps);
  T *o = out + (size_t)r * C;
#pragma unroll
  for (int i = 0; i < MAXV; ++i) {
    const int n = t + i * 256;
    if (n < C4) {
      float y[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) y[k] = (v[i][k] - mean) * rstd * (1.0f + scale[i][k]) + shift[i][k];
      store4<T>(o + 4 * n, y[0], y[1], y[2], y[3]);
    }
  }
}

template <typename T>
hipError_t launch_ln_mod(const float *X, int R, int C, const float *table, const float *t0, int shift_row,
                         float eps, void *out, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (C > 4 * 256 * 2 || C % 4) return hipErrorInvalidValue;
  rc_launch(ln_mod_kernel<T>, dim3(R), dim3(256), 0, s, X, R, C, table, t0, shift_row, eps,
                     (T *)out);
  return hipGetLastError();
}
template hipError_t launch_ln_mod<bf16>(const float *, int, int, const float *, const float *, int, float, void *, hipStream_t);
template hipError_t launch_ln_mod<float>(const float *, int, int, const float *, const float *, int, float, void *, hipStream_t);

// Timestep features e(t) = [cos(t f_k), sin(t f_k)], f_k = 10000^(-k/128).
__global__ void timestep_features_kernel(float t, float *e) {
  const int k = threadIdx.x;
  if (k >= 128) return;
  const float f = exp2f(-(float)k / 128.0f * 13.287712379549449f);
  const float arg = t * f;
  e[k] = cosf(arg);
  e[128 + k] = sinf(arg);
}

hipError_t launch_timestep_features(float t, float *e, hipStream_t s) {
  rc_launch(timestep_features_kernel, dim3(1), dim3(128), 0, s, t, e);
  return hipGetLastError();
}

// y[n] = act_out( W[n] . act_in(x) + b[n] ), one wave per output.
// 8 consecutive inputs of one row as floats (16-byte loads).
template <typename T> __device__ __forceinline__ void load8(const T *p, float *v);
template <> __device__ __forceinline__ void load8<float>(const float *p, float *v) {
  const f32x4 a = *(const f32x4 *)p, b = *(const f32x4 *)(p + 4);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    v[q] = a[q];
    v[4 + q] = b[q];
  }
}
template <> __device__ __forceinline__ void load8<bf16>(const bf16 *p, float *v) {
  const bf16x8 a = *(const bf16x8 *)p;
#pragma unroll
  for (int q = 0; q < 8; ++q) v[q] = (float)a[q];
}

// y[n] = act(W[n] . act_in(x) + b[n]); one wave per output, each lane takes
// 8 consecutive inputs per pass (K % 8 == 0, K <= 1536), every load first.
template <typename T>
__global__ __launch_bounds__(256) void gemv_kernel(const T *W, const float *bias, const float *x, int N, int K,
                                                   int silu_in, int silu_out, float *y) {
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= N) return;
  const T *w = W + (size_t)n * K;
  constexpr int MAXC = 3;
  float wv[MAXC][8], xv[MAXC][8];
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int k0 = 8 * (lane + 64 * i);
    if (k0 < K) {
      load8<T>(w + k0, wv[i]);
      load8<float>(x + k0, xv[i]);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) wv[i][q] = xv[i][q] = 0.0f;
    }
  }
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc += wv[i][q] * (silu_in ? silu(xv[i][q]) : xv[i][q]);
  acc = wave_sum(acc);
  if (lane == 0) {
    float v = acc + (bias ? bias[n] : 0.0f);
    y[n] = silu_out ? silu(v) : v;
  }
}

template <typename T>
hipError_t launch_gemv(const void *W, const float *bias, const float *x, int N, int K, int silu_in, int silu_out,
                       float *y, hipStream_t s) {
  if (K % 8 || K > 64 * 8 * 3) return hipErrorInvalidValue;
  rc_launch(gemv_kernel<T>, dim3((N + 3) / 4), dim3(256), 0, s, (const T *)W, bias, x, N, K, silu_in,
                     silu_out, y);
  return hipGetLastError();
}
template hipError_t launch_gemv<bf16>(const void *, const float *, const float *, int, int, int, int, float *, hipStream_t);
template hipError_t launch_gemv<float>(const void *, const float *, const float *, int, int, int, int, float *, hipStream_t);

// Final layer + DDIM for each computed row: eps = (LN(X)(1+sc)+sh) W_f^T + b_f
// for the noise channels of the 2x2 patch, then x' = ca * x + cb * eps written
// to the output latent and (if given) to the cached trajectory entry.  A
// workgroup stages the 16 noise rows of W_f in LDS once and serves 8 rows
// (two per wave); each output is a wave-wide dot product.
constexpr int FIN_ROWS = 4;  // one row per wave

template <typename T>
__global__ __launch_bounds__(256) void final_ddim_kernel(FinalArgs a) {
  extern __shared__ __attribute__((aligned(16))) char fin_lds[];
  T *wl = (T *)fin_lds;  // [16][C]: output o = pix*4 + c is W_f row pix*out_ch + c
  const int C = a.C, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const T *W = (const T *)a.fin_w;
  {
    constexpr int EPC = 16 / sizeof(T);  // elements per 16-byte chunk
    const int cpr = C / EPC;
    for (int i = threadIdx.x; i < 16 * cpr; i += 256) {
      const int o = i / cpr, j = i - o * cpr;
      *(V16 *)(wl + (size_t)o * C + j * EPC) = *(const V16 *)(W + (size_t)((o >> 2) * a.out_ch + (o & 3)) * C + j * EPC);
    }
  }
  __syncthreads();
  const int r = blockIdx.x * FIN_ROWS + wave;
  if (r >= a.R) return;
  // guided: the wave of a conditional row also takes the unconditional row
  // of the same token (same position in the paired chain); waves of
  // unconditional rows have nothing to do
  int r_u = -1;
  if (a.guided) {
    const int b = row_chain(a.rows[r]);
    if (b & 1) return;
    r_u = r + (a.offsets[b + 1] - a.offsets[b]);
  }
  float eps[16];
  auto noise = [&](int row, float *e16) {
    // lane chunk i holds inputs 8*(lane + 64 i) .. +8 (C % 8 == 0, C <= 1536)
    constexpr int MAXC = 3;
    const float *x = a.X + (size_t)row * C;
    float v[MAXC][8], sh[MAXC][8], sc[MAXC][8];
    float s = 0.0f;
  #pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      const int k0 = 8 * (lane + 64 * i);
      if (k0 < C) {
        float t0[8];
        load8<float>(x + k0, v[i]);
        load8<float>(a.fin_sst + k0, sh[i]);
        load8<float>(a.fin_sst + C + k0, sc[i]);
        load8<float>(a.t_emb + k0, t0);
  #pragma unroll
        for (int q = 0; q < 8; ++q) {
          sh[i][q] += t0[q];
          sc[i][q] += t0[q];
        }
      } else {
  #pragma unroll
        for (int q = 0; q < 8; ++q) v[i][q] = sh[i][q] = sc[i][q] = 0.0f;
      }
  #pragma unroll
      for (int q = 0; q < 8; ++q) s += v[i][q];
    }
    const float mean = wave_sum(s) / C;
    float qs = 0.0f;
  #pragma unroll
    for (int i = 0; i < MAXC; ++i)
      if (8 * (lane + 64 * i) < C)
  #pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float d = v[i][q] - mean;
          qs += d * d;
        }
    const float rstd = rsqrtf(wave_sum(qs) / C + a.eps);
  #pragma unroll
    for (int i = 0; i < MAXC; ++i)
  #pragma unroll
      for (int q = 0; q < 8; ++q) v[i][q] = (v[i][q] - mean) * rstd * (1.0f + sc[i][q]) + sh[i][q];
  #pragma unroll
    for (int o = 0; o < 16; ++o) {
      float acc = 0.0f;
  #pragma unroll
      for (int i = 0; i < MAXC; ++i) {
        const int k0 = 8 * (lane + 64 * i);
        if (k0 < C) {
          float wv[8];
          load8<T>(wl + (size_t)o * C + k0, wv);
  #pragma unroll
          for (int q = 0; q < 8; ++q) acc += v[i][q] * wv[q];
        }
      }
      e16[o] = wave_sum(acc);
    }
  };
  noise(r, eps);
  if (r_u >= 0) {
    float eu[16];
    noise(r_u, eu);
#pragma unroll
    for (int o = 0; o < 16; ++o) eps[o] = eu[o] + a.gscale * (eps[o] - eu[o]);
  }
  if (lane < 16) {
    const int o = lane, pix = o >> 2, c = o & 3, pi = pix >> 1, qi = pix & 1;
    float e = 0.0f;
#pragma unroll
    for (int k = 0; k < 16; ++k)
      if (k == o) e = eps[k];
    e += a.fin_b[pix * a.out_ch + c];
    const int pk = a.rows[r];
    const int b = row_chain(pk), tok = row_token(pk);
    const int y = tok / a.gw, xx = tok - y * a.gw;
    const int Hl = a.gh * 2, Wl = a.gw * 2;
    const size_t li = (((size_t)b * 4 + c) * Hl + 2 * y + pi) * Wl + 2 * xx + qi;
    const float xn = a.ca * a.latent_in[li] + a.cb * e;
    a.latent_out[li] = xn;
    if (a.traj_next) a.traj_next[b * a.traj_chain_stride + (li - (size_t)b * 4 * Hl * Wl)] = xn;
    if (r_u >= 0) {  // the unconditional chain of the pair gets the same update
      const size_t lu = li + (size_t)4 * Hl * Wl;
      a.latent_out[lu] = xn;
      if (a.traj_next) a.traj_next[(b + 1) * a.traj_chain_stride + (li - (size_t)b * 4 * Hl * Wl)] = xn;
    }
  }
}

template <typename T> hipError_t launch_final_ddim(const FinalArgs &a, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  if (a.C % 8 || a.C > 64 * 8 * 3 || a.out_ch < 4) return hipErrorInvalidValue;
  const size_t lds = (size_t)16 * a.C * sizeof(T);
  rc_launch(final_ddim_kernel<T>, dim3((a.R + FIN_ROWS - 1) / FIN_ROWS), dim3(256), lds, s, a);
  return hipGetLastError();
}
template hipError_t launch_final_ddim<bf16>(const FinalArgs &, hipStream_t);
template hipError_t launch_final_ddim<float>(const FinalArgs &, hipStream_t);

// Strided float copy of per-chain latents: dst[b] = src[b] (n floats each).
__global__ void copy_chains_kernel(float *dst, long long dst_stride, const float *src, long long src_stride, int n,
                                   int B) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)n * B) return;
  const int b = i / n, k = i - (long)b * n;
  dst[b * dst_stride + k] = src[b * src_stride + k];
}

hipError_t launch_copy_chains(float *dst, long long dst_stride, const float *src, long long src_stride, int n, int B,
                              hipStream_t s) {
  const long tot = (long)n * B;
  if (tot <= 0) return hipSuccess;
  rc_launch(copy_chains_kernel, dim3((tot + 255) / 256), dim3(256), 0, s, dst, dst_stride, src, src_stride,
                     n, B);
  return hipGetLastError();
}

// Write-back of the rows a step computed from a device staging slot to the
// same rows of a cache slot (the host-resident pool of the pipelined step):
// for every packed row (chain << 16 | token), the token's key and value rows
// of every head and its hidden-state row, in 16-byte vectors.  Consecutive
// threads walk consecutive vectors of one row, so each hidden row is one
// contiguous write and each key/value head row nine.  A grid-stride loop
// keeps the workgroup count small: the copy runs beside the next block.
__global__ __launch_bounds__(256) void writeback_rows_kernel(const int *rows, int R, const V16 *stage,
                                                             long long stage_chain_vec, V16 *dst,
                                                             long long dst_chain_vec, int heads, int tokens,
                                                             int hidden_vec) {
  constexpr int HV = kHeadDim * 2 / 16;  // 16-byte vectors per head row of 72 bf16
  const int kv_vec = heads * HV;         // key (or value) vectors of one token
  const int per_row = 2 * kv_vec + hidden_vec;
  const long long half = (long long)heads * tokens * HV;  // vectors of the K (or V) array of one slot
  const long total = (long)R * per_row;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < total; i += (long)gridDim.x * 256) {
    const int r = (int)(i / per_row), v = (int)(i - (long)r * per_row);
    const int pk = rows[r];
    const long long cs = (long long)row_chain(pk), tok = row_token(pk);
    long long off;
    if (v < 2 * kv_vec) {
      const int part = v / kv_vec, w = v - part * kv_vec, h = w / HV, e = w - h * HV;
      off = part * half + ((long long)h * tokens + tok) * HV + e;
    } else {
      off = 2 * half + tok * hidden_vec + (v - 2 * kv_vec);
    }
    dst[cs * dst_chain_vec + off] = stage[cs * stage_chain_vec + off];
  }
}

hipError_t launch_writeback_rows(const int *rows, int R, const void *stage, long long stage_chain_bytes, void *dst,
                                 long long dst_chain_bytes, int heads, int tokens, int hidden_bytes, bool bf16_elems,
                                 int workgroups, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (!bf16_elems || hidden_bytes % 16 || stage_chain_bytes % 16 || dst_chain_bytes % 16 || workgroups < 1)
    return hipErrorInvalidValue;
  rc_launch(writeback_rows_kernel, dim3(workgroups), dim3(256), 0, s, rows, R, (const V16 *)stage,
            stage_chain_bytes / 16, (V16 *)dst, dst_chain_bytes / 16, heads, tokens, hidden_bytes / 16);
  return hipGetLastError();
}

// H slot scatter: hslot(chain)[token][:] = src[r][:] for every active row,
// 16-byte vectors; the chain of row r is found from the offsets.
__global__ void scatter_rows_kernel(const int *offsets, const int *idx, int B, const V16 *src, int R,
                                    int vec_per_row, V16 *hslot, long long chain_stride_vec) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)R * vec_per_row) return;
  const int r = i / vec_per_row, c = i - (long)r * vec_per_row;
  int b = 0;
  while (b + 1 < B && offsets[b + 1] <= r) ++b;
  hslot[b * chain_stride_vec + (long)idx[r] * vec_per_row + c] = src[i];
}

hipError_t launch_scatter_rows(const int *offsets, const int *idx, int B, const void *src, int R, int row_bytes,
                               void *hslot, long long chain_stride_bytes, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  const int vpr = row_bytes / 16;
  const long tot = (long)R * vpr;
  rc_launch(scatter_rows_kernel, dim3((tot + 255) / 256), dim3(256), 0, s, offsets, idx, B,
                     (const V16 *)src, R, vpr, (V16 *)hslot, chain_stride_bytes / 16);
  return hipGetLastError();
}

// Zero-fill with a kernel (no memset nodes in captured graphs).
__global__ void zero_kernel(V16 *p, long n) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = V16{{0u, 0u, 0u, 0u}};
}

hipError_t launch_zero(void *p, size_t bytes, hipStream_t s) {
  const long n = bytes / 16;
  if (n <= 0) return hipSuccess;
  rc_launch(zero_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (V16 *)p, n);
  return hipGetLastError();
}

}  // namespace rc
