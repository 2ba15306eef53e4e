// Edit-region localisation (Sec. 3.2): cross-attention maps of the delta text
// tokens aggregated over heads and blocks, a per-token-map threshold derived
// from each map's range, union over delta tokens, grid dilation, and the
// stable compaction of the resulting mask into per-chain token lists.
#include "rc_common.h"
#include "rc_launch.h"
#include "rc_elem.h"

#include <climits>

namespace rc {

constexpr int LG_TOK = 16;  // tokens per workgroup, 4 per wave
constexpr int LG_HC = 4;    // heads whose rows a wave loads at once

// Max over the 16 lanes of a DPP row (the steps of row16_sum).
// IEEE maximum (NaN-propagating): one v_maximum3/v_maximum on gfx950, with
// no operand canonicalisation as fmaxf needs.
__device__ __forceinline__ float fmax_(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float row16_max(float v) {
  v = fmax_(v, dpp_mov<0xB1>(v));   // quad_perm [1,0,3,2]
  v = fmax_(v, dpp_mov<0x4E>(v));   // quad_perm [2,3,0,1]
  v = fmax_(v, dpp_mov<0x141>(v));  // row_half_mirror
  return fmax_(v, dpp_mov<0x140>(v));  // row_mirror
}

// partial[l][tok][j] = sum_h softmax(Z[l][h][tok][:])[delta_j].  One
// workgroup per (16-token tile, layer), each wave 4 tokens.  A row of the
// logits (text_len <= 128 bf16, 16-byte chunks) is spread over one 16-lane
// group (one token per group), so one load instruction covers four
// consecutive rows -- contiguous memory -- and the row's max and sum are
// 16-lane DPP reductions.  A wave issues the rows of LG_HC heads before it
// reduces any (4 KB in flight per wave at 40 VGPRs, eight waves per SIMD).
// The exponent runs on the raw v_exp_f32: its argument z - max is <= 0, so a
// flushed denormal moves a row sum that is >= 1 by less than 2^-126, and the
// row's reciprocal is one v_rcp_f32 (1 ulp).  Lane j of a group owns delta
// column j: it re-reads that one logit (a cache hit) and accumulates its
// probability over the heads in order.
__global__ __launch_bounds__(256) void maps_from_logits_kernel(const uint16_t *Z, int heads, int tokens,
                                                               int text_len, MapsDelta dl, float *partial) {
  const int l = blockIdx.y, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int grp = lane >> 4, j16 = lane & 15;
  const int tok = blockIdx.x * LG_TOK + wave * 4 + grp;  // this lane group's token
  const int row_vec = text_len / 8;                       // 16-byte chunks per row
  const bool ok = tok < tokens;
  const bool lane_on = j16 < row_vec && ok;
  const bool owner = j16 < dl.n && ok;
  int my_col = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if (j == j16) my_col = dl.col[j];
  constexpr float kLog2e = 1.4426950408889634f;
  float acc = 0.0f;
  for (int h0 = 0; h0 < heads; h0 += LG_HC) {
    V16 v[LG_HC];
    uint16_t zd[LG_HC];
#pragma unroll
    for (int c = 0; c < LG_HC; ++c) {
      const uint16_t *row = Z + ((size_t)(l * heads + h0 + c) * tokens + tok) * text_len;
      const bool on = h0 + c < heads;
      v[c] = V16{{0u, 0u, 0u, 0u}};
      if (on && lane_on) v[c] = *(const V16 *)(row + j16 * 8);
      zd[c] = (on && owner) ? row[my_col] : (uint16_t)0;
    }
#pragma unroll
    for (int c = 0; c < LG_HC; ++c) {
      const bool on = h0 + c < heads;
      float z[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        z[2 * q] = __uint_as_float(v[c].w[q] << 16);
        z[2 * q + 1] = __uint_as_float(v[c].w[q] & 0xFFFF0000u);
      }
      float m = -INFINITY;
      if (on && lane_on)
        m = fmax_(fmax_(fmax_(z[0], z[1]), fmax_(z[2], z[3])), fmax_(fmax_(z[4], z[5]), fmax_(z[6], z[7])));
      m = row16_max(m);
      const float mc = m * kLog2e;
      float sum = 0.0f;
      if (on && lane_on)
#pragma unroll
        for (int q = 0; q < 8; ++q) sum += __builtin_amdgcn_exp2f(__builtin_fmaf(z[q], kLog2e, -mc));
      sum = row16_sum(sum);
      if (on && owner)
        acc += __builtin_amdgcn_exp2f(__builtin_fmaf(__uint_as_float((uint32_t)zd[c] << 16), kLog2e, -mc)) *
               __builtin_amdgcn_rcpf(sum);
    }
  }
  if (owner) partial[((size_t)l * tokens + tok) * dl.n + j16] = acc;
}

hipError_t launch_maps_from_logits(const uint16_t *logits, int n_layers, int heads, int tokens, int text_len,
                                   const int *delta, int n_delta, float *partial, hipStream_t s) {
  if (text_len % 8 || text_len > 128 || n_delta < 1 || n_delta > 8) return hipErrorInvalidValue;
  MapsDelta dl;
  dl.n = n_delta;
  for (int j = 0; j < 8; ++j) dl.col[j] = j < n_delta ? delta[j] : 0;
  dim3 grid((tokens + LG_TOK - 1) / LG_TOK, n_layers);
  rc_launch(maps_from_logits_kernel, grid, dim3(256), 0, s, logits, heads, tokens, text_len, dl, partial);
  return hipGetLastError();
}

// out[i] = sum_p partial[p][i] in order p = 0, 1, ...
__global__ void sum_partials_kernel(const float *partial, int n_parts, int n, float *out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = 0.0f;
  for (int p = 0; p < n_parts; ++p) s += partial[(size_t)p * n + i];
  out[i] = s;
}

hipError_t launch_sum_partials(const float *partial, int n_parts, int n, float *out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  rc_launch(sum_partials_kernel, dim3((n + 255) / 256), dim3(256), 0, s, partial, n_parts, n, out);
  return hipGetLastError();
}

// One workgroup per chain: range of each delta map, threshold, union, dilation.
__global__ __launch_bounds__(1024) void localize_kernel(const float *maps, int gh, int gw, int n_delta,
                                                        float threshold, int radius, uint8_t *mask) {
  extern __shared__ uint8_t sel[];
  __shared__ float red_lo[16], red_hi[16];
  const int b = blockIdx.x, tid = threadIdx.x, N = gh * gw;
  const int lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const float *m = maps + (size_t)b * N * n_delta;
  for (int i = tid; i < N; i += blockDim.x) sel[i] = 0;
  for (int j = 0; j < n_delta; ++j) {
    float lo = INFINITY, hi = -INFINITY;
    for (int i = tid; i < N; i += blockDim.x) {
      const float v = m[(size_t)i * n_delta + j];
      lo = fminf(lo, v);
      hi = fmaxf(hi, v);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      lo = fminf(lo, __shfl_xor(lo, o, 64));
      hi = fmaxf(hi, __shfl_xor(hi, o, 64));
    }
    __syncthreads();
    if (lane == 0) {
      red_lo[wave] = lo;
      red_hi[wave] = hi;
    }
    __syncthreads();
    lo = red_lo[0];
    hi = red_hi[0];
    for (int w = 1; w < nw; ++w) {
      lo = fminf(lo, red_lo[w]);
      hi = fmaxf(hi, red_hi[w]);
    }
    if (hi > lo) {
      const float inv = 1.0f / (hi - lo);
      for (int i = tid; i < N; i += blockDim.x)
        if ((m[(size_t)i * n_delta + j] - lo) * inv >= threshold) sel[i] = 1;
    }
  }
  __syncthreads();
  for (int i = tid; i < N; i += blockDim.x) {
    const int y = i / gw, x = i - (i / gw) * gw;
    uint8_t on = 0;
    for (int dy = -radius; dy <= radius && !on; ++dy) {
      const int yy = y + dy;
      if (yy < 0 || yy >= gh) continue;
      for (int dx = -radius; dx <= radius; ++dx) {
        const int xx = x + dx;
        if (xx >= 0 && xx < gw && sel[yy * gw + xx]) {
          on = 1;
          break;
        }
      }
    }
    mask[(size_t)b * N + i] = on;
  }
}

hipError_t launch_localize(const float *maps, int B, int gh, int gw, int n_delta, float threshold, int radius,
                           uint8_t *mask, hipStream_t s) {
  rc_launch(localize_kernel, dim3(B), dim3(1024), (size_t)gh * gw, s, maps, gh, gw, n_delta, threshold,
                     radius, mask);
  return hipGetLastError();
}

// Single-workgroup stable compaction over all chains: per 1024-token chunk a
// ballot/popcount prefix within each wave plus an LDS prefix over waves.
__global__ __launch_bounds__(1024) void compact_kernel(const uint8_t *mask, int B, int N, int *idx, int *offsets) {
  __shared__ int wave_tot[16];
  __shared__ int wave_pre[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int base = 0;
  for (int b = 0; b < B; ++b) {
    if (tid == 0) offsets[b] = base;
    for (int i0 = 0; i0 < N; i0 += 1024) {
      const int i = i0 + tid;
      const bool on = i < N && mask[(size_t)b * N + i] != 0;
      const uint64_t bal = __ballot(on);
      const int within = __popcll(bal & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
      if (lane == 0) wave_tot[wave] = __popcll(bal);
      __syncthreads();
      if (tid == 0) {
        int acc = 0;
        for (int w = 0; w < 16; ++w) {
          wave_pre[w] = acc;
          acc += wave_tot[w];
        }
        wave_tot[0] = acc;  // chunk total
      }
      __syncthreads();
      if (on) idx[base + wave_pre[wave] + within] = i;
      base += wave_tot[0];
      __syncthreads();
    }
  }
  if (tid == 0) offsets[B] = base;
}

// Validity of an active set (device offsets already checked equal to the
// host copy, so every chain's range lies inside idx[0, total)): the first
// position p, in index order, whose token is outside [0, N) or not larger
// than the token before it in the same chain; -1 if there is none.  One
// workgroup; each thread keeps its smallest bad position, then a fixed-order
// reduction; thread 0 writes the verdict.
__global__ __launch_bounds__(1024) void validate_active_kernel(const int *offsets, const int *idx, int B, int N,
                                                               int *verdict) {
  __shared__ int red[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int bad = INT_MAX;
  for (int b = 0; b < B; ++b) {
    const int lo = offsets[b], hi = offsets[b + 1];
    for (int i = lo + tid; i < hi; i += 1024) {
      const int v = idx[i];
      const bool ok = v >= 0 && v < N && (i == lo || idx[i - 1] < v);
      if (!ok) bad = min(bad, i);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) bad = min(bad, __shfl_xor(bad, o, 64));
  if (lane == 0) red[wave] = bad;
  __syncthreads();
  if (tid == 0) {
    int m = red[0];
    for (int w = 1; w < 16; ++w) m = min(m, red[w]);
    verdict[0] = m == INT_MAX ? -1 : m;
  }
}

hipError_t launch_validate_active(const int *offsets, const int *idx, int B, int N, int *verdict, hipStream_t s) {
  rc_launch(validate_active_kernel, dim3(1), dim3(1024), 0, s, offsets, idx, B, N, verdict);
  return hipGetLastError();
}

hipError_t launch_compact(const uint8_t *mask, int B, int N, int *idx, int *offsets, hipStream_t s) {
  rc_launch(compact_kernel, dim3(1), dim3(1024), 0, s, mask, B, N, idx, offsets);
  return hipGetLastError();
}

}  // namespace rc
