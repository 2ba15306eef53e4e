// Edit-region localisation (Sec. 3.2): cross-attention maps of the delta text
// tokens aggregated over heads and blocks, a per-token-map threshold derived
// from each map's range, union over delta tokens, grid dilation, and the
// stable compaction of the resulting mask into per-chain token lists.
#include "rc_common.h"
#include "rc_launch.h"
#include "rc_elem.h"

namespace rc {

constexpr int LG_ROWS = 256;  // logits rows (tokens) per workgroup

// partial[l][tok][j] = sum_h softmax(Z[l][h][tok][:])[delta_j]; one workgroup
// per (256-token tile, layer); each head's 256 rows are one contiguous block
// of the logits, staged through LDS with 16-byte coalesced loads, then each
// thread reduces its own row.
__global__ __launch_bounds__(256) void maps_from_logits_kernel(const uint16_t *Z, int heads, int tokens,
                                                               int text_len, MapsDelta dl, float *partial) {
  extern __shared__ __attribute__((aligned(16))) uint16_t rowbuf[];
  const int l = blockIdx.y, tok0 = blockIdx.x * LG_ROWS, tid = threadIdx.x;
  const int nrows = min(LG_ROWS, tokens - tok0);
  const int row_vec = text_len / 8;                       // 16-byte vectors per row
  const int ld = (row_vec & 1) ? text_len : text_len + 8; // odd count of 16-byte slots per row
  float acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
  for (int h = 0; h < heads; ++h) {
    const uint16_t *src = Z + (((size_t)l * heads + h) * tokens + tok0) * text_len;
    const int nvec = nrows * row_vec;
    __syncthreads();
    for (int v = tid; v < nvec; v += 256) {
      const int r = v / row_vec, c = v - r * row_vec;
      *(V16 *)(rowbuf + r * ld + c * 8) = *(const V16 *)(src + (size_t)v * 8);
    }
    __syncthreads();
    if (tid < nrows) {
      const uint16_t *row = rowbuf + tid * ld;
      uint32_t w[64];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        V16 t = V16{{0u, 0u, 0u, 0u}};
        if (v < row_vec) t = *(const V16 *)(row + v * 8);
#pragma unroll
        for (int q = 0; q < 4; ++q) w[v * 4 + q] = t.w[q];
      }
      float m = -INFINITY;
#pragma unroll
      for (int k = 0; k < 128; ++k) {
        const float z = __uint_as_float((k & 1) ? (w[k >> 1] & 0xFFFF0000u) : (w[k >> 1] << 16));
        if (k < text_len) m = fmaxf(m, z);
      }
      float s = 0.0f;
#pragma unroll
      for (int k = 0; k < 128; ++k) {
        const float z = __uint_as_float((k & 1) ? (w[k >> 1] & 0xFFFF0000u) : (w[k >> 1] << 16));
        if (k < text_len) s += __expf(z - m);
      }
      const float inv = 1.0f / s;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j < dl.n) acc[j] += __expf(__uint_as_float((uint32_t)row[dl.col[j]] << 16) - m) * inv;
    }
  }
  if (tid < nrows) {
    for (int j = 0; j < dl.n; ++j) partial[((size_t)l * tokens + tok0 + tid) * dl.n + j] = acc[j];
  }
}

hipError_t launch_maps_from_logits(const uint16_t *logits, int n_layers, int heads, int tokens, int text_len,
                                   const int *delta, int n_delta, float *partial, hipStream_t s) {
  MapsDelta dl;
  dl.n = n_delta;
  for (int j = 0; j < 8; ++j) dl.col[j] = j < n_delta ? delta[j] : 0;
  dim3 grid((tokens + LG_ROWS - 1) / LG_ROWS, n_layers);
  const int ld = ((text_len / 8) & 1) ? text_len : text_len + 8;
  const size_t lds = (size_t)LG_ROWS * ld * sizeof(uint16_t);
  rc_launch(maps_from_logits_kernel, grid, dim3(256), lds, s, logits, heads, tokens, text_len, dl, partial);
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

hipError_t launch_compact(const uint8_t *mask, int B, int N, int *idx, int *offsets, hipStream_t s) {
  rc_launch(compact_kernel, dim3(1), dim3(1024), 0, s, mask, B, N, idx, offsets);
  return hipGetLastError();
}

}  // namespace rc
