// Matrix-core GEMM over ragged active-row sets: Y[M][N] = A[M][K] . W[N][K]^T
// with fused epilogues.  The QKV epilogue writes fresh active keys and values
// straight to their token positions in the cache slot (the fusion of
// Sec. 3.4, "Kernel Fusing"), and the residual epilogue can scatter the
// merged hidden state into the cached H (Sec. 3.3 merge).
//
// Tiling: 256 threads = 4 waves arranged 2x2; a BMxBN tile with a K step of
// 128 bytes per row (64 bf16 or 32 f32).  Each wave owns a (BM/2)x(BN/2)
// sub-tile made of 32x32 MFMA blocks.  Operands go global -> registers ->
// LDS (rows padded by 16 bytes) with the next K step's global loads issued
// before the current step's MFMAs.
#include "rc_common.h"
#include "rc_launch.h"
#include "rc_internal.h"

namespace rc {

template <typename T, int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
  constexpr int VE = 16 / sizeof(T);      // elements per 16-byte chunk
  constexpr int KT = 128 / sizeof(T);     // K step in elements
  constexpr int LDS_LD = KT + VE;         // padded LDS row (elements)
  constexpr int CPR = KT / VE;            // 16-byte chunks per tile row (8)
  constexpr int A_CH = BM * CPR / 256;    // chunks per thread
  constexpr int B_CH = BN * CPR / 256;
  constexpr int WM = BM / 2, WN = BN / 2; // wave sub-tile
  constexpr int FM = WM / 32, FN = WN / 32;
  constexpr int KS = Mfma<T>::KS;
  typedef typename Mfma<T>::frag frag;

  __shared__ __attribute__((aligned(16))) T As[BM * LDS_LD];
  __shared__ __attribute__((aligned(16))) T Bs[BN * LDS_LD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const T *A = (const T *)g.A;
  const T *W = (const T *)g.W;

  V16 ra[A_CH], rb[B_CH];
  auto load = [&](int k0) {
#pragma unroll
    for (int c = 0; c < A_CH; ++c) {
      int ch = tid + c * 256, r = ch / CPR, col = (ch % CPR) * VE;
      int gr = m0 + r;
      if (gr < g.M) ra[c] = *(const V16 *)(A + (size_t)gr * g.lda + k0 + col);
      else ra[c] = V16{{0u, 0u, 0u, 0u}};
    }
#pragma unroll
    for (int c = 0; c < B_CH; ++c) {
      int ch = tid + c * 256, r = ch / CPR, col = (ch % CPR) * VE;
      rb[c] = *(const V16 *)(W + (size_t)(n0 + r) * g.K + k0 + col);
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int c = 0; c < A_CH; ++c) {
      int ch = tid + c * 256, r = ch / CPR, col = (ch % CPR) * VE;
      *(V16 *)(As + r * LDS_LD + col) = ra[c];
    }
#pragma unroll
    for (int c = 0; c < B_CH; ++c) {
      int ch = tid + c * 256, r = ch / CPR, col = (ch % CPR) * VE;
      *(V16 *)(Bs + r * LDS_LD + col) = rb[c];
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  const int nk = g.K / KT;
  load(0);
  store();
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) load((kt + 1) * KT);
#pragma unroll
    for (int kk = 0; kk < KT / (2 * KS); ++kk) {
      const int kc = kk * 2 * KS + (lane >> 5) * KS;
      frag a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = *(const frag *)(As + (wm * WM + i * 32 + (lane & 31)) * LDS_LD + kc);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = *(const frag *)(Bs + (wn * WN + j * 32 + (lane & 31)) * LDS_LD + kc);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::mma(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
    if (kt + 1 < nk) {
      store();
      __syncthreads();
    }
  }

  // ---------------------------------------------------------------- epilogue
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int n = n0 + wn * WN + j * 32 + (lane & 31);
    const float bn = g.bias ? g.bias[n] : 0.0f;
    float gate = 1.0f;
    if (EPI == EPI_RESID && g.gate) gate = g.gate[n] + (g.gate2 ? g.gate2[n] : 0.0f);
    int part = 0, hh = 0, dd = 0;
    if (EPI == EPI_QKV || EPI == EPI_TEXTKV) {
      part = n / g.hidden;
      int c = n - part * g.hidden;
      hh = c / kHeadDim;
      dd = c - hh * kHeadDim;
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + wm * WM + i * 32 + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
        if (m >= g.M) continue;
        const float v = acc[i][j][e] + bn;
        if (EPI == EPI_STORE) {
          ((T *)g.out)[(size_t)m * g.ldo + n] = from_f<T>(v);
        } else if (EPI == EPI_GELU) {
          ((T *)g.out)[(size_t)m * g.ldo + n] = from_f<T>(gelu_tanh(v));
        } else if (EPI == EPI_RESID) {
          float *xp = g.X + (size_t)m * g.ldx + n;
          const float x = *xp + gate * v;
          *xp = x;
          if (g.xt) ((T *)g.xt)[(size_t)m * g.ldx + n] = from_f<T>(x);
          if (g.hrows) ((T *)g.hrows)[(size_t)m * g.N + n] = from_f<T>(x);
          if (g.hslot) {
            const int pk = g.rows[m];
            ((T *)g.hslot)[row_chain(pk) * g.chain_stride + (size_t)row_token(pk) * g.hidden + n] =
                from_f<T>(x);
          }
        } else if (EPI == EPI_QKV) {
          if (part == 0) {
            ((T *)g.out)[(size_t)m * g.ldo + n] = from_f<T>(v);
          } else {
            const int pk = g.rows[m];
            const size_t cb = (size_t)row_chain(pk) * g.chain_stride;
            const int tok = row_token(pk);
            if (part == 1)
              ((T *)g.kslot)[cb + ((size_t)hh * g.tokens + tok) * kHeadDim + dd] = from_f<T>(v);
            else
              ((T *)g.vslot)[cb + ((size_t)hh * g.tokens + tok) * kHeadDim + dd] = from_f<T>(v);
          }
        } else if (EPI == EPI_TEXTKV) {
          const int b = m / g.text_len, t = m - b * g.text_len;
          T *base = (T *)g.tkv + (size_t)b * g.tkv_chain_stride;
          const size_t half = (size_t)(g.hidden / kHeadDim) * g.text_pad * kHeadDim;
          if (part == 0)
            base[((size_t)hh * g.text_pad + t) * kHeadDim + dd] = from_f<T>(v);
          else
            base[half + ((size_t)hh * kHeadDim + dd) * g.text_pad + t] = from_f<T>(v);
        }
      }
    }
  }
}

template <typename T, int BM, int BN>
static hipError_t launch_tile(const GemmArgs &a, int epi, hipStream_t s) {
  dim3 grid(a.N / BN, (a.M + BM - 1) / BM);
  switch (epi) {
    case EPI_STORE: rc_launch(gemm_kernel<T, BM, BN, EPI_STORE>, grid, dim3(256), 0, s, a); break;
    case EPI_GELU: rc_launch(gemm_kernel<T, BM, BN, EPI_GELU>, grid, dim3(256), 0, s, a); break;
    case EPI_RESID: rc_launch(gemm_kernel<T, BM, BN, EPI_RESID>, grid, dim3(256), 0, s, a); break;
    case EPI_QKV: rc_launch(gemm_kernel<T, BM, BN, EPI_QKV>, grid, dim3(256), 0, s, a); break;
    case EPI_TEXTKV: rc_launch(gemm_kernel<T, BM, BN, EPI_TEXTKV>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Tile choice: the largest tile that still gives every CU at least two
// workgroups, falling back to 64x64 for the narrow low-row GEMMs.
template <typename T> hipError_t launch_gemm(const GemmArgs &a, int epi, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  if (a.N % 64 != 0 || a.K % (128 / (int)sizeof(T)) != 0) return hipErrorInvalidValue;
  auto wgs = [&](int bm, int bn) { return (long)((a.M + bm - 1) / bm) * (a.N / bn); };
  if (a.N % 128 == 0 && wgs(128, 128) >= 512) return launch_tile<T, 128, 128>(a, epi, s);
  if (a.N % 128 == 0 && wgs(64, 128) >= 384) return launch_tile<T, 64, 128>(a, epi, s);
  return launch_tile<T, 64, 64>(a, epi, s);
}

template hipError_t launch_gemm<bf16>(const GemmArgs &, int, hipStream_t);
template hipError_t launch_gemm<float>(const GemmArgs &, int, hipStream_t);

}  // namespace rc
