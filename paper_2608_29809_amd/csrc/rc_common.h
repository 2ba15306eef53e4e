// Device-side helpers shared by the HIP kernels of the region-reuse step.
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>

namespace rc {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kLdsBytes = 160 * 1024;  // LDS per CU
constexpr int kHeadDim = 72;

// Matrix-core traits per storage type.  Both use the 32x32 output block whose
// lane layout is: lane l holds column l%32 and rows i*8 + (l/32)*4 + j in
// accumulator element i*4 + j.  Operand A supplies row l%32, operand B
// column l%32, each with KS consecutive k values starting at (l/32)*KS; one
// instruction reduces over 2*KS values of k.
template <typename T> struct Mfma;

template <> struct Mfma<bf16> {
  static constexpr int KS = 8;
  typedef bf16x8 frag;
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag zero() {
    frag z;
#pragma unroll
    for (int i = 0; i < 8; ++i) z[i] = (bf16)0.0f;
    return z;
  }
};

template <> struct Mfma<float> {
  static constexpr int KS = 1;
  typedef float frag;
  static __device__ __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ frag zero() { return 0.0f; }
};

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16>(bf16 v) { return (float)v; }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return (bf16)v; }

// 16-byte vector of storage elements
struct alignas(16) V16 { uint32_t w[4]; };

// Sum over the 16 lanes of a DPP row, in the vector ALU (no LDS permute):
// neighbours, pairs, half-row mirror, row mirror.  Every step combines two
// partial results that both lanes of a pair hold bit for bit, so all 16
// lanes end with the same value.
template <int CTRL> __device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_mov<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_mov<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_mov<0x141>(v);  // row_half_mirror
  return v + dpp_mov<0x140>(v);  // row_mirror
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
// Sum over a 256-thread workgroup in a fixed order (waves 0..3); `red` is 4
// floats of LDS.  Every thread of the workgroup must call it.
__device__ __forceinline__ float block4_sum(float v, float *red) {
  v = wave_sum(v);
  __syncthreads();  // earlier readers of red are done
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// tanh-approximated GELU, 0.5 x (1 + tanh u) with u = sqrt(2/pi) (x + 0.044715 x^3),
// evaluated through the identity 0.5 (1 + tanh u) = 1 / (1 + e^(-2u)): one
// exp2 and one reciprocal.  Saturates to x / 0 correctly for large |x|.
__device__ __forceinline__ float gelu_tanh(float x) {
  constexpr float k = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  const float e = exp2f(k * x * (1.0f + 0.044715f * x * x));
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}
__device__ __forceinline__ float silu(float x) { return x / (1.0f + __expf(-x)); }

// XCD-aware renumbering of a grid.  Workgroups are dealt to the eight XCDs
// round-robin by linear id p, so XCD x runs p = x, x+8, x+16, ...  The
// logical id returned packs each XCD's workgroups into one contiguous range
// (XCD x gets [off_x, off_x + count_x)), so that logically adjacent work --
// which the caller arranges to share operands -- shares that XCD's L2.  A
// bijection on [0, T) for any T.
__device__ __forceinline__ int xcd_logical_id(int p, int T) {
  const int x = p & 7, q = T >> 3, rem = T & 7;
  const int off = x * q + min(x, rem);
  return off + (p >> 3);
}

// Maximum of v over the two 32-lane halves of a wave (lane l and l ^ 32),
// exchanged by v_permlane32_swap in the vector ALU rather than through the
// LDS queue, so it does not wait behind in-flight LDS reads.
__device__ __forceinline__ float half_swap_max(float v) {
  const unsigned u = __float_as_uint(v);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Copy of 16 bytes per lane from global memory straight into LDS (lane i's
// bytes land at lds_wave_base + 16 i; the base must be uniform over the
// wave).  Issued as inline assembly so that the compiler does not see an
// LDS write in flight and does not make every later LDS read wait for all
// outstanding vector loads; the caller orders the copy against its readers
// with explicit s_waitcnt vmcnt and a barrier.  M0 is written one wait state
// before the load that reads it.
__device__ __forceinline__ void lds_dma16(const void *gsrc, const void *lds_wave_base) {
  const unsigned base = __builtin_amdgcn_readfirstlane(
      (unsigned)(uintptr_t)(const __attribute__((address_space(3))) char *)lds_wave_base);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gsrc), "s"(base)
               : "memory", "m0");
}

// Memory-side cache warm-up of a buffer a later kernel reads: one dword of
// each 128-byte line is copied into a 256-byte LDS scratch of the calling
// wave that nothing reads, so no register is held; the lines are then
// served from the Infinity Cache instead of HBM.  Caller `part` of `parts`
// (one wave per workgroup) covers its contiguous share of the lines.  Called
// before the kernel's own first loads: loads retire in order, so the
// kernel's first vmcnt waits also retire these copies (the warming kernel
// pays for part of their latency), and the calling wave has waited for them
// before it ends, as it waits for its own LDS copies.
__device__ __forceinline__ void warm_lines(const void *p, long long lines, long long part, long long parts,
                                           const void *lds_wave_scratch) {
  if (lines <= 0) return;
  const unsigned base = __builtin_amdgcn_readfirstlane(
      (unsigned)(uintptr_t)(const __attribute__((address_space(3))) char *)lds_wave_scratch);
  const long long per = (lines + parts - 1) / parts, l0 = part * per, l1 = min(l0 + per, lines);
  for (long long i = l0 + (threadIdx.x & 63); i < l1; i += 64) {
    const char *src = (const char *)p + i * 128;
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off" ::"v"(src), "s"(base)
                 : "memory", "m0");
  }
}

// Row r of the active set is packed as (chain << 16) | token.
__device__ __forceinline__ int row_chain(int packed) { return packed >> 16; }
__device__ __forceinline__ int row_token(int packed) { return packed & 0xFFFF; }

}  // namespace rc
