// Launch interface of the row-wise / elementwise kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rc {

struct MapsDelta {
  int n;
  int col[8];
};

struct EmbedArgs {
  const int *rows;        // packed (chain<<16)|token
  float *X;               // [R][C] residual stream
  int C, N, gh, gw;
  const float *latent;    // [B][4][2gh][2gw] (patch mode)
  const void *pe_w;       // [C][16] E
  const float *pe_b;      // [C]
  const void *tokens_in;  // token mode: [B][N][C] E, else null
};

struct FinalArgs {
  const int *rows;
  const float *X;         // [R][C]
  int R, C, gh, gw, out_ch;
  float eps;
  const void *fin_w;      // [p*p*out_ch][C] E
  const float *fin_b, *fin_sst, *t_emb;
  const float *latent_in;  // [B][4][2gh][2gw]
  float *latent_out;       // [B][4][2gh][2gw]
  float *traj_next;        // chain 0's trajectory entry t+1, or null
  long long traj_chain_stride;  // floats between chains' entries
  float ca, cb;            // DDIM: x' = ca*x + cb*eps
  // classifier-free guidance: chains 2p (conditional) and 2p+1
  // (unconditional) are paired row by row through the row offsets
  const int *offsets;      // [B+1] device row offsets (guided only)
  int guided;
  float gscale;
};

hipError_t launch_build_rows(const int *offsets, const int *idx, int B, int R, int *rows, hipStream_t s);
hipError_t launch_dense_offsets(int *offsets, int B, int N, hipStream_t s);
template <typename T> hipError_t launch_embed(const EmbedArgs &a, int R, hipStream_t s);
template <typename T>
hipError_t launch_ln_mod(const float *X, int R, int C, const float *table, const float *t0, int shift_row,
                         float eps, void *out, hipStream_t s);
hipError_t launch_timestep_features(float t, float *e, hipStream_t s);
template <typename T>
hipError_t launch_gemv(const void *W, const float *bias, const float *x, int N, int K, int silu_in, int silu_out,
                       float *y, hipStream_t s);
template <typename T> hipError_t launch_final_ddim(const FinalArgs &a, hipStream_t s);
// Copy of the key, value and hidden-state rows of `rows` (packed chain/token)
// from a staging slot to a cache slot of the same layout (bf16 only; the
// strides are between consecutive chains, in bytes).
hipError_t launch_writeback_rows(const int *rows, int R, const void *stage, long long stage_chain_bytes, void *dst,
                                 long long dst_chain_bytes, int heads, int tokens, int hidden_bytes, bool bf16_elems,
                                 int workgroups, hipStream_t s);
hipError_t launch_copy_chains(float *dst, long long dst_stride, const float *src, long long src_stride, int n, int B,
                              hipStream_t s);
hipError_t launch_scatter_rows(const int *offsets, const int *idx, int B, const void *src, int R, int row_bytes,
                               void *hslot, long long chain_stride_bytes, hipStream_t s);
hipError_t launch_zero(void *p, size_t bytes, hipStream_t s);

// localisation
hipError_t launch_maps_from_logits(const uint16_t *logits, int n_layers, int heads, int tokens, int text_len,
                                   const int *delta, int n_delta, float *partial, hipStream_t s);
hipError_t launch_sum_partials(const float *partial, int n_parts, int n, float *out, hipStream_t s);
hipError_t launch_localize(const float *maps, int B, int gh, int gw, int n_delta, float threshold, int radius,
                           uint8_t *mask, hipStream_t s);
hipError_t launch_compact(const uint8_t *mask, int B, int N, int *idx, int *offsets, hipStream_t s);
// verdict[0] = first invalid position of an active set, or -1 (offsets must be valid).
hipError_t launch_validate_active(const int *offsets, const int *idx, int B, int N, int *verdict, hipStream_t s);

}  // namespace rc
