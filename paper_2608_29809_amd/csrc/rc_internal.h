// Internal launch interface between the C-ABI layer and the HIP kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace rc {

enum GemmEpi {
  EPI_STORE = 0,   // out = E(acc + bias)
  EPI_GELU = 1,    // out = E(gelu_tanh(acc + bias))
  EPI_RESID = 2,   // X += gate * (acc + bias); optional E copies of X (xt, H slot scatter, hidden rows)
  EPI_QKV = 3,     // q -> out (compact), k -> K slot, v -> V slot (token-major rows, like K)
  EPI_TEXTKV = 4,  // text keys/values -> per-chain text K / transposed V
  // out = E(gelu_tanh(r (acc - mu u) + v + bias)): a LayerNorm + modulation of
  // the A rows folded into the GEMM (see GemmArgs::fold_*)
  EPI_GELU_FOLD = 5,
};

struct GemmArgs {
  const void *A;  // [M][K] E, row stride lda
  const void *W;  // [N][K] E
  const float *bias;
  int M, N, K, lda;
  // EPI_STORE / EPI_GELU / EPI_QKV (queries)
  void *out;
  int ldo;
  // EPI_RESID
  float *X;
  int ldx;
  const float *gate;  // [N] or null (gate 1); the gate is gate[n] + gate2[n]
  const float *gate2; // [N] or null
  void *xt;           // [M][ldx] E copy of the updated X, or null
  void *hrows;        // [M][N] E copy of the updated X (active hidden rows), or null
  // scatter targets (EPI_RESID H slot, EPI_QKV K/V slots)
  const int *rows;    // packed (chain<<16)|token per row
  void *hslot;        // H of chain 0's slot, or null
  void *kslot;        // K of chain 0's slot
  void *vslot;        // V of chain 0's slot (row-major like K)
  long long chain_stride;  // elements between consecutive chains' slots
  int tokens;              // N tokens per chain
  int hidden;              // C
  // EPI_TEXTKV
  void *tkv;        // entry (layer, chain 0)
  int text_len, text_pad;
  long long tkv_chain_stride;
  // buffer a later kernel reads, warmed into the memory-side cache (or null)
  const void *warm;
  long long warm_lines;  // 128-byte lines
  // LayerNorm + modulation folded into the next GEMM.  With h = (x - mu) r
  // (1 + scale) + shift (r = 1/sqrt(var + eps) over the row), h W^T =
  // r (x~ W^T - mu u) + v, where x~ = x (1 + scale), u = W (1 + scale) and
  // v = W shift.  Producer (EPI_RESID, fold_stats set): xt receives E(x~)
  // instead of E(x); per row and BN-column tile, the mean and the sum of
  // squared deviations of the updated x go to fold_stats[m * fold_nt + tile];
  // the workgroups of row tile 0 write 1 + scale and shift into fold_extra,
  // each as two rows: its bf16 rounding, then the bf16 rounding of the
  // remainder.  Consumer (EPI_GELU_FOLD): a BM-row tile holds BM - 4 rows of
  // A (= x~) and fold_extra's four rows, whose products summed in pairs are
  // u and v; fold_stats is merged per row (in tile order) into mu and r.
  const float *fold_scale[2];  // scale = fold_scale[0] + fold_scale[1], [N] each (producer)
  const float *fold_shift[2];  // shift = fold_shift[0] + fold_shift[1] (producer)
  float2 *fold_stats;          // [M][fold_nt] (mean, sum of squared deviations)
  int fold_nt;                 // producer column tiles (K / fold_nt columns each)
  void *fold_extra;            // [4][C] E
  float fold_eps;              // consumer
};
// most producer column tiles a folded LayerNorm merges per row
constexpr int kFoldMaxTiles = 24;


constexpr int kArgChains = 16;  // chains whose row offsets travel in the kernel arguments

struct AttnArgs {
  const void *Q;         // [R][C] E compact queries (chains concatenated)
  const void *K;         // chain 0, head 0 keys [n_keys][72]
  const void *V;         // chain 0, head 0 values: [n_keys][72] (v_rowmajor) or transposed [72][n_keys]
  int v_rowmajor;        // 1 for the cache's values, 0 for the transposed text values
  long long chain_stride;  // elements between chains for K and V
  long long head_stride;   // elements between heads (n_keys*72)
  const int *offsets;    // [B+1] device row offsets of chains
  int n_keys;            // keys per chain (multiple of 64)
  int n_valid;           // keys >= n_valid are masked out
  const int *text_valid; // device [chains] per-chain valid key counts (clamped to 1..n_valid), or null
  int hidden;            // C = heads*72
  int splits;            // key-range splits (grid.y = heads*splits)
  void *O;               // [R][C] E output (splits == 1)
  float *Opart;          // [splits][R][C] split outputs (splits > 1): fp32 unnormalised (fp32 path) or bf16 normalised (launch_attention3)
  float *ML;             // [splits][R][heads][2] running max (log2 domain) and sum
  int total_rows;        // R (stride of the partial arrays)
  // map emission (cross-attention)
  int n_delta;
  int delta[8];
  float *pmaps;          // [heads][R][n_delta]
  float scale_log2;      // log2(e)/sqrt(72)
  const void *warm;      // buffer a later kernel reads, warmed into the memory-side cache (or null)
  long long warm_lines;  // 128-byte lines
  // query projection computed inside the cross-attention (launch_attention2q):
  // Q = E(Xq . Wq^T + bq), Xq [R][hidden] E, Wq [hidden][hidden] E (row n =
  // output column n), bq [hidden] fp32; Q above is then unused
  const void *q_x;
  const void *q_w;
  const float *q_b;
  // offsets[0..n_arg_offs] by value (the host's copy): chains b < n_arg_offs
  // read their row range from the kernel arguments, one dependent load less
  // at kernel start, when every cache line is cold
  int n_arg_offs;
  int arg_offs[kArgChains + 1];
};

// Row range [first, last) of chain b.
__device__ __forceinline__ int2 chain_rows(const AttnArgs &a, int b) {
  if (b < a.n_arg_offs) return make_int2(a.arg_offs[b], a.arg_offs[b + 1]);
  return make_int2(a.offsets[b], a.offsets[b + 1]);
}

template <typename T> hipError_t launch_gemm(const GemmArgs &a, int epi, hipStream_t s);

// bf16 GEMM with direct-to-LDS staging and optional split-K (rc_gemm2.hip).
struct GemmPlan {
  int bm, bn, splits, kg;  // kg: K groups inside one workgroup
  int stages;              // LDS ring depth per K group
  int wgm, wgn;            // waves of one K group along M and N (4 or 8 waves)
};
GemmPlan plan_gemm2(int M, int N, int K, size_t partial_cap_floats);
// LayerNorm + modulation of the next block applied to the rows a residual
// GEMM has just completed: out = E(LN(X) * (1 + scale) + shift) with shift and
// scale = rows shift_row and shift_row+1 of sst + t0.
struct LnNext {
  const float *sst;
  const float *t0;
  int shift_row;
  float eps;
  void *out;  // [M][N] E
};
// The tiles of a bf16 GEMM; with a split plan they write fp32 partials,
// which launch_gemm2_finish then sums.
hipError_t launch_gemm2(const GemmArgs &a, int epi, const GemmPlan &plan, float *partial, hipStream_t s);
// Sum of a split plan's partials with the epilogue.  With `ln` non-null the
// reduction of an EPI_RESID GEMM also applies `ln` (one pass over each
// finished row); *ln_done tells the caller whether it did.
hipError_t launch_gemm2_finish(const GemmArgs &a, int epi, const GemmPlan &plan, const float *partial,
                               hipStream_t s, const LnNext *ln = nullptr, bool *ln_done = nullptr);
template <typename T> hipError_t launch_attention(const AttnArgs &a, int n_chains, int max_rows,
                                                  bool emit_maps, hipStream_t s);
// bf16 cross-attention to the transposed text values with its query
// projection fused in: each workgroup projects its own 64 rows of one head
// from a.q_x / a.q_w / a.q_b, then attends; emits the delta-column maps when
// a.pmaps is set (rc_attn2.hip).  hidden 1152, at most 128 keys, one key
// range.
hipError_t launch_attention2q(const AttnArgs &a, int n_chains, int max_rows, hipStream_t s);
// bf16 self-attention with the next tile's score MFMAs overlapping the
// softmax (rc_attn3.hip); no map emission.
hipError_t launch_attention3(const AttnArgs &a, int n_chains, int max_rows, hipStream_t s);
// Split combine for launch_attention3: Opart holds normalised bf16 split
// outputs [splits][R][C], ML the log2-domain maxima and denominators.
hipError_t launch_attn_combine_norm(const void *Opart, const float *ML, void *O, int R, int heads, int splits,
                                    hipStream_t s);
hipError_t launch_attn_combine(const float *Opart, const float *ML, void *O, bool bf16_out, int R,
                               int heads, int splits, hipStream_t s);
hipError_t launch_maps_reduce(const float *pmaps, const int *rows, float *maps, int R, int heads,
                              int n_delta, int tokens, hipStream_t s);

}  // namespace rc
