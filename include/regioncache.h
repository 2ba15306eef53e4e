/*
 * regioncache.h -- C ABI of the region-reuse DiT denoising step (RegionCache).
 *
 * The library runs one PixArt-alpha-shaped diffusion transformer step on an
 * MI355X (gfx950) in two forms: a dense step that recomputes every token and
 * fills the cache pool, and a region-reuse step that recomputes only the
 * active (edited) tokens and reuses the cached state of the others.  It also
 * localises the edit region from cross-attention maps.
 *
 * Paper passages the calls implement (RegionCache, arxiv 2608.29809):
 *   build cache      -- Sec. 3.2, "Hidden-State-Oriented Caching": per-step,
 *                       per-block keys, values and block outputs of every token
 *                       of a turn, kept for the next turn to reuse.
 *   localize region  -- Sec. 3.2: the edit region is the set of image tokens
 *                       whose aggregated cross-attention to a new or modified
 *                       text token reaches a threshold derived from that map.
 *   reuse step       -- Sec. 3.3, "Region-Level Sparse Attention": only active
 *                       tokens form queries; keys and values span all tokens;
 *                       inactive outputs come from the cache and are merged.
 *                       Sec. 3.4, "Kernel Fusing": fresh active keys/values are
 *                       written to their cached positions by the projection
 *                       GEMM itself.
 *   update cache     -- Sec. 3.2: hidden states of edit-affected regions are
 *                       recomputed and written back into the pool.
 *
 * Conventions shared by every call
 *   - All pointers named as device pointers are HIP device memory owned by the
 *     caller; the library allocates no device memory and frees nothing.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls only
 *     enqueue work and return; buffers must stay alive until the stream has
 *     executed it.  Calls that fill a host output (`*_host`) synchronise.
 *   - Every argument the host can check is checked before the first launch;
 *     a failed check returns a negative rc_status, launches nothing and
 *     leaves a message for rc_last_error().  HIP launch/runtime failures
 *     return RC_ERR_HIP.  No call aborts the process or throws.
 *   - Element type "E" is the model storage type: float (RC_F32) or bfloat16
 *     (RC_BF16).  Bias vectors, modulation tables, latents and attention maps
 *     are always float32.
 *   - Tokens are numbered row-major over the grid_h x grid_w patch grid
 *     (i = y*grid_w + x).  A "chain" is one independent edit sequence.
 *   - Device pointers must be 16-byte aligned.
 *
 * Model internals (the paper evaluates PixArt-alpha and does not restate it):
 * LayerNorm without affine (eps = ln_eps), adaLN-single modulation
 * x*(1+scale)+shift with per-block tables added to a shared timestep
 * projection, self-attention, ungated cross-attention to the text, GELU-tanh
 * MLP, 2x2 patch embedding with a fixed 2-D sin-cos position table, a final
 * modulated linear layer and a deterministic DDIM update.
 */
#ifndef REGIONCACHE_H
#define REGIONCACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RC_OK = 0,
  RC_ERR_INVALID_ARG = -1, /* null pointer, bad enum, negative size */
  RC_ERR_SHAPE = -2,       /* sizes inconsistent with the model config */
  RC_ERR_ALIGN = -3,       /* device pointer not 16-byte aligned */
  RC_ERR_INDEX = -4,       /* offsets not monotone / out of range */
  RC_ERR_CAPACITY = -5,    /* caller buffer smaller than required */
  RC_ERR_NO_DEVICE = -6,   /* no usable HIP device */
  RC_ERR_HIP = -7,         /* a HIP runtime call or launch failed */
  RC_ERR_UNSUPPORTED = -8  /* config outside what the kernels implement */
} rc_status;

typedef enum { RC_F32 = 0, RC_BF16 = 1 } rc_dtype;

/* Model and grid shape.  Supported: head_dim == 72, hidden == heads*72,
 * hidden and mlp multiples of 128, grid_h*grid_w a multiple of 64 and at most
 * 16384, text_len <= 128, latent_ch*patch*patch == 16, patch == 2,
 * out_ch*patch*patch <= 64, text_dim a multiple of 64. */
typedef struct {
  int32_t hidden;     /* C, 1152 */
  int32_t heads;      /* 16 */
  int32_t head_dim;   /* 72 */
  int32_t mlp;        /* 4608 */
  int32_t layers;     /* L */
  int32_t text_len;   /* M, 120 */
  int32_t text_dim;   /* width of the raw text features (4096), == hidden in token mode */
  int32_t grid_h, grid_w;
  int32_t latent_ch;  /* 4 */
  int32_t patch;      /* 2 */
  int32_t out_ch;     /* 8: noise channels followed by variance channels */
  int32_t dtype;      /* rc_dtype */
  int32_t token_mode; /* 1: single-block form -- hidden tokens in, block output out,
                         timestep vector given directly, text already hidden-wide;
                         no patch embedding, final layer or sampler */
  float ln_eps;       /* 1e-6 */
} rc_model_config;

/* One block's parameters (device pointers).  Matrices are [out][in] row-major
 * in E; biases and the modulation table are float32. */
typedef struct {
  const void *qkv_w;   /* [3C][C]: rows 0..C-1 query, C..2C-1 key, 2C..3C-1 value; head h owns
                          rows h*72..h*72+71 of each part */
  const void *proj_w;  /* [C][C] self-attention output projection */
  const void *xq_w;    /* [C][C] cross-attention query */
  const void *xkv_w;   /* [2C][C] cross-attention key (first C rows) and value */
  const void *xproj_w; /* [C][C] cross-attention output projection */
  const void *fc1_w;   /* [F][C] */
  const void *fc2_w;   /* [C][F] */
  const float *qkv_b, *proj_b, *xq_b, *xkv_b, *xproj_b, *fc1_b, *fc2_b;
  const float *sst;    /* [6][C]: shift1, scale1, gate1, shift2, scale2, gate2 (before adding t0) */
} rc_layer_weights;

/* Whole-model parameters (device pointers; `layers` is a HOST array of
 * config.layers entries that rc_create copies).  In token mode only `layers`,
 * tblock_w and tblock_b are read. */
typedef struct {
  const rc_layer_weights *layers;
  const void *pe_w;     /* [C][latent_ch*p*p]; input index c*p*p + pi*p + qi */
  const float *pe_b;    /* [C] */
  const void *temb_w1;  /* [C][256] on [cos(t f_k), sin(t f_k)], f_k = 10000^(-k/128) */
  const float *temb_b1;
  const void *temb_w2;  /* [C][C] */
  const float *temb_b2;
  const void *tblock_w; /* [6C][C] adaLN-single projection of silu(t_emb) */
  const float *tblock_b;
  const void *cap_w1;   /* [C][text_dim] caption projection, GELU-tanh between the two layers */
  const float *cap_b1;
  const void *cap_w2;   /* [C][C] */
  const float *cap_b2;
  const void *fin_w;    /* [p*p*out_ch][C]; output (pi*p+qi)*out_ch + c is channel c of pixel (pi,qi) */
  const float *fin_b;
  const float *fin_sst; /* [2][C]: shift, scale of the final layer (before adding t_emb) */
} rc_weights;

/* The cache pool (Sec. 3.2): one caller-owned device buffer of
 * rc_cache_bytes(ctx, batch, steps) bytes holding, for every chain b, step t
 * and block l, a slot of three E arrays -- K [H][N][72], V [H][N][72] and
 * the block-output hidden state H [N][C] -- followed (not in
 * token mode) by the float32 latent trajectory [batch][steps+1][c][2gh][2gw],
 * where entry t is the latent entering step t and entry t+1 the latent it
 * produced.  rc_cache_offsets gives the byte offsets. */
typedef struct {
  void *base;
  size_t bytes;
  int32_t batch;
  int32_t steps;
} rc_cache_view;

/* Active token set (device arrays + host copy of the offsets).  Tokens of
 * chain b are idx[offsets[b] .. offsets[b+1]-1], chain-local and strictly
 * ascending.  The host checks only the per-chain counts (offsets_host);
 * ascending order, range and agreement of the device offsets with
 * offsets_host are the caller's promise unless it asks for the device check
 * (rc_validate_active, or RC_VALIDATE on rc_reuse_step): without it an
 * out-of-range token is written outside its slot.  rc_localize_region and
 * rc_compact_mask produce valid sets. */
typedef struct {
  const int32_t *idx;          /* device [offsets[batch]] */
  const int32_t *offsets;      /* device [batch+1] */
  const int32_t *offsets_host; /* host [batch+1], offsets_host[0] == 0 */
  int32_t batch;
} rc_active_set;

typedef struct rc_ctx rc_ctx;

/* Message of the last failed call on this thread ("" if none). */
const char *rc_last_error(void);

/* Validate the config, copy it and the weight pointers into a host-side
 * context.  Touches no device.  RC_ERR_UNSUPPORTED for shapes outside the
 * list above.  A context holds host-side state (timing records and, once a
 * host-resident step has run, its side streams and events): calls on one
 * context must not overlap from several host threads. */
rc_status rc_create(const rc_model_config *config, const rc_weights *weights, rc_ctx **out);
void rc_destroy(rc_ctx *ctx);

/* Sizes in bytes of the caller-owned buffers. */
size_t rc_cache_bytes(const rc_ctx *ctx, int32_t batch, int32_t steps);
size_t rc_text_kv_bytes(const rc_ctx *ctx, int32_t batch);
/* Workspace for a step over up to `max_rows` active rows in total across
 * `batch` chains (a dense step uses batch*N rows). */
size_t rc_workspace_bytes(const rc_ctx *ctx, int32_t max_rows, int32_t batch);

/* Byte offsets inside the cache of slot (b, t, l): K, V and H;
 * and of latent trajectory entry (b, t) (returns RC_ERR_SHAPE in token mode
 * for the latent). */
rc_status rc_cache_offsets(const rc_ctx *ctx, const rc_cache_view *cache, int32_t b, int32_t t,
                           int32_t l, size_t *k_off, size_t *v_off, size_t *h_off);
rc_status rc_cache_latent_offset(const rc_ctx *ctx, const rc_cache_view *cache, int32_t b,
                                 int32_t t, size_t *off);

/* Per-turn text preparation: caption projection (skipped in token mode) and,
 * for every block, the cross-attention keys and values of the text tokens.
 * txt: device E [batch][text_len][text_dim].  text_kv: device E buffer of
 * rc_text_kv_bytes(ctx, batch); entry (l, b) holds K [H][Mp][72] then V
 * transposed [H][72][Mp], Mp = text_len rounded up to 64, padding zero. */
rc_status rc_prepare_text(rc_ctx *ctx, const void *txt, int32_t batch, void *text_kv,
                          void *workspace, size_t workspace_bytes, void *stream);

/* Inputs of one step.
 *   input   -- device; latent float32 [batch][c][2gh][2gw] (the x_t entering
 *              the step), or in token mode hidden tokens E [batch][N][C].
 *   t_vec   -- token mode only: device float32 [C] timestep vector, 16-byte aligned; else NULL.
 *   timestep, timestep_next -- integer DDPM timesteps of this step and of the
 *              next one (-1 after the last step); ignored in token mode.
 *   text_kv -- from rc_prepare_text for the same batch.
 *   delta_cols_host, n_delta -- text columns of new or modified prompt tokens
 *              (host array, 0 <= n_delta <= 8).  When maps != NULL the step
 *              ADDS, for every computed token, the sum over heads and blocks
 *              of its cross-attention probability on each delta column into
 *              maps [batch][N][n_delta] (device float32).
 *   latent_out -- device float32 [batch][c][2gh][2gw] (NULL in token mode).
 *   text_valid -- device int32 [batch]: the number of valid (unpadded)
 *              prompt tokens of each chain; cross-attention of chain b sees
 *              text tokens 0 .. text_valid[b]-1 only (values are clamped to
 *              1 .. text_len; delta columns of a chain should be valid
 *              tokens, others get probability 0).  NULL: all text_len
 *              tokens are valid.
 *   guided, guidance_scale -- classifier-free guidance (not in the paper;
 *              PixArt-alpha's sampling practice).  guided = 1: the batch holds
 *              pairs of chains, 2p conditional and 2p+1 unconditional (null
 *              prompt), with the same input latent, the same trajectory and
 *              the same active tokens (equal counts are checked; equal
 *              indices are the caller's promise).  The noise prediction of
 *              each token is eps_u + guidance_scale * (eps_c - eps_u) and both
 *              chains of a pair receive the same DDIM update.  guided = 0:
 *              chains are independent. */
typedef struct {
  const void *input;
  const float *t_vec;
  int32_t timestep, timestep_next;
  const void *text_kv;
  const int32_t *delta_cols_host;
  int32_t n_delta;
  float *maps;
  float *latent_out;
  const int32_t *text_valid;
  int32_t guided;
  float guidance_scale;
} rc_step_io;

/* BUILD CACHE (Sec. 3.2): dense step `step` over every token of every chain.
 * Writes the whole slot (K, V, H of every block) of step `step`, the latent
 * trajectory entries `step` (input) and `step+1` (output), and latent_out. */
rc_status rc_build_cache(rc_ctx *ctx, const rc_cache_view *cache, int32_t step, const rc_step_io *io,
                         void *workspace, size_t workspace_bytes, void *stream);

/* Flags of rc_reuse_step. */
#define RC_FUSE_UPDATE 1u /* write active hidden rows straight into the slot's H */
#define RC_VALIDATE 2u    /* check the active set on the device first (as rc_validate_active,
                             with the first 16 bytes of the workspace as scratch): an invalid
                             set returns RC_ERR_INDEX before any of the step's launches.
                             Synchronises the stream. */

/* RUN REUSE STEP (Sec. 3.3, 3.4): region-sparse step `step` over the active
 * set.  Per block, fresh keys/values of active tokens are written into the
 * slot before attention, active queries attend over all N keys of the slot,
 * and (with RC_FUSE_UPDATE) the active block outputs are written into the
 * slot's H, which then holds the merged hidden state.  Without the flag the
 * active outputs go to active_hidden, device E [L][total][C], and the slot's H
 * is left for rc_update_cache.  latent_out receives the cached trajectory
 * entry step+1 with the active patches replaced by their DDIM update, and
 * the same patches are written into trajectory entry step+1.  An empty set
 * leaves the slot unchanged and copies the cached latent. */
rc_status rc_reuse_step(rc_ctx *ctx, const rc_cache_view *cache, int32_t step,
                        const rc_active_set *active, const rc_step_io *io, void *active_hidden,
                        uint32_t flags, void *workspace, size_t workspace_bytes, void *stream);

/* UPDATE CACHE (Sec. 3.2): scatter active_hidden [L][total][C] (E) into the
 * H arrays of slot `step` at the active tokens. */
rc_status rc_update_cache(rc_ctx *ctx, const rc_cache_view *cache, int32_t step,
                          const rc_active_set *active, const void *active_hidden, void *stream);

/* Device check of an active set (the active token set of Sec. 3.3) for a
 * pool of `batch` chains: the host counts as in rc_reuse_step, then the
 * device offsets must equal offsets_host and every chain's tokens must be
 * strictly ascending (hence unique) and inside [0, N).  Returns RC_OK, or
 * RC_ERR_INDEX with the first offending chain, entry and token in
 * rc_last_error().  scratch: >= 16 bytes of caller device memory (overwritten).
 * Reads the active set only, writes nothing else, synchronises the stream. */
rc_status rc_validate_active(const rc_ctx *ctx, const rc_active_set *active, int32_t batch, void *scratch,
                             size_t scratch_bytes, void *stream);

/* HOST-RESIDENT POOL (Sec. 3.4, pipelined execution).  The cache pool may
 * live in pinned host memory (hipHostMalloc or torch pin_memory: page-locked
 * and device-accessible; rc_cache_bytes and the slot layout are unchanged)
 * when it does not fit in device memory.  A step then computes block l in
 * entry l % 3 of a caller-owned device staging ring of
 * rc_staging_bytes(ctx, batch) bytes: the copy engine uploads the keys and
 * values of block l from the pool while earlier blocks compute, and after
 * block l a small kernel writes the rows the step computed (keys, values and
 * hidden state of every computed token) back into the pool while block l+1
 * computes.  Both side streams are owned by the context (default priority),
 * fork from `stream` at the start of the call and join it before the step's
 * work on `stream` completes: the pool holds the step's results once
 * `stream` has drained.  Results equal those of rc_reuse_step with
 * RC_FUSE_UPDATE / rc_build_cache on a device pool of the same contents.
 * bf16 storage only (RC_ERR_UNSUPPORTED otherwise); RC_ERR_INVALID_ARG if
 * cache->base is not pinned host memory or staging is not device memory.
 * All steps of one context that use the pool must run on one device.  The
 * staging ring holds no state between calls. */
size_t rc_staging_bytes(const rc_ctx *ctx, int32_t batch);
rc_status rc_reuse_step_hosted(rc_ctx *ctx, const rc_cache_view *cache, int32_t step,
                               const rc_active_set *active, const rc_step_io *io, void *staging,
                               size_t staging_bytes, void *workspace, size_t workspace_bytes,
                               void *stream);
/* The dense step with the pool in host memory: nothing is uploaded, every
 * row of every block is written back. */
rc_status rc_build_cache_hosted(rc_ctx *ctx, const rc_cache_view *cache, int32_t step,
                                const rc_step_io *io, void *staging, size_t staging_bytes,
                                void *workspace, size_t workspace_bytes, void *stream);

/* LOCALIZE REGION (Sec. 3.2): for each chain and delta column j, the map
 * a_j = maps[b][:, j] (device float32 [batch][N][n_delta], any positive
 * scale) is min-max normalised over the chain's tokens; token i joins the
 * region when (a_j(i) - min)/(max - min) >= threshold for some j (a constant
 * map selects nothing); the region is dilated by a (2*radius+1)^2 square
 * clipped at the grid border, written as mask [batch][N] (device u8) and
 * compacted to idx (device, capacity batch*N) and offsets [batch+1]
 * (device).  If offsets_host != NULL the call synchronises and copies the
 * offsets there.  0 <= radius <= 4. */
rc_status rc_localize_region(rc_ctx *ctx, const float *maps, int32_t batch, int32_t n_delta,
                             float threshold, int32_t radius, uint8_t *mask, int32_t *idx,
                             int32_t *offsets, int32_t *offsets_host, void *stream);

/* Cross-attention maps from raw logits (Sec. 3.2 aggregation over heads and
 * blocks): logits device bf16 [n_layers][heads][tokens][text_len]; maps_out
 * device float32 [tokens][n_delta] receives, for each delta column, the sum
 * over (layer, head) of the softmax over the text_len columns.  `partial`
 * is device scratch of rc_maps_from_logits_scratch_bytes bytes.
 * tokens must be a multiple of 64, text_len <= 128, n_delta <= 8. */
size_t rc_maps_from_logits_scratch_bytes(int32_t n_layers, int32_t tokens, int32_t n_delta);
rc_status rc_maps_from_logits(const void *logits, int32_t n_layers, int32_t heads, int32_t tokens,
                              int32_t text_len, const int32_t *delta_cols_host, int32_t n_delta,
                              float *maps_out, void *partial, size_t partial_bytes, void *stream);

/* ALLOCATION-FREE VARIANT of rc_maps_from_logits, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same computation and results, with
 * the per-layer partial maps in a library-owned static device array of
 * RC_STATIC_SCRATCH_BYTES instead of the caller's `partial`.  Each GPU the
 * library runs on holds its own copy of that array until the process ends;
 * its address is looked up once per device on the first call there.  The
 * call allocates and frees nothing.
 *   - n_layers*tokens*n_delta*4 must not exceed RC_STATIC_SCRATCH_BYTES
 *     (16 MiB: up to 32 layers x 16384 tokens x 8 delta columns), else
 *     RC_ERR_CAPACITY before any launch.  Other arguments as above.
 *   - Every call on one GPU shares the array and leaves its contents behind;
 *     each call overwrites the part it reads before reading it, so nothing
 *     needs clearing.  Calls that overlap on one GPU (several streams or
 *     host threads without ordering) race on the array: their maps are
 *     undefined.  Order such calls on one stream. */
#define RC_STATIC_SCRATCH_BYTES ((size_t)16 << 20)
rc_status rc_maps_from_logits_noalloc(const void *logits, int32_t n_layers, int32_t heads, int32_t tokens,
                                      int32_t text_len, const int32_t *delta_cols_host, int32_t n_delta,
                                      float *maps_out, void *stream);

/* Stable compaction of masks [batch][tokens] (device u8, nonzero = active)
 * into idx (device, capacity batch*tokens) and offsets [batch+1] (device);
 * offsets_host as in rc_localize_region. */
rc_status rc_compact_mask(const uint8_t *mask, int32_t batch, int32_t tokens, int32_t *idx,
                          int32_t *offsets, int32_t *offsets_host, void *stream);

/* Wait for `stream`; returns RC_ERR_HIP if any enqueued work failed. */
rc_status rc_sync(void *stream);

/* Per-kernel timing for profiling: while enabled, every operation of the
 * context is bracketed by a pair of HIP events on its stream, stamped by the
 * dispatches of its first and last kernel; every class is one kernel per
 * operation except RC_KC_MISC.  Query returns the summed duration (ms) and
 * operation count of one kernel class since enabling (it synchronises).
 * Classes are the RC_KC_* values. */
enum {
  RC_KC_GEMM = 0, RC_KC_ATTN_SELF = 1, RC_KC_ATTN_CROSS = 2, RC_KC_ATTN_COMBINE = 3,
  RC_KC_NORM = 4, RC_KC_EMBED = 5, RC_KC_FINAL = 6, RC_KC_COND = 7, RC_KC_MISC = 8,
  RC_KC_GEMM_QKV = 9, RC_KC_GEMM_FC1 = 10, RC_KC_GEMM_FC2 = 11, RC_KC_GEMM_PROJ = 12,
  RC_KC_GEMM_XQ = 13, /* float32 contexts only: bf16 projects the cross query inside RC_KC_ATTN_CROSS */
  RC_KC_GEMM_XPROJ = 14,
  RC_KC_SPLIT_FINISH = 15, /* sum of a split-K GEMM's partials (+ the next block's LayerNorm) */
  RC_KC_COUNT = 16
};
rc_status rc_set_kernel_timing(rc_ctx *ctx, int32_t enable);
rc_status rc_get_kernel_timing(rc_ctx *ctx, int32_t kernel_class, double *total_ms, int64_t *launches);

#ifdef __cplusplus
}
#endif
#endif /* REGIONCACHE_H */
