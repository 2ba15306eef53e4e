// C ABI of the region-reuse DiT step: host-side validation, buffer layouts
// and the kernel sequence of each call.  The library allocates no device
// memory; every buffer is the caller's.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/regioncache.h"
#include "rc_common.h"
#include "rc_elem.h"
#include "rc_launch.h"
#include "rc_internal.h"

using rc::bf16;

namespace rc {
LaunchTiming &launch_timing() {
  static thread_local LaunchTiming t;
  return t;
}
}  // namespace rc

namespace {

thread_local std::string g_err;

rc_status fail(rc_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
rc_status fail(rc_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define RC_HIP(expr)                                                                        \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return fail(RC_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define RC_CHECK(cond, st, ...)                  \
  do {                                           \
    if (!(cond)) return fail((st), __VA_ARGS__); \
  } while (0)

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

// Library-owned scratch of the allocation-free maps call
// (rc_maps_from_logits_noalloc): the per-layer partial maps, at most
// kStaticScratchBytes.  Every GPU the library runs on holds its own copy
// until the process ends.  In host code `scratch` names a host-side stand-in,
// not device memory: kernels get the address static_scratch() looks up.
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

// Entries of the device staging ring of the host-resident pool (layers in
// flight: one computing, one uploaded, one uploading).
constexpr int kRing = 3;

struct rc_ctx {
  rc_model_config cfg;
  rc_weights w;
  std::vector<rc_layer_weights> layers;
  int N, C, H, F, L, M, Mp;
  size_t esz;
  // per-kernel timing
  bool timing = false;
  struct Rec { int cls; hipEvent_t a, b; };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  size_t pool_used = 0;
  // host-resident pool: an upload stream and a write-back stream (default
  // priority, created on first use on device pipe_device) and the events
  // that order them against the caller's stream
  int pipe_device = -1;
  hipStream_t copy_s = nullptr, wb_s = nullptr;
  hipEvent_t up_ev[kRing] = {}, wb_ev[kRing] = {}, cmp_ev = nullptr, fork_ev = nullptr, join_ev = nullptr;
};

namespace {

// ------------------------------------------------------------------ layouts

size_t slot_elems(const rc_ctx *c) { return (size_t)3 * c->N * c->C; }
size_t latent_floats(const rc_ctx *c) {
  return (size_t)c->cfg.latent_ch * c->cfg.grid_h * c->cfg.patch * c->cfg.grid_w * c->cfg.patch;
}
size_t slots_bytes(const rc_ctx *c, int B, int T) { return align256((size_t)B * T * c->L * slot_elems(c) * c->esz); }
size_t cache_bytes(const rc_ctx *c, int B, int T) {
  size_t b = slots_bytes(c, B, T);
  if (!c->cfg.token_mode) b += (size_t)B * (T + 1) * latent_floats(c) * sizeof(float);
  return b;
}
size_t slot_offset(const rc_ctx *c, int T, int b, int t, int l) {
  return (((size_t)b * T + t) * c->L + l) * slot_elems(c) * c->esz;
}
size_t latent_offset(const rc_ctx *c, int B, int T, int b, int t) {
  return slots_bytes(c, B, T) + ((size_t)b * (T + 1) + t) * latent_floats(c) * sizeof(float);
}
size_t text_kv_elems_per_entry(const rc_ctx *c) { return (size_t)2 * c->H * c->Mp * rc::kHeadDim; }

constexpr int kMaxSplits = 8;
int part_cap_rows(int max_rows) { return kMaxSplits * std::min(max_rows, 1024); }

struct WsLayout {
  size_t rows, offsets, X, A1, Q, O, G, part, ml, pmaps, e, th, temb, t0, gpart, fstats, fextra, total;
  size_t gpart_floats;
  size_t txt_h, txt_y, txt_total;
};

WsLayout ws_layout(const rc_ctx *c, int max_rows, int B) {
  WsLayout w{};
  size_t o = 0;
  auto take = [&](size_t bytes) { size_t at = o; o = align256(o + bytes); return at; };
  const size_t R = (size_t)std::max(max_rows, 1);
  w.rows = take(R * 4);
  w.offsets = take((size_t)(B + 1) * 4);
  w.X = take(R * c->C * 4);
  w.A1 = take(R * c->C * c->esz);
  w.Q = take(R * c->C * c->esz);
  w.O = take(R * c->C * c->esz);
  w.G = take(R * c->F * c->esz);
  const size_t pr = (size_t)part_cap_rows(max_rows);
  w.part = take(pr * c->C * 4);
  w.ml = take(pr * c->H * 2 * 4);
  w.pmaps = take((size_t)c->H * R * 8 * 4);
  w.e = take(256 * 4);
  w.th = take((size_t)c->C * 4);
  w.temb = take((size_t)c->C * 4);
  w.t0 = take((size_t)6 * c->C * 4);
  w.gpart_floats = (size_t)std::min(max_rows, 2048) * 8 * c->C;
  w.gpart = take(w.gpart_floats * 4);
  w.fstats = take(R * rc::kFoldMaxTiles * 8 + 256);  // + the 16-byte reads' overhang
  w.fextra = take((size_t)4 * c->C * c->esz);
  w.total = o;
  // text preparation reuses the front of the workspace
  size_t t = 0;
  auto take2 = [&](size_t bytes) { size_t at = t; t = align256(t + bytes); return at; };
  w.txt_h = take2((size_t)B * c->M * c->C * c->esz);
  w.txt_y = take2((size_t)B * c->M * c->C * c->esz);
  w.txt_total = t;
  return w;
}

// ------------------------------------------------------------------ timing

template <typename F> rc_status timed(rc_ctx *c, int cls, hipStream_t s, F &&launch) {
  if (!c->timing) {
    RC_HIP(launch());
    return RC_OK;
  }
  if (c->pool_used + 2 > c->pool.size()) {
    for (int i = 0; i < 256; ++i) {
      hipEvent_t e;
      RC_HIP(hipEventCreate(&e));
      c->pool.push_back(e);
    }
  }
  // the dispatches stamp the pair themselves: start of the first kernel of
  // the operation, end of its last kernel
  hipEvent_t a = c->pool[c->pool_used], b = c->pool[c->pool_used + 1];
  ::rc::LaunchTiming &lt = ::rc::launch_timing();
  lt = ::rc::LaunchTiming{a, b, 0};
  const hipError_t e = launch();
  const int n = lt.launches;
  lt = ::rc::LaunchTiming{};
  RC_HIP(e);
  if (n > 0) {
    c->pool_used += 2;
    c->recs.push_back({cls, a, b});
  }
  return RC_OK;
}

#define RC_TRY(expr)                  \
  do {                                \
    rc_status st_ = (expr);           \
    if (st_ != RC_OK) return st_;     \
  } while (0)

// ------------------------------------------------------------------ validation helpers

rc_status check_cache(const rc_ctx *c, const rc_cache_view *cache, int step) {
  RC_CHECK(cache, RC_ERR_INVALID_ARG, "cache is null");
  RC_CHECK(cache->base, RC_ERR_INVALID_ARG, "cache->base is null");
  RC_CHECK(aligned16(cache->base), RC_ERR_ALIGN, "cache->base not 16-byte aligned");
  RC_CHECK(cache->batch >= 1 && cache->batch <= 32767, RC_ERR_SHAPE, "cache->batch %d out of range", cache->batch);
  RC_CHECK(cache->steps >= 1, RC_ERR_SHAPE, "cache->steps %d < 1", cache->steps);
  RC_CHECK(step >= 0 && step < cache->steps, RC_ERR_SHAPE, "step %d outside [0, %d)", step, cache->steps);
  const size_t need = cache_bytes(c, cache->batch, cache->steps);
  RC_CHECK(cache->bytes >= need, RC_ERR_CAPACITY, "cache has %zu bytes, needs %zu", cache->bytes, need);
  return RC_OK;
}

rc_status check_io(const rc_ctx *c, const rc_step_io *io) {
  RC_CHECK(io, RC_ERR_INVALID_ARG, "io is null");
  RC_CHECK(io->input, RC_ERR_INVALID_ARG, "io->input is null");
  RC_CHECK(aligned16(io->input), RC_ERR_ALIGN, "io->input not 16-byte aligned");
  RC_CHECK(io->text_kv, RC_ERR_INVALID_ARG, "io->text_kv is null");
  RC_CHECK(aligned16(io->text_kv), RC_ERR_ALIGN, "io->text_kv not 16-byte aligned");
  RC_CHECK(io->n_delta >= 0 && io->n_delta <= 8, RC_ERR_INVALID_ARG, "n_delta %d outside [0, 8]", io->n_delta);
  if (io->maps && io->n_delta > 0) {
    RC_CHECK(io->delta_cols_host, RC_ERR_INVALID_ARG, "delta_cols_host is null");
    for (int j = 0; j < io->n_delta; ++j)
      RC_CHECK(io->delta_cols_host[j] >= 0 && io->delta_cols_host[j] < c->M, RC_ERR_INDEX,
               "delta column %d = %d outside [0, %d)", j, io->delta_cols_host[j], c->M);
  }
  if (c->cfg.token_mode) {
    RC_CHECK(io->t_vec, RC_ERR_INVALID_ARG, "token mode needs t_vec");
    RC_CHECK(aligned16(io->t_vec), RC_ERR_ALIGN, "io->t_vec not 16-byte aligned");
  } else {
    RC_CHECK(io->latent_out, RC_ERR_INVALID_ARG, "io->latent_out is null");
    RC_CHECK(io->timestep >= 0 && io->timestep < 1000, RC_ERR_INVALID_ARG, "timestep %d outside [0, 1000)",
             io->timestep);
    RC_CHECK(io->timestep_next >= -1 && io->timestep_next < 1000, RC_ERR_INVALID_ARG,
             "timestep_next %d outside [-1, 1000)", io->timestep_next);
  }
  RC_CHECK(io->guided == 0 || io->guided == 1, RC_ERR_INVALID_ARG, "guided must be 0 or 1");
  RC_CHECK(!io->guided || !c->cfg.token_mode, RC_ERR_UNSUPPORTED, "guidance needs the latent path");
  RC_CHECK(!io->guided || std::isfinite(io->guidance_scale), RC_ERR_INVALID_ARG, "guidance_scale not finite");
  return RC_OK;
}

// A guided step pairs chains 2p (conditional) and 2p+1 (unconditional) row
// by row: the batch must be even and each pair's active counts equal.
rc_status check_guided(const rc_step_io *io, int batch, const rc_active_set *act) {
  if (!io->guided) return RC_OK;
  RC_CHECK(batch % 2 == 0, RC_ERR_SHAPE, "guided step needs (conditional, unconditional) chain pairs, batch %d",
           batch);
  if (act)
    for (int b = 0; b < batch; b += 2) {
      const int n0 = act->offsets_host[b + 1] - act->offsets_host[b];
      const int n1 = act->offsets_host[b + 2] - act->offsets_host[b + 1];
      RC_CHECK(n0 == n1, RC_ERR_INDEX, "guided pair %d: %d and %d active tokens", b / 2, n0, n1);
    }
  return RC_OK;
}

// DDPM linear-beta schedule (1e-4 .. 0.02 over 1000 steps), cumulative product.
double alpha_bar(int t) {
  if (t < 0) return 1.0;
  double a = 1.0;
  for (int i = 0; i <= t; ++i) a *= 1.0 - (1e-4 + (0.02 - 1e-4) * (double)i / 999.0);
  return a;
}

// ------------------------------------------------------------------ the step

// One GEMM of the step: bf16 goes through the direct-to-LDS kernel with a
// per-shape tile/split plan, fp32 through the register-staged kernel.
template <typename T>
rc_status gemm(rc_ctx *c, int cls, const rc::GemmArgs &g, int epi, float *part, size_t part_floats, hipStream_t s,
               const rc::LnNext *ln = nullptr, bool *ln_done = nullptr) {
  if (ln_done) *ln_done = false;
  if constexpr (sizeof(T) == 2) {
    const rc::GemmPlan pl = rc::plan_gemm2(g.M, g.N, g.K, part ? part_floats : 0);
    RC_TRY(timed(c, cls, s, [&] { return rc::launch_gemm2(g, epi, pl, part, s); }));
    if (pl.splits == 1) return RC_OK;
    return timed(c, RC_KC_SPLIT_FINISH, s, [&] { return rc::launch_gemm2_finish(g, epi, pl, part, s, ln, ln_done); });
  } else {
    return timed(c, cls, s, [&] { return rc::launch_gemm<T>(g, epi, s); });
  }
}

// ------------------------------------------------------------------ host-resident pool

// Pipelined execution with the cache pool in pinned host memory (Sec. 3.4):
// block l computes in entry l % kRing of a device staging ring, whose keys
// and values were uploaded from the pool by the copy engine while earlier
// blocks computed; after block l the rows it computed (keys, values, hidden
// state) are written back to the pool by a small kernel on a second stream
// while block l+1 computes, and the freed entry takes the upload of block
// l + kRing.  Events order the three streams; the caller's stream waits for
// the last write-back before the step's work on it completes.
struct HostPipe {
  char *staging;       // device ring: kRing entries of `entry_bytes`
  size_t entry_bytes;  // batch * slot bytes
  const char *host;    // the pool, host address (uploads)
};

rc_status ensure_pipe(rc_ctx *c) {
  int dev = -1;
  RC_HIP(hipGetDevice(&dev));
  if (c->copy_s) {
    RC_CHECK(dev == c->pipe_device, RC_ERR_INVALID_ARG,
             "host-resident steps of one context must run on one device (%d, now %d)", c->pipe_device, dev);
    return RC_OK;
  }
  RC_HIP(hipStreamCreateWithFlags(&c->copy_s, hipStreamNonBlocking));
  RC_HIP(hipStreamCreateWithFlags(&c->wb_s, hipStreamNonBlocking));
  // the events inside a step only order work on this device (no host reads
  // what they guard), so they skip the system-scope fence; the final join,
  // after which the host may read the pool, keeps it
  const unsigned order_only = hipEventDisableTiming | hipEventDisableSystemFence;
  for (int r = 0; r < kRing; ++r) {
    RC_HIP(hipEventCreateWithFlags(&c->up_ev[r], order_only));
    RC_HIP(hipEventCreateWithFlags(&c->wb_ev[r], order_only));
  }
  RC_HIP(hipEventCreateWithFlags(&c->cmp_ev, order_only));
  RC_HIP(hipEventCreateWithFlags(&c->fork_ev, order_only));
  RC_HIP(hipEventCreateWithFlags(&c->join_ev, hipEventDisableTiming));
  c->pipe_device = dev;
  return RC_OK;
}

// Joins the write-back stream into the caller's stream when the step leaves
// (also on an error return), so no write into the pool outlives the step.
struct PipeJoin {
  rc_ctx *c;
  hipStream_t s;
  bool forked = false;
  ~PipeJoin() {
    if (forked && hipEventRecord(c->join_ev, c->wb_s) == hipSuccess) (void)hipStreamWaitEvent(s, c->join_ev, 0);
  }
};

template <typename T>
rc_status run_step(rc_ctx *c, const rc_cache_view *cache, int step, const rc_step_io *io, bool dense,
                   const rc_active_set *act, void *active_hidden, bool fuse, void *ws, size_t ws_bytes,
                   hipStream_t s, const HostPipe *hp = nullptr) {
  const int B = cache->batch, N = c->N, C = c->C, H = c->H, F = c->F, L = c->L, T_ = cache->steps;
  std::vector<int> counts(B);
  int R = 0, max_rb = 0;
  if (dense) {
    for (int b = 0; b < B; ++b) counts[b] = N;
    R = B * N;
    max_rb = N;
  } else {
    for (int b = 0; b < B; ++b) {
      counts[b] = act->offsets_host[b + 1] - act->offsets_host[b];
      max_rb = std::max(max_rb, counts[b]);
    }
    R = act->offsets_host[B];
  }
  const WsLayout wl = ws_layout(c, R, B);
  RC_CHECK(ws, RC_ERR_INVALID_ARG, "workspace is null");
  RC_CHECK(aligned16(ws), RC_ERR_ALIGN, "workspace not 16-byte aligned");
  RC_CHECK(ws_bytes >= wl.total, RC_ERR_CAPACITY, "workspace has %zu bytes, needs %zu for %d rows", ws_bytes,
           wl.total, R);
  if (!dense && !fuse && R > 0) {
    RC_CHECK(active_hidden, RC_ERR_INVALID_ARG, "active_hidden is null without RC_FUSE_UPDATE");
    RC_CHECK(aligned16(active_hidden), RC_ERR_ALIGN, "active_hidden not 16-byte aligned");
  }

  char *wsb = (char *)ws;
  char *cb = (char *)cache->base;
  const size_t n_lat = c->cfg.token_mode ? 0 : latent_floats(c);
  const long long lat_chain_stride = (long long)(T_ + 1) * n_lat;
  float *traj_t = c->cfg.token_mode ? nullptr : (float *)(cb + latent_offset(c, B, T_, 0, step));
  float *traj_next = c->cfg.token_mode ? nullptr : (float *)(cb + latent_offset(c, B, T_, 0, step + 1));

  if (R == 0) {  // nothing active: slot untouched, latent from the cached trajectory
    if (!c->cfg.token_mode)
      RC_TRY(timed(c, RC_KC_MISC, s, [&] {
        return rc::launch_copy_chains(io->latent_out, n_lat, traj_next, lat_chain_stride, n_lat, B, s);
      }));
    return RC_OK;
  }

  int *rows = (int *)(wsb + wl.rows);
  const int *offsets_dev = dense ? (int *)(wsb + wl.offsets) : act->offsets;
  // the first chains' row offsets, passed by value to the attention kernels
  int n_arg_offs = std::min(B, rc::kArgChains), arg_offs[rc::kArgChains + 1];
  for (int b = 0; b <= n_arg_offs; ++b) arg_offs[b] = dense ? b * N : act->offsets_host[b];
  auto set_offsets = [&](rc::AttnArgs &a) {
    a.offsets = offsets_dev;
    a.n_arg_offs = n_arg_offs;
    for (int b = 0; b <= n_arg_offs; ++b) a.arg_offs[b] = arg_offs[b];
  };
  float *X = (float *)(wsb + wl.X);
  void *A1 = wsb + wl.A1, *Q = wsb + wl.Q, *O = wsb + wl.O, *G = wsb + wl.G;
  float *part = (float *)(wsb + wl.part), *ml = (float *)(wsb + wl.ml), *pmaps = (float *)(wsb + wl.pmaps);
  float *e = (float *)(wsb + wl.e), *th = (float *)(wsb + wl.th), *temb = (float *)(wsb + wl.temb);
  float *t0 = (float *)(wsb + wl.t0);
  float *gpart = (float *)(wsb + wl.gpart);
  const size_t gpf = wl.gpart_floats;
  float2 *fstats = (float2 *)(wsb + wl.fstats);
  void *fextra = wsb + wl.fextra;
  // bf16: the MLP-up LayerNorm folds into the GEMMs on either side of it
  // when both run unsplit.  The cross out-projection's epilogue writes each
  // row's mean and sum of squared deviations over its column tile and the
  // modulated copy x~ = x (1 + scale); the MLP-up GEMM takes four more A rows
  // per tile, (1 + scale) and shift as bf16 pairs, and applies
  // h W^T = r (x~ W^T - mean u) + v after its K loop (u, v: the products of
  // those rows).
  int fold_nt = 0;
  if (sizeof(T) == 2) {
    const rc::GemmPlan px = rc::plan_gemm2(R, C, C, gpf), p1 = rc::plan_gemm2(R, F, C, gpf);
    if (px.splits == 1 && p1.splits == 1 && C % px.bn == 0 && C / px.bn <= rc::kFoldMaxTiles) fold_nt = C / px.bn;
  }

  if (dense) RC_TRY(timed(c, RC_KC_MISC, s, [&] { return rc::launch_dense_offsets((int *)offsets_dev, B, N, s); }));
  RC_TRY(timed(c, RC_KC_MISC, s, [&] {
    return rc::launch_build_rows(offsets_dev, dense ? nullptr : act->idx, B, R, rows, s);
  }));

  // conditioning (adaLN-single)
  const rc_weights &W = c->w;
  if (c->cfg.token_mode) {
    RC_TRY(timed(c, RC_KC_COND, s, [&] {
      return rc::launch_gemv<T>(W.tblock_w, W.tblock_b, io->t_vec, 6 * C, C, 1, 0, t0, s);
    }));
  } else {
    RC_TRY(timed(c, RC_KC_COND, s, [&] { return rc::launch_timestep_features((float)io->timestep, e, s); }));
    RC_TRY(timed(c, RC_KC_COND, s, [&] { return rc::launch_gemv<T>(W.temb_w1, W.temb_b1, e, C, 256, 0, 1, th, s); }));
    RC_TRY(timed(c, RC_KC_COND, s, [&] { return rc::launch_gemv<T>(W.temb_w2, W.temb_b2, th, C, C, 0, 0, temb, s); }));
    RC_TRY(timed(c, RC_KC_COND, s, [&] {
      return rc::launch_gemv<T>(W.tblock_w, W.tblock_b, temb, 6 * C, C, 1, 0, t0, s);
    }));
  }

  // entry: gather + embed the computed tokens
  {
    rc::EmbedArgs ea{};
    ea.rows = rows;
    ea.X = X;
    ea.C = C;
    ea.N = N;
    ea.gh = c->cfg.grid_h;
    ea.gw = c->cfg.grid_w;
    if (c->cfg.token_mode) {
      ea.tokens_in = io->input;
    } else {
      ea.latent = (const float *)io->input;
      ea.pe_w = W.pe_w;
      ea.pe_b = W.pe_b;
    }
    RC_TRY(timed(c, RC_KC_EMBED, s, [&] { return rc::launch_embed<T>(ea, R, s); }));
  }

  // self-attention key splits: fill 2 workgroups x 256 CUs with as few
  // splits as possible (the bf16 kernel takes uneven splits)
  long qtiles = 0;
  for (int b = 0; b < B; ++b) qtiles += (counts[b] + 127) / 128;
  int splits = 1;
  if (sizeof(T) == 2) {
    double best = -1.0;
    const int max_s = std::min(N / 64, 16);
    for (int sp = 1; sp <= max_s; ++sp) {
      if ((long)R * sp > part_cap_rows(R) && sp > 1) break;
      const long wgs = qtiles * H * sp;
      const double eff = wgs / (std::ceil(wgs / 512.0) * 512.0) - 0.01 * sp;  // 2 workgroups per CU
      if (eff > best) { best = eff; splits = sp; }
    }
  } else {
    while (splits < kMaxSplits && qtiles * H * splits < 512 && N % (64 * splits * 2) == 0 &&
           (long)R * splits * 2 <= part_cap_rows(R))
      splits *= 2;
  }

  const bool emit = io->maps && io->n_delta > 0;
  // device pool: slot (b, step, l) in place; host-resident pool: entry
  // l % kRing of the staging ring, chains one slot apart
  const long long slot_chain_stride = hp ? (long long)slot_elems(c) : (long long)T_ * L * slot_elems(c);
  const size_t kv_half = (size_t)H * N * rc::kHeadDim;
  const float scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)rc::kHeadDim));

  PipeJoin pipe_join{c, s};
  auto upload = [&](int l) -> rc_status {  // keys and values of block l, every chain, on the copy stream
    char *dst = hp->staging + (size_t)(l % kRing) * hp->entry_bytes;
    for (int b = 0; b < B; ++b)
      RC_HIP(hipMemcpyAsync(dst + (size_t)b * slot_elems(c) * c->esz, hp->host + slot_offset(c, T_, b, step, l),
                            2 * kv_half * c->esz, hipMemcpyHostToDevice, c->copy_s));
    RC_HIP(hipEventRecord(c->up_ev[l % kRing], c->copy_s));
    return RC_OK;
  };
  if (hp) {
    RC_TRY(ensure_pipe(c));
    RC_HIP(hipEventRecord(c->fork_ev, s));  // earlier work on the caller's stream (and on the pool) first
    RC_HIP(hipStreamWaitEvent(c->copy_s, c->fork_ev, 0));
    RC_HIP(hipStreamWaitEvent(c->wb_s, c->fork_ev, 0));
    pipe_join.forked = true;
    if (!dense)  // a dense step recomputes every row: nothing to upload
      for (int l = 0; l < std::min(kRing, L); ++l) RC_TRY(upload(l));
  }

  // Weights of a block's later GEMMs are warmed into the memory-side cache
  // by earlier kernels of the block (each warming kernel pays for its extra
  // loads, so the pairs are the measured winners): for a region step the
  // out-projections and the MLP-down weights, warmed by GEMMs; for a dense
  // step also the cross query and MLP-up weights and the next block's QKV
  // weights, warmed by the attention kernels and the MLP-up GEMM.
  auto wlines = [&](long long n, long long k) { return n * k * (long long)c->esz / 128; };
  const long long fc2_lines = wlines(C, F), fc2_half = fc2_lines / 2;
  bool a1_ready = false;  // the previous block's MLP reduction already wrote this block's LN1 rows
  for (int l = 0; l < L; ++l) {
    const rc_layer_weights &lw = c->layers[l];
    T *slot = hp ? (T *)(hp->staging + (size_t)(l % kRing) * hp->entry_bytes)
                 : (T *)(cb + slot_offset(c, T_, 0, step, l));
    T *Ks = slot, *Vs = slot + kv_half, *Hs = slot + 2 * kv_half;
    if (hp) {
      if (!dense) RC_HIP(hipStreamWaitEvent(s, c->up_ev[l % kRing], 0));  // this block's keys/values are in
      else if (l >= kRing) RC_HIP(hipStreamWaitEvent(s, c->wb_ev[l % kRing], 0));  // the entry was written back
    }

    if (!a1_ready)
      RC_TRY(timed(c, RC_KC_NORM, s, [&] { return rc::launch_ln_mod<T>(X, R, C, lw.sst, t0, 0, c->cfg.ln_eps, A1, s); }));
    a1_ready = false;
    {  // QKV with the K/V scatter into the slot
      rc::GemmArgs g{};
      g.A = A1; g.W = lw.qkv_w; g.bias = lw.qkv_b; g.M = R; g.N = 3 * C; g.K = C; g.lda = C;
      g.out = Q; g.ldo = C; g.rows = rows; g.kslot = Ks; g.vslot = Vs;
      g.chain_stride = slot_chain_stride; g.tokens = N; g.hidden = C;
      g.warm = lw.proj_w; g.warm_lines = wlines(C, C);
      RC_TRY(gemm<T>(c, RC_KC_GEMM_QKV, g, rc::EPI_QKV, gpart, gpf, s));
    }
    {  // region-level sparse self-attention over the whole slot
      rc::AttnArgs a{};
      a.Q = Q; a.K = Ks; a.V = Vs; a.v_rowmajor = 1; a.chain_stride = slot_chain_stride; a.head_stride = (long long)N * rc::kHeadDim;
      set_offsets(a); a.n_keys = N; a.n_valid = N; a.hidden = C; a.splits = splits;
      a.O = O; a.Opart = part; a.ML = ml; a.total_rows = R; a.scale_log2 = scale_log2;
      if (dense) { a.warm = lw.xq_w; a.warm_lines = wlines(C, C); }
      RC_TRY(timed(c, RC_KC_ATTN_SELF, s, [&] {
        return sizeof(T) == 2 ? rc::launch_attention3(a, B, max_rb, s)
                              : rc::launch_attention<T>(a, B, max_rb, false, s);
      }));
      if (splits > 1)
        RC_TRY(timed(c, RC_KC_ATTN_COMBINE, s, [&] {
          return sizeof(T) == 2 ? rc::launch_attn_combine_norm(part, ml, O, R, H, splits, s)
                                : rc::launch_attn_combine(part, ml, O, false, R, H, splits, s);
        }));
    }
    {  // out-projection + gate + residual; E copy of X for the cross query
      rc::GemmArgs g{};
      g.A = O; g.W = lw.proj_w; g.bias = lw.proj_b; g.M = R; g.N = C; g.K = C; g.lda = C;
      g.X = X; g.ldx = C; g.gate = lw.sst + 2 * C; g.gate2 = t0 + 2 * C; g.xt = A1;
      g.warm = lw.xproj_w; g.warm_lines = wlines(C, C);
      RC_TRY(gemm<T>(c, RC_KC_GEMM_PROJ, g, rc::EPI_RESID, gpart, gpf, s));
    }
    if (sizeof(T) != 2) {  // cross-attention query (bf16: projected inside the cross-attention)
      rc::GemmArgs g{};
      g.A = A1; g.W = lw.xq_w; g.bias = lw.xq_b; g.M = R; g.N = C; g.K = C; g.lda = C; g.out = Q; g.ldo = C;
      RC_TRY(gemm<T>(c, RC_KC_GEMM_XQ, g, rc::EPI_STORE, gpart, gpf, s));
    }
    {  // cross-attention to the text, emitting the delta-token maps
      const T *tkv = (const T *)io->text_kv + (size_t)l * B * text_kv_elems_per_entry(c);
      rc::AttnArgs a{};
      a.Q = Q; a.K = tkv; a.V = tkv + (size_t)H * c->Mp * rc::kHeadDim; a.v_rowmajor = 0;
      a.chain_stride = (long long)text_kv_elems_per_entry(c); a.head_stride = (long long)c->Mp * rc::kHeadDim;
      set_offsets(a); a.n_keys = c->Mp; a.n_valid = c->M; a.text_valid = io->text_valid;
      a.hidden = C; a.splits = 1;
      a.O = O; a.total_rows = R; a.scale_log2 = scale_log2;
      a.q_x = A1; a.q_w = lw.xq_w; a.q_b = lw.xq_b;
      if (dense) { a.warm = lw.fc1_w; a.warm_lines = wlines(F, C); }
      else { a.warm = lw.fc2_w; a.warm_lines = fc2_half; }
      if (emit) {
        a.n_delta = io->n_delta;
        for (int j = 0; j < io->n_delta; ++j) a.delta[j] = io->delta_cols_host[j];
        a.pmaps = pmaps;
      }
      RC_TRY(timed(c, RC_KC_ATTN_CROSS, s, [&] {
        return sizeof(T) == 2 ? rc::launch_attention2q(a, B, max_rb, s)
                              : rc::launch_attention<T>(a, B, max_rb, emit, s);
      }));
      if (emit)
        RC_TRY(timed(c, RC_KC_MISC, s, [&] {
          return rc::launch_maps_reduce(pmaps, rows, io->maps, R, H, io->n_delta, N, s);
        }));
    }
    {  // cross out-projection + residual (no gate); the fold's statistics and x~
      rc::GemmArgs g{};
      g.A = O; g.W = lw.xproj_w; g.bias = lw.xproj_b; g.M = R; g.N = C; g.K = C; g.lda = C;
      g.X = X; g.ldx = C;
      if (fold_nt) {
        g.xt = A1;
        g.fold_scale[0] = lw.sst + 4 * C; g.fold_scale[1] = t0 + 4 * C;
        g.fold_shift[0] = lw.sst + 3 * C; g.fold_shift[1] = t0 + 3 * C;
        g.fold_stats = fstats; g.fold_nt = fold_nt; g.fold_extra = fextra;
      }
      if (!dense) { g.warm = (const char *)lw.fc2_w + fc2_half * 128; g.warm_lines = fc2_lines - fc2_half; }
      else { g.warm = lw.fc2_w; g.warm_lines = fc2_lines; }
      RC_TRY(gemm<T>(c, RC_KC_GEMM_XPROJ, g, rc::EPI_RESID, gpart, gpf, s));
    }
    if (!fold_nt)
      RC_TRY(timed(c, RC_KC_NORM, s, [&] { return rc::launch_ln_mod<T>(X, R, C, lw.sst, t0, 3, c->cfg.ln_eps, A1, s); }));
    {  // MLP up + GELU
      rc::GemmArgs g{};
      g.A = A1; g.W = lw.fc1_w; g.bias = lw.fc1_b; g.M = R; g.N = F; g.K = C; g.lda = C; g.out = G; g.ldo = F;
      if (dense && l + 1 < L) { g.warm = c->layers[l + 1].qkv_w; g.warm_lines = wlines(3 * C, C); }
      if (fold_nt) { g.fold_stats = fstats; g.fold_nt = fold_nt; g.fold_extra = fextra; g.fold_eps = c->cfg.ln_eps; }
      RC_TRY(gemm<T>(c, RC_KC_GEMM_FC1, g, fold_nt ? rc::EPI_GELU_FOLD : rc::EPI_GELU, gpart, gpf, s));
    }
    {  // MLP down + gate + residual; merge into the cached hidden state
      rc::GemmArgs g{};
      g.A = G; g.W = lw.fc2_w; g.bias = lw.fc2_b; g.M = R; g.N = C; g.K = F; g.lda = F;
      g.X = X; g.ldx = C; g.gate = lw.sst + 5 * C; g.gate2 = t0 + 5 * C;
      g.rows = rows; g.hidden = C; g.chain_stride = slot_chain_stride;
      if (dense || fuse) g.hslot = Hs;
      else g.hrows = (T *)active_hidden + (size_t)l * R * C;
      if (l + 1 < L) {
        const rc::LnNext ln{c->layers[l + 1].sst, t0, 0, c->cfg.ln_eps, A1};
        RC_TRY(gemm<T>(c, RC_KC_GEMM_FC2, g, rc::EPI_RESID, gpart, gpf, s, &ln, &a1_ready));
      } else {
        RC_TRY(gemm<T>(c, RC_KC_GEMM_FC2, g, rc::EPI_RESID, gpart, gpf, s));
      }
    }
    if (hp) {  // write block l's rows back to the pool beside block l+1, then reuse the entry
      const int r = l % kRing;
      RC_HIP(hipEventRecord(c->cmp_ev, s));
      RC_HIP(hipStreamWaitEvent(c->wb_s, c->cmp_ev, 0));
      char *dst = cb + slot_offset(c, T_, 0, step, l);
      RC_HIP(rc::launch_writeback_rows(rows, R, slot, (long long)slot_elems(c) * c->esz, dst,
                                       (long long)T_ * L * slot_elems(c) * c->esz, H, N, C * (int)c->esz,
                                       c->esz == 2, 64, c->wb_s));
      RC_HIP(hipEventRecord(c->wb_ev[r], c->wb_s));
      if (!dense && l + kRing < L) {
        RC_HIP(hipStreamWaitEvent(c->copy_s, c->wb_ev[r], 0));
        RC_TRY(upload(l + kRing));
      }
    }
  }

  if (!c->cfg.token_mode) {
    if (dense) {
      RC_TRY(timed(c, RC_KC_MISC, s, [&] {
        return rc::launch_copy_chains(traj_t, lat_chain_stride, (const float *)io->input, n_lat, n_lat, B, s);
      }));
    } else {
      RC_TRY(timed(c, RC_KC_MISC, s, [&] {
        return rc::launch_copy_chains(io->latent_out, n_lat, traj_next, lat_chain_stride, n_lat, B, s);
      }));
    }
    const double at = alpha_bar(io->timestep), an = alpha_bar(io->timestep_next);
    rc::FinalArgs fa{};
    fa.rows = rows; fa.X = X; fa.R = R; fa.C = C; fa.gh = c->cfg.grid_h; fa.gw = c->cfg.grid_w;
    fa.out_ch = c->cfg.out_ch; fa.eps = c->cfg.ln_eps; fa.fin_w = W.fin_w; fa.fin_b = W.fin_b;
    fa.fin_sst = W.fin_sst; fa.t_emb = temb; fa.latent_in = (const float *)io->input;
    fa.latent_out = io->latent_out; fa.traj_next = traj_next; fa.traj_chain_stride = lat_chain_stride;
    fa.offsets = offsets_dev; fa.guided = io->guided; fa.gscale = io->guidance_scale;
    fa.ca = (float)(std::sqrt(an) / std::sqrt(at));
    fa.cb = (float)(std::sqrt(1.0 - an) - std::sqrt(an) * std::sqrt(1.0 - at) / std::sqrt(at));
    RC_TRY(timed(c, RC_KC_FINAL, s, [&] { return rc::launch_final_ddim<T>(fa, s); }));
  }
  return RC_OK;
}

template <typename T>
rc_status run_text(rc_ctx *c, const void *txt, int B, void *text_kv, void *ws, size_t ws_bytes, hipStream_t s) {
  const int C = c->C, M = c->M;
  const WsLayout wl = ws_layout(c, 1, B);
  RC_CHECK(ws, RC_ERR_INVALID_ARG, "workspace is null");
  RC_CHECK(aligned16(ws), RC_ERR_ALIGN, "workspace not 16-byte aligned");
  RC_CHECK(ws_bytes >= wl.txt_total, RC_ERR_CAPACITY, "workspace has %zu bytes, text preparation needs %zu",
           ws_bytes, wl.txt_total);
  char *wsb = (char *)ws;
  const size_t kv_bytes = (size_t)c->L * B * text_kv_elems_per_entry(c) * c->esz;
  RC_TRY(timed(c, RC_KC_MISC, s, [&] { return rc::launch_zero(text_kv, kv_bytes, s); }));
  const void *y = txt;
  if (!c->cfg.token_mode) {
    rc::GemmArgs g{};
    g.A = txt; g.W = c->w.cap_w1; g.bias = c->w.cap_b1; g.M = B * M; g.N = C; g.K = c->cfg.text_dim;
    g.lda = c->cfg.text_dim; g.out = wsb + wl.txt_h; g.ldo = C;
    RC_TRY(gemm<T>(c, RC_KC_GEMM, g, rc::EPI_GELU, nullptr, 0, s));
    rc::GemmArgs g2{};
    g2.A = wsb + wl.txt_h; g2.W = c->w.cap_w2; g2.bias = c->w.cap_b2; g2.M = B * M; g2.N = C; g2.K = C;
    g2.lda = C; g2.out = wsb + wl.txt_y; g2.ldo = C;
    RC_TRY(gemm<T>(c, RC_KC_GEMM, g2, rc::EPI_STORE, nullptr, 0, s));
    y = wsb + wl.txt_y;
  }
  for (int l = 0; l < c->L; ++l) {
    rc::GemmArgs g{};
    g.A = y; g.W = c->layers[l].xkv_w; g.bias = c->layers[l].xkv_b; g.M = B * M; g.N = 2 * C; g.K = C; g.lda = C;
    g.tkv = (T *)text_kv + (size_t)l * B * text_kv_elems_per_entry(c);
    g.text_len = M; g.text_pad = c->Mp; g.tkv_chain_stride = (long long)text_kv_elems_per_entry(c); g.hidden = C;
    RC_TRY(gemm<T>(c, RC_KC_GEMM, g, rc::EPI_TEXTKV, nullptr, 0, s));
  }
  return RC_OK;
}

bool device_present() {
  int n = 0;
  return hipGetDeviceCount(&n) == hipSuccess && n > 0;
}

// Arguments of the maps-from-logits calls (everything but the scratch).
rc_status check_maps_args(const void *logits, int n_layers, int heads, int tokens, int text_len,
                          const int32_t *delta_cols_host, int n_delta, const float *maps_out) {
  RC_CHECK(logits && delta_cols_host && maps_out, RC_ERR_INVALID_ARG, "null argument");
  RC_CHECK(aligned16(logits), RC_ERR_ALIGN, "logits not 16-byte aligned");
  RC_CHECK(n_layers >= 1 && heads >= 1, RC_ERR_SHAPE, "n_layers/heads must be positive");
  RC_CHECK(tokens >= 64 && tokens % 64 == 0, RC_ERR_UNSUPPORTED, "tokens %d must be a positive multiple of 64",
           tokens);
  RC_CHECK(text_len >= 8 && text_len <= 128 && text_len % 8 == 0, RC_ERR_UNSUPPORTED,
           "text_len %d must be a multiple of 8 in [8, 128]", text_len);
  RC_CHECK(n_delta >= 1 && n_delta <= 8, RC_ERR_INVALID_ARG, "n_delta %d outside [1, 8]", n_delta);
  for (int j = 0; j < n_delta; ++j)
    RC_CHECK(delta_cols_host[j] >= 0 && delta_cols_host[j] < text_len, RC_ERR_INDEX, "delta column %d out of range",
             delta_cols_host[j]);
  RC_CHECK(tokens <= (1 << 24) && n_layers <= (1 << 16), RC_ERR_SHAPE, "tokens %d / n_layers %d too large", tokens,
           n_layers);
  return RC_OK;
}

// Per-layer partial maps (one kernel) summed over layers in order (another).
rc_status launch_maps(const void *logits, int n_layers, int heads, int tokens, int text_len,
                      const int32_t *delta_cols_host, int n_delta, float *maps_out, float *partial, hipStream_t s) {
  RC_HIP(rc::launch_maps_from_logits((const uint16_t *)logits, n_layers, heads, tokens, text_len, delta_cols_host,
                                     n_delta, partial, s));
  RC_HIP(rc::launch_sum_partials(partial, n_layers, tokens * n_delta, maps_out, s));
  return RC_OK;
}

// Device address of the static scratch array on the current device, looked
// up once per device (each GPU holds its own copy of the array, at its own
// address).  Host code uses only this address, never the array's name.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

rc_status static_scratch(void **out) {
  int dev = -1;
  RC_HIP(hipGetDevice(&dev));
  RC_CHECK(dev >= 0 && dev < kMaxDevices, RC_ERR_UNSUPPORTED, "device %d outside the library's table", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    RC_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    RC_CHECK(p, RC_ERR_HIP, "hipGetSymbolAddress returned a null address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return RC_OK;
}

}  // namespace

// ====================================================================== C ABI

extern "C" {

const char *rc_last_error(void) { return g_err.c_str(); }

rc_status rc_create(const rc_model_config *cfg, const rc_weights *w, rc_ctx **out) {
  g_err.clear();
  RC_CHECK(cfg && w && out, RC_ERR_INVALID_ARG, "null argument to rc_create");
  *out = nullptr;
  RC_CHECK(cfg->dtype == RC_F32 || cfg->dtype == RC_BF16, RC_ERR_INVALID_ARG, "dtype %d unknown", cfg->dtype);
  RC_CHECK(cfg->head_dim == rc::kHeadDim, RC_ERR_UNSUPPORTED, "head_dim %d != 72", cfg->head_dim);
  RC_CHECK(cfg->heads >= 1 && cfg->hidden == cfg->heads * cfg->head_dim, RC_ERR_SHAPE,
           "hidden %d != heads %d * head_dim", cfg->hidden, cfg->heads);
  RC_CHECK(cfg->hidden % 128 == 0 && cfg->hidden <= 1536, RC_ERR_UNSUPPORTED,
           "hidden %d must be a multiple of 128 and <= 1536", cfg->hidden);
  RC_CHECK(cfg->mlp > 0 && cfg->mlp % 128 == 0, RC_ERR_UNSUPPORTED, "mlp %d must be a multiple of 128", cfg->mlp);
  RC_CHECK(cfg->layers >= 1, RC_ERR_SHAPE, "layers %d < 1", cfg->layers);
  RC_CHECK(cfg->text_len >= 1 && cfg->text_len <= 128, RC_ERR_UNSUPPORTED, "text_len %d outside [1, 128]",
           cfg->text_len);
  RC_CHECK(cfg->grid_h >= 1 && cfg->grid_w >= 1, RC_ERR_SHAPE, "empty grid");
  const long N = (long)cfg->grid_h * cfg->grid_w;
  RC_CHECK(N % 64 == 0 && N <= 16384, RC_ERR_UNSUPPORTED, "grid_h*grid_w = %ld must be a multiple of 64, <= 16384",
           N);
  RC_CHECK(cfg->ln_eps > 0.0f, RC_ERR_INVALID_ARG, "ln_eps must be positive");
  RC_CHECK(w->layers, RC_ERR_INVALID_ARG, "weights->layers is null");
  if (cfg->token_mode) {
    RC_CHECK(cfg->text_dim == cfg->hidden, RC_ERR_SHAPE, "token mode needs text_dim == hidden");
  } else {
    RC_CHECK(cfg->patch == 2 && cfg->latent_ch * 4 == 16, RC_ERR_UNSUPPORTED,
             "patch must be 2 and latent_ch*patch^2 == 16");
    RC_CHECK(cfg->out_ch >= cfg->latent_ch && cfg->out_ch * 4 <= 64, RC_ERR_UNSUPPORTED,
             "out_ch %d unsupported", cfg->out_ch);
    RC_CHECK(cfg->text_dim > 0 && cfg->text_dim % 64 == 0, RC_ERR_UNSUPPORTED,
             "text_dim %d must be a multiple of 64", cfg->text_dim);
    RC_CHECK(w->pe_w && w->pe_b && w->temb_w1 && w->temb_b1 && w->temb_w2 && w->temb_b2 && w->cap_w1 &&
                 w->cap_b1 && w->cap_w2 && w->cap_b2 && w->fin_w && w->fin_b && w->fin_sst,
             RC_ERR_INVALID_ARG, "a global weight pointer is null");
  }
  RC_CHECK(w->tblock_w && w->tblock_b, RC_ERR_INVALID_ARG, "tblock weights are null");
  for (int l = 0; l < cfg->layers; ++l) {
    const rc_layer_weights &lw = w->layers[l];
    RC_CHECK(lw.qkv_w && lw.proj_w && lw.xq_w && lw.xkv_w && lw.xproj_w && lw.fc1_w && lw.fc2_w && lw.qkv_b &&
                 lw.proj_b && lw.xq_b && lw.xkv_b && lw.xproj_b && lw.fc1_b && lw.fc2_b && lw.sst,
             RC_ERR_INVALID_ARG, "layer %d has a null weight pointer", l);
    const void *mats[] = {lw.qkv_w, lw.proj_w, lw.xq_w, lw.xkv_w, lw.xproj_w, lw.fc1_w, lw.fc2_w};
    for (const void *p : mats) RC_CHECK(aligned16(p), RC_ERR_ALIGN, "layer %d weight not 16-byte aligned", l);
  }
  rc_ctx *c = new rc_ctx();
  c->cfg = *cfg;
  c->w = *w;
  c->layers.assign(w->layers, w->layers + cfg->layers);
  c->w.layers = c->layers.data();
  c->N = (int)N;
  c->C = cfg->hidden;
  c->H = cfg->heads;
  c->F = cfg->mlp;
  c->L = cfg->layers;
  c->M = cfg->text_len;
  c->Mp = (cfg->text_len + 63) / 64 * 64;
  c->esz = cfg->dtype == RC_BF16 ? 2 : 4;
  *out = c;
  return RC_OK;
}

void rc_destroy(rc_ctx *c) {
  if (!c) return;
  for (hipEvent_t e : c->pool) (void)hipEventDestroy(e);
  if (c->copy_s) {
    (void)hipStreamSynchronize(c->copy_s);
    (void)hipStreamSynchronize(c->wb_s);
    (void)hipStreamDestroy(c->copy_s);
    (void)hipStreamDestroy(c->wb_s);
    for (int r = 0; r < kRing; ++r) {
      (void)hipEventDestroy(c->up_ev[r]);
      (void)hipEventDestroy(c->wb_ev[r]);
    }
    (void)hipEventDestroy(c->cmp_ev);
    (void)hipEventDestroy(c->fork_ev);
    (void)hipEventDestroy(c->join_ev);
  }
  delete c;
}

size_t rc_cache_bytes(const rc_ctx *c, int32_t batch, int32_t steps) {
  if (!c || batch < 1 || steps < 1) return 0;
  return cache_bytes(c, batch, steps);
}

size_t rc_text_kv_bytes(const rc_ctx *c, int32_t batch) {
  if (!c || batch < 1) return 0;
  return (size_t)c->L * batch * text_kv_elems_per_entry(c) * c->esz;
}

size_t rc_workspace_bytes(const rc_ctx *c, int32_t max_rows, int32_t batch) {
  if (!c || batch < 1 || max_rows < 0) return 0;
  const WsLayout w = ws_layout(c, max_rows, batch);
  return std::max(w.total, w.txt_total);
}

rc_status rc_cache_offsets(const rc_ctx *c, const rc_cache_view *cache, int32_t b, int32_t t, int32_t l,
                           size_t *k_off, size_t *v_off, size_t *h_off) {
  RC_CHECK(c && cache, RC_ERR_INVALID_ARG, "null argument");
  RC_CHECK(b >= 0 && b < cache->batch && t >= 0 && t < cache->steps && l >= 0 && l < c->L, RC_ERR_SHAPE,
           "slot (%d, %d, %d) out of range", b, t, l);
  const size_t base = slot_offset(c, cache->steps, b, t, l);
  const size_t half = (size_t)c->H * c->N * rc::kHeadDim * c->esz;
  if (k_off) *k_off = base;
  if (v_off) *v_off = base + half;
  if (h_off) *h_off = base + 2 * half;
  return RC_OK;
}

rc_status rc_cache_latent_offset(const rc_ctx *c, const rc_cache_view *cache, int32_t b, int32_t t, size_t *off) {
  RC_CHECK(c && cache && off, RC_ERR_INVALID_ARG, "null argument");
  RC_CHECK(!c->cfg.token_mode, RC_ERR_SHAPE, "token mode keeps no latent trajectory");
  RC_CHECK(b >= 0 && b < cache->batch && t >= 0 && t <= cache->steps, RC_ERR_SHAPE, "latent (%d, %d) out of range",
           b, t);
  *off = latent_offset(c, cache->batch, cache->steps, b, t);
  return RC_OK;
}

rc_status rc_prepare_text(rc_ctx *c, const void *txt, int32_t batch, void *text_kv, void *ws, size_t ws_bytes,
                          void *stream) {
  g_err.clear();
  RC_CHECK(c && txt && text_kv, RC_ERR_INVALID_ARG, "null argument to rc_prepare_text");
  RC_CHECK(batch >= 1 && batch <= 32767, RC_ERR_SHAPE, "batch %d out of range", batch);
  RC_CHECK(aligned16(txt) && aligned16(text_kv), RC_ERR_ALIGN, "txt/text_kv not 16-byte aligned");
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  hipStream_t s = (hipStream_t)stream;
  return c->esz == 2 ? run_text<bf16>(c, txt, batch, text_kv, ws, ws_bytes, s)
                     : run_text<float>(c, txt, batch, text_kv, ws, ws_bytes, s);
}

rc_status rc_build_cache(rc_ctx *c, const rc_cache_view *cache, int32_t step, const rc_step_io *io, void *ws,
                         size_t ws_bytes, void *stream) {
  g_err.clear();
  RC_CHECK(c, RC_ERR_INVALID_ARG, "ctx is null");
  RC_TRY(check_cache(c, cache, step));
  RC_TRY(check_io(c, io));
  RC_TRY(check_guided(io, cache->batch, nullptr));
  RC_CHECK((long)cache->batch * c->N <= (1L << 30), RC_ERR_SHAPE, "batch too large");
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  hipStream_t s = (hipStream_t)stream;
  return c->esz == 2 ? run_step<bf16>(c, cache, step, io, true, nullptr, nullptr, true, ws, ws_bytes, s)
                     : run_step<float>(c, cache, step, io, true, nullptr, nullptr, true, ws, ws_bytes, s);
}

static rc_status check_active(const rc_ctx *c, const rc_cache_view *cache, const rc_active_set *a) {
  RC_CHECK(a, RC_ERR_INVALID_ARG, "active set is null");
  RC_CHECK(a->batch == cache->batch, RC_ERR_SHAPE, "active batch %d != cache batch %d", a->batch, cache->batch);
  RC_CHECK(a->offsets_host, RC_ERR_INVALID_ARG, "offsets_host is null");
  RC_CHECK(a->offsets_host[0] == 0, RC_ERR_INDEX, "offsets_host[0] = %d != 0", a->offsets_host[0]);
  for (int b = 0; b < a->batch; ++b) {
    const int n = a->offsets_host[b + 1] - a->offsets_host[b];
    RC_CHECK(n >= 0 && n <= c->N, RC_ERR_INDEX, "chain %d has %d active tokens (N = %d)", b, n, c->N);
  }
  if (a->offsets_host[a->batch] > 0)
    RC_CHECK(a->idx && a->offsets, RC_ERR_INVALID_ARG, "idx/offsets device arrays are null");
  return RC_OK;
}

// Device check of an active set whose host-side counts check_active has
// accepted: the device offsets equal the host copy, and every chain's
// tokens are strictly ascending and inside [0, N).  verdict_dev: 4 bytes of
// device scratch.  Synchronises the stream; launches nothing else.
static rc_status validate_active(const rc_ctx *c, const rc_active_set *a, int *verdict_dev, hipStream_t s) {
  const int B = a->batch, total = a->offsets_host[B];
  if (total == 0) return RC_OK;
  std::vector<int> offs(B + 1);
  RC_HIP(hipMemcpyAsync(offs.data(), a->offsets, sizeof(int) * (B + 1), hipMemcpyDeviceToHost, s));
  RC_HIP(hipStreamSynchronize(s));
  for (int b = 0; b <= B; ++b)
    RC_CHECK(offs[b] == a->offsets_host[b], RC_ERR_INDEX, "device offsets[%d] = %d differs from offsets_host[%d] = %d",
             b, offs[b], b, a->offsets_host[b]);
  RC_HIP(rc::launch_validate_active(a->offsets, a->idx, B, c->N, verdict_dev, s));
  int v = -1;
  RC_HIP(hipMemcpyAsync(&v, verdict_dev, sizeof(int), hipMemcpyDeviceToHost, s));
  RC_HIP(hipStreamSynchronize(s));
  if (v < 0) return RC_OK;
  const int b = (int)(std::upper_bound(offs.begin(), offs.end(), v) - offs.begin()) - 1;
  int tok[2] = {0, 0};
  const bool first = v == offs[b];
  RC_HIP(hipMemcpyAsync(tok, a->idx + (first ? v : v - 1), sizeof(int) * (first ? 1 : 2), hipMemcpyDeviceToHost, s));
  RC_HIP(hipStreamSynchronize(s));
  if (first)
    return fail(RC_ERR_INDEX, "active set: chain %d, entry %d: token %d outside [0, %d)", b, v - offs[b], tok[0],
                c->N);
  return fail(RC_ERR_INDEX, "active set: chain %d, entry %d: token %d after %d (not strictly ascending in [0, %d))", b,
              v - offs[b], tok[1], tok[0], c->N);
}

rc_status rc_reuse_step(rc_ctx *c, const rc_cache_view *cache, int32_t step, const rc_active_set *active,
                        const rc_step_io *io, void *active_hidden, uint32_t flags, void *ws, size_t ws_bytes,
                        void *stream) {
  g_err.clear();
  RC_CHECK(c, RC_ERR_INVALID_ARG, "ctx is null");
  RC_TRY(check_cache(c, cache, step));
  RC_TRY(check_io(c, io));
  RC_TRY(check_active(c, cache, active));
  RC_TRY(check_guided(io, cache->batch, active));
  RC_CHECK((flags & ~(RC_FUSE_UPDATE | RC_VALIDATE)) == 0, RC_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
  if (flags & RC_VALIDATE)
    RC_CHECK(ws && aligned16(ws) && ws_bytes >= 16, RC_ERR_INVALID_ARG, "RC_VALIDATE needs the workspace");
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  hipStream_t s = (hipStream_t)stream;
  const bool fuse = (flags & RC_FUSE_UPDATE) != 0;
  if (flags & RC_VALIDATE) RC_TRY(validate_active(c, active, (int *)ws, s));
  return c->esz == 2 ? run_step<bf16>(c, cache, step, io, false, active, active_hidden, fuse, ws, ws_bytes, s)
                     : run_step<float>(c, cache, step, io, false, active, active_hidden, fuse, ws, ws_bytes, s);
}

rc_status rc_update_cache(rc_ctx *c, const rc_cache_view *cache, int32_t step, const rc_active_set *active,
                          const void *active_hidden, void *stream) {
  g_err.clear();
  RC_CHECK(c, RC_ERR_INVALID_ARG, "ctx is null");
  RC_TRY(check_cache(c, cache, step));
  RC_TRY(check_active(c, cache, active));
  const int R = active->offsets_host[active->batch];
  if (R == 0) return RC_OK;
  RC_CHECK(active_hidden, RC_ERR_INVALID_ARG, "active_hidden is null");
  RC_CHECK(aligned16(active_hidden), RC_ERR_ALIGN, "active_hidden not 16-byte aligned");
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  hipStream_t s = (hipStream_t)stream;
  const size_t row_bytes = (size_t)c->C * c->esz;
  const long long chain_stride = (long long)cache->steps * c->L * slot_elems(c) * c->esz;
  const size_t half = (size_t)c->H * c->N * rc::kHeadDim * c->esz;
  for (int l = 0; l < c->L; ++l) {
    char *hs = (char *)cache->base + slot_offset(c, cache->steps, 0, step, l) + 2 * half;
    const char *src = (const char *)active_hidden + (size_t)l * R * row_bytes;
    RC_TRY(timed(c, RC_KC_MISC, s, [&] {
      return rc::launch_scatter_rows(active->offsets, active->idx, active->batch, src, R, (int)row_bytes, hs,
                                     chain_stride, s);
    }));
  }
  return RC_OK;
}

rc_status rc_validate_active(const rc_ctx *c, const rc_active_set *active, int32_t batch, void *scratch,
                             size_t scratch_bytes, void *stream) {
  g_err.clear();
  RC_CHECK(c && active, RC_ERR_INVALID_ARG, "null argument to rc_validate_active");
  RC_CHECK(batch >= 1 && batch <= 32767, RC_ERR_SHAPE, "batch %d out of range", batch);
  rc_cache_view v{};
  v.batch = batch;
  RC_TRY(check_active(c, &v, active));
  RC_CHECK(scratch && aligned16(scratch) && scratch_bytes >= 16, RC_ERR_INVALID_ARG,
           "scratch must be >= 16 bytes of 16-byte aligned device memory");
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  return validate_active(c, active, (int *)scratch, (hipStream_t)stream);
}

size_t rc_staging_bytes(const rc_ctx *c, int32_t batch) {
  if (!c || batch < 1) return 0;
  return (size_t)kRing * batch * slot_elems(c) * c->esz;
}

// Checks of a host-resident pool and its staging ring; on success `dev`
// is the pool's view at its device-accessible address and `hp` the pipeline.
static rc_status check_hosted(const rc_ctx *c, const rc_cache_view *cache, void *staging, size_t staging_bytes,
                              rc_cache_view *dev, HostPipe *hp) {
  RC_CHECK(c->esz == 2, RC_ERR_UNSUPPORTED, "the host-resident pool needs bf16 storage");
  RC_CHECK(staging, RC_ERR_INVALID_ARG, "staging is null");
  RC_CHECK(aligned16(staging), RC_ERR_ALIGN, "staging not 16-byte aligned");
  const size_t entry = (size_t)cache->batch * slot_elems(c) * c->esz;
  RC_CHECK(staging_bytes >= kRing * entry, RC_ERR_CAPACITY, "staging has %zu bytes, needs %zu", staging_bytes,
           kRing * entry);
  hipPointerAttribute_t ha{}, sa{};
  const hipError_t eh = hipPointerGetAttributes(&ha, cache->base);
  const hipError_t es = hipPointerGetAttributes(&sa, staging);
  (void)hipGetLastError();  // a plain (unpinned) host pointer is reported as an error: not sticky, cleared
  RC_CHECK(eh == hipSuccess && ha.type == hipMemoryTypeHost && ha.devicePointer, RC_ERR_INVALID_ARG,
           "cache->base is not pinned, device-accessible host memory");
  RC_CHECK(es == hipSuccess && sa.type == hipMemoryTypeDevice, RC_ERR_INVALID_ARG, "staging is not device memory");
  *dev = *cache;
  dev->base = ha.devicePointer;
  hp->staging = (char *)staging;
  hp->entry_bytes = entry;
  hp->host = (const char *)cache->base;
  return RC_OK;
}

rc_status rc_reuse_step_hosted(rc_ctx *c, const rc_cache_view *cache, int32_t step, const rc_active_set *active,
                               const rc_step_io *io, void *staging, size_t staging_bytes, void *ws, size_t ws_bytes,
                               void *stream) {
  g_err.clear();
  RC_CHECK(c, RC_ERR_INVALID_ARG, "ctx is null");
  RC_TRY(check_cache(c, cache, step));
  RC_TRY(check_io(c, io));
  RC_TRY(check_active(c, cache, active));
  RC_TRY(check_guided(io, cache->batch, active));
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  rc_cache_view dev{};
  HostPipe hp{};
  RC_TRY(check_hosted(c, cache, staging, staging_bytes, &dev, &hp));
  return run_step<bf16>(c, &dev, step, io, false, active, nullptr, true, ws, ws_bytes, (hipStream_t)stream, &hp);
}

rc_status rc_build_cache_hosted(rc_ctx *c, const rc_cache_view *cache, int32_t step, const rc_step_io *io,
                                void *staging, size_t staging_bytes, void *ws, size_t ws_bytes, void *stream) {
  g_err.clear();
  RC_CHECK(c, RC_ERR_INVALID_ARG, "ctx is null");
  RC_TRY(check_cache(c, cache, step));
  RC_TRY(check_io(c, io));
  RC_TRY(check_guided(io, cache->batch, nullptr));
  RC_CHECK((long)cache->batch * c->N <= (1L << 30), RC_ERR_SHAPE, "batch too large");
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  rc_cache_view dev{};
  HostPipe hp{};
  RC_TRY(check_hosted(c, cache, staging, staging_bytes, &dev, &hp));
  return run_step<bf16>(c, &dev, step, io, true, nullptr, nullptr, true, ws, ws_bytes, (hipStream_t)stream, &hp);
}

rc_status rc_localize_region(rc_ctx *c, const float *maps, int32_t batch, int32_t n_delta, float threshold,
                             int32_t radius, uint8_t *mask, int32_t *idx, int32_t *offsets, int32_t *offsets_host,
                             void *stream) {
  g_err.clear();
  RC_CHECK(c && maps && mask && idx && offsets, RC_ERR_INVALID_ARG, "null argument to rc_localize_region");
  RC_CHECK(batch >= 1 && batch <= 32767, RC_ERR_SHAPE, "batch %d out of range", batch);
  RC_CHECK(n_delta >= 1 && n_delta <= 8, RC_ERR_INVALID_ARG, "n_delta %d outside [1, 8]", n_delta);
  RC_CHECK(radius >= 0 && radius <= 4, RC_ERR_INVALID_ARG, "radius %d outside [0, 4]", radius);
  RC_CHECK(std::isfinite(threshold), RC_ERR_INVALID_ARG, "threshold is not finite");
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  hipStream_t s = (hipStream_t)stream;
  RC_TRY(timed(c, RC_KC_MISC, s, [&] {
    return rc::launch_localize(maps, batch, c->cfg.grid_h, c->cfg.grid_w, n_delta, threshold, radius, mask, s);
  }));
  RC_TRY(timed(c, RC_KC_MISC, s, [&] { return rc::launch_compact(mask, batch, c->N, idx, offsets, s); }));
  if (offsets_host) {
    RC_HIP(hipMemcpyAsync(offsets_host, offsets, sizeof(int32_t) * (batch + 1), hipMemcpyDeviceToHost, s));
    RC_HIP(hipStreamSynchronize(s));
  }
  return RC_OK;
}

size_t rc_maps_from_logits_scratch_bytes(int32_t n_layers, int32_t tokens, int32_t n_delta) {
  if (n_layers < 1 || tokens < 1 || n_delta < 1) return 0;
  return (size_t)n_layers * tokens * n_delta * sizeof(float);
}

rc_status rc_maps_from_logits(const void *logits, int32_t n_layers, int32_t heads, int32_t tokens, int32_t text_len,
                              const int32_t *delta_cols_host, int32_t n_delta, float *maps_out, void *partial,
                              size_t partial_bytes, void *stream) {
  g_err.clear();
  RC_TRY(check_maps_args(logits, n_layers, heads, tokens, text_len, delta_cols_host, n_delta, maps_out));
  RC_CHECK(partial, RC_ERR_INVALID_ARG, "null argument");
  const size_t need = rc_maps_from_logits_scratch_bytes(n_layers, tokens, n_delta);
  RC_CHECK(partial_bytes >= need, RC_ERR_CAPACITY, "scratch has %zu bytes, needs %zu", partial_bytes, need);
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  return launch_maps(logits, n_layers, heads, tokens, text_len, delta_cols_host, n_delta, maps_out, (float *)partial,
                     (hipStream_t)stream);
}

rc_status rc_maps_from_logits_noalloc(const void *logits, int32_t n_layers, int32_t heads, int32_t tokens,
                                      int32_t text_len, const int32_t *delta_cols_host, int32_t n_delta,
                                      float *maps_out, void *stream) {
  g_err.clear();
  RC_TRY(check_maps_args(logits, n_layers, heads, tokens, text_len, delta_cols_host, n_delta, maps_out));
  const size_t need = rc_maps_from_logits_scratch_bytes(n_layers, tokens, n_delta);
  RC_CHECK(need <= kStaticScratchBytes, RC_ERR_CAPACITY,
           "n_layers*tokens*n_delta*4 = %zu bytes exceeds the library's static scratch of %zu bytes", need,
           kStaticScratchBytes);
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  void *sp = nullptr;
  RC_TRY(static_scratch(&sp));
  return launch_maps(logits, n_layers, heads, tokens, text_len, delta_cols_host, n_delta, maps_out, (float *)sp,
                     (hipStream_t)stream);
}

rc_status rc_compact_mask(const uint8_t *mask, int32_t batch, int32_t tokens, int32_t *idx, int32_t *offsets,
                          int32_t *offsets_host, void *stream) {
  g_err.clear();
  RC_CHECK(mask && idx && offsets, RC_ERR_INVALID_ARG, "null argument to rc_compact_mask");
  RC_CHECK(batch >= 1 && batch <= 32767, RC_ERR_SHAPE, "batch %d out of range", batch);
  RC_CHECK(tokens >= 1 && tokens <= 65535, RC_ERR_SHAPE, "tokens %d out of range", tokens);
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  hipStream_t s = (hipStream_t)stream;
  RC_HIP(rc::launch_compact(mask, batch, tokens, idx, offsets, s));
  if (offsets_host) {
    RC_HIP(hipMemcpyAsync(offsets_host, offsets, sizeof(int32_t) * (batch + 1), hipMemcpyDeviceToHost, s));
    RC_HIP(hipStreamSynchronize(s));
  }
  return RC_OK;
}

rc_status rc_sync(void *stream) {
  g_err.clear();
  RC_CHECK(device_present(), RC_ERR_NO_DEVICE, "no HIP device");
  RC_HIP(hipStreamSynchronize((hipStream_t)stream));
  RC_HIP(hipGetLastError());
  return RC_OK;
}

rc_status rc_set_kernel_timing(rc_ctx *c, int32_t enable) {
  g_err.clear();
  RC_CHECK(c, RC_ERR_INVALID_ARG, "ctx is null");
  c->timing = enable != 0;
  c->recs.clear();
  c->pool_used = 0;
  return RC_OK;
}

rc_status rc_get_kernel_timing(rc_ctx *c, int32_t cls, double *total_ms, int64_t *launches) {
  g_err.clear();
  RC_CHECK(c && total_ms && launches, RC_ERR_INVALID_ARG, "null argument");
  RC_CHECK(cls >= 0 && cls < RC_KC_COUNT, RC_ERR_INVALID_ARG, "kernel class %d unknown", cls);
  double tot = 0.0;
  int64_t n = 0;
  for (const auto &r : c->recs) {
    if (r.cls != cls) continue;
    RC_HIP(hipEventSynchronize(r.b));
    float ms = 0.0f;
    RC_HIP(hipEventElapsedTime(&ms, r.a, r.b));
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return RC_OK;
}

}  // extern "C"
