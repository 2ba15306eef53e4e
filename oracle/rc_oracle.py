"""Plain float64 CPU oracle of the region-reuse DiT step.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Each function states the passage of the paper it follows.  Where the paper is
silent (model internals, sampler, threshold rule), the function states the
reading it takes; the same readings are listed in the design notes.

Conventions
-----------
* A chain is one independent edit sequence (one image).  Functions here work
  on one chain; tests loop over chains.
* Tokens are numbered row-major over the gh x gw patch grid: i = y*gw + x.
* Per-layer cache contents: K and V as [H, N, D] (head-major), hidden state
  H as [N, C].  The oracle keeps them in float64 and never rounds them.
* Attention-map buffers hold *sums* over heads and layers of the cross-
  attention probabilities of the delta text columns; the spatial vector of
  Sec. 3.2 is their mean, and the min-max normalisation used to threshold it
  is invariant to that positive scale.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "layer_norm", "modulate", "gelu_tanh", "silu", "softmax", "attention",
    "timestep_sinusoid", "timestep_embedding", "adaln_single", "layer_modulation",
    "final_modulation", "pos_embed_2d", "patchify", "patch_embed", "caption_projection",
    "text_kv", "cross_and_mlp", "block_dense", "block_reuse", "latent_to_patches", "patches_to_latent", "final_layer", "eps_from_output",
    "alphas_cumprod", "ddim_update", "dense_step", "reuse_step",
    "dense_block_tokens", "reuse_block_tokens", "maps_from_logits", "dilate",
    "compact", "localize", "cosine_similarity", "reuse_cutoff", "step_plan", "guided_noise", "guided_latent",
]

LN_EPS = 1e-6


def _f(x, dt=np.float64):
    return np.asarray(x, dtype=dt)


# ---------------------------------------------------------------------------
# elementwise pieces of the PixArt-alpha block (Sec. 4.1 backbone)
# ---------------------------------------------------------------------------

def layer_norm(x, eps: float = LN_EPS):
    """LayerNorm over the last axis without affine parameters; biased variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def modulate(x, shift, scale):
    """adaLN modulation x * (1 + scale) + shift."""
    return x * (1.0 + scale) + shift


def gelu_tanh(x):
    """GELU, tanh approximation."""
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def silu(x):
    return x / (1.0 + np.exp(-x))


def softmax(s, axis: int = -1):
    m = s.max(axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=axis, keepdims=True)


def attention(q, k, v, return_probs: bool = False):
    """Scaled dot-product attention per head.

    q: [R, H, D] queries, k and v: [N, H, D] keys/values.  Every query attends
    to all N keys with scale 1/sqrt(D) and a softmax over the keys.
    Returns O [R, H, D] (and P [H, R, N] if asked)."""
    R, Hh, D = q.shape
    out = np.empty_like(q)
    probs = np.empty((Hh, R, k.shape[0]), dtype=q.dtype) if return_probs else None
    scale = 1.0 / math.sqrt(D)
    for h in range(Hh):
        s = (q[:, h, :] @ k[:, h, :].T) * scale
        p = softmax(s, axis=-1)
        out[:, h, :] = p @ v[:, h, :]
        if return_probs:
            probs[h] = p
    return (out, probs) if return_probs else out


# ---------------------------------------------------------------------------
# conditioning: timestep embedding and adaLN-single (PixArt-alpha)
# ---------------------------------------------------------------------------

def timestep_sinusoid(t: float, dim: int = 256, max_period: float = 10000.0, dt=np.float64):
    """[cos(t f_k), sin(t f_k)] with f_k = max_period^(-k/(dim/2)), k < dim/2."""
    half = dim // 2
    freqs = np.exp(-math.log(max_period) * np.arange(half, dtype=dt) / half)
    args = dt(t) * freqs
    return np.concatenate([np.cos(args), np.sin(args)])


def timestep_embedding(W, t: float, dt=np.float64):
    """t_emb = W2 silu(W1 e(t) + b1) + b2."""
    e = timestep_sinusoid(t, dt=dt)
    h = silu(_f(W["temb_w1"], dt) @ e + _f(W["temb_b1"], dt))
    return _f(W["temb_w2"], dt) @ h + _f(W["temb_b2"], dt)


def adaln_single(W, t_emb, dt=np.float64):
    """t0 = W_tb silu(t_emb) + b_tb, reshaped to [6, C]; shared by all blocks."""
    C = t_emb.shape[0]
    t0 = _f(W["tblock_w"], dt) @ silu(t_emb) + _f(W["tblock_b"], dt)
    return t0.reshape(6, C)


def layer_modulation(lw, t0, dt=np.float64):
    """Per-block table plus t0, in the order
    (shift_1, scale_1, gate_1, shift_2, scale_2, gate_2)."""
    m = _f(lw["sst"], dt) + t0
    return tuple(m[i] for i in range(6))


def final_modulation(W, t_emb, dt=np.float64):
    """(shift, scale) of the final layer: its own 2-row table plus t_emb."""
    m = _f(W["fin_sst"], dt) + t_emb[None, :]
    return m[0], m[1]


# ---------------------------------------------------------------------------
# token embedding and text preparation
# ---------------------------------------------------------------------------

def pos_embed_2d(gh: int, gw: int, C: int, dt=np.float64):
    """Fixed 2-D sin-cos table [gh*gw, C]: the first C/2 columns encode the
    column coordinate x, the last C/2 the row coordinate y; each half is
    [sin(pos w_k), cos(pos w_k)] with w_k = 10000^(-k/(C/4)), k < C/4."""
    quarter = C // 4
    w = 1.0 / (10000.0 ** (np.arange(quarter, dtype=dt) / quarter))
    ys, xs = np.divmod(np.arange(gh * gw), gw)

    def enc(pos):
        a = pos.astype(dt)[:, None] * w[None, :]
        return np.concatenate([np.sin(a), np.cos(a)], axis=1)

    return np.concatenate([enc(xs), enc(ys)], axis=1)


def patchify(latent, p: int):
    """latent [c, gh*p, gw*p] -> [N, c*p*p]; entry index c*p*p + pi*p + qi holds
    latent[c, y*p + pi, x*p + qi] of token (y, x)."""
    c, Hh, Ww = latent.shape
    gh, gw = Hh // p, Ww // p
    t = latent.reshape(c, gh, p, gw, p).transpose(1, 3, 0, 2, 4)
    return t.reshape(gh * gw, c * p * p)


def patch_embed(W, latent, gh: int, gw: int, p: int, dt=np.float64):
    """Token embedding of every patch: patchify . W_pe^T + b_pe + pos."""
    C = W["pe_b"].shape[0]
    x = patchify(_f(latent, dt), p)
    return x @ _f(W["pe_w"], dt).T + _f(W["pe_b"], dt) + pos_embed_2d(gh, gw, C, dt)


def caption_projection(W, txt, dt=np.float64):
    """y = W2 gelu_tanh(W1 txt + b1) + b2, per text token."""
    h = gelu_tanh(_f(txt, dt) @ _f(W["cap_w1"], dt).T + _f(W["cap_b1"], dt))
    return h @ _f(W["cap_w2"], dt).T + _f(W["cap_b2"], dt)


def text_kv(lw, y, heads: int, dt=np.float64):
    """Cross-attention keys and values of the text tokens for one block:
    [K | V] = y W_kv^T + b, each reshaped to [M, H, D]."""
    M, C = y.shape
    kv = _f(y, dt) @ _f(lw["xkv_w"], dt).T + _f(lw["xkv_b"], dt)
    return kv[:, :C].reshape(M, heads, C // heads), kv[:, C:].reshape(M, heads, C // heads)


# ---------------------------------------------------------------------------
# transformer block: dense (every token) and region-reuse (active tokens)
# ---------------------------------------------------------------------------

def cross_and_mlp(lw, X, mod, textK, textV, heads, delta, dt):
    """Cross-attention to the text (residual, no norm, no gate) followed by the
    gated MLP branch.  Returns the new X and, if `delta` is given, the
    per-token sums over heads of the attention probability on each delta
    column (the cross-attention map of Sec. 3.2)."""
    R, C = X.shape
    D = C // heads
    _, _, _, sh2, sc2, g2 = mod
    qc = (X @ _f(lw["xq_w"], dt).T + _f(lw["xq_b"], dt)).reshape(R, heads, D)
    oc, pc = attention(qc, textK, textV, return_probs=True)
    X = X + oc.reshape(R, C) @ _f(lw["xproj_w"], dt).T + _f(lw["xproj_b"], dt)
    maps = None
    if delta is not None:
        maps = pc[:, :, np.asarray(delta)].sum(axis=0)  # [R, n_delta]
    h2 = modulate(layer_norm(X), sh2, sc2)
    f = gelu_tanh(h2 @ _f(lw["fc1_w"], dt).T + _f(lw["fc1_b"], dt))
    X = X + g2 * (f @ _f(lw["fc2_w"], dt).T + _f(lw["fc2_b"], dt))
    return X, maps


def block_dense(lw, X, mod, textK, textV, heads: int, delta=None, dt=np.float64):
    """Full PixArt-alpha block over all N tokens (the dense computation that
    region reuse avoids).  Returns (X_out, K [H,N,D], V [H,N,D], maps)."""
    N, C = X.shape
    D = C // heads
    sh1, sc1, g1 = mod[0], mod[1], mod[2]
    h = modulate(layer_norm(X), sh1, sc1)
    qkv = (h @ _f(lw["qkv_w"], dt).T + _f(lw["qkv_b"], dt)).reshape(N, 3, heads, D)
    q, k, v = qkv[:, 0], qkv[:, 1], qkv[:, 2]
    o = attention(q, k, v)
    X = X + g1 * (o.reshape(N, C) @ _f(lw["proj_w"], dt).T + _f(lw["proj_b"], dt))
    X, maps = cross_and_mlp(lw, X, mod, textK, textV, heads, delta, dt)
    return X, k.transpose(1, 0, 2).copy(), v.transpose(1, 0, 2).copy(), maps


def block_reuse(lw, X_act, idx, mod, textK, textV, cacheK, cacheV, cacheH, heads: int,
                delta=None, dt=np.float64):
    """Region-level sparse attention block (Sec. 3.3).

    Only the active hidden states X_act [R, C] (tokens `idx`) are instantiated.
    Their keys and values overwrite the cached ones at their positions before
    attention (Sec. 3.4, Kernel Fusing); the active queries then attend over
    the keys and values of all N tokens, fresh for active tokens and cached
    for the rest.  The active outputs are merged into the cached hidden state
    (Sec. 3.3); inactive rows are taken from the cache unchanged.

    Returns (X_out [R,C], K [H,N,D], V [H,N,D], H [N,C], maps)."""
    R, C = X_act.shape
    D = C // heads
    idx = np.asarray(idx, dtype=np.int64)
    sh1, sc1, g1 = mod[0], mod[1], mod[2]
    h = modulate(layer_norm(X_act), sh1, sc1)
    qkv = (h @ _f(lw["qkv_w"], dt).T + _f(lw["qkv_b"], dt)).reshape(R, 3, heads, D)
    q, k, v = qkv[:, 0], qkv[:, 1], qkv[:, 2]
    K = _f(cacheK, dt).copy()
    V = _f(cacheV, dt).copy()
    K[:, idx, :] = k.transpose(1, 0, 2)
    V[:, idx, :] = v.transpose(1, 0, 2)
    o = attention(q, K.transpose(1, 0, 2), V.transpose(1, 0, 2))
    X = X_act + g1 * (o.reshape(R, C) @ _f(lw["proj_w"], dt).T + _f(lw["proj_b"], dt))
    X, maps = cross_and_mlp(lw, X, mod, textK, textV, heads, delta, dt)
    Hm = _f(cacheH, dt).copy()
    Hm[idx] = X
    return X, K, V, Hm, maps


# ---------------------------------------------------------------------------
# final layer and sampler
# ---------------------------------------------------------------------------

def final_layer(W, X, t_emb, dt=np.float64):
    """(LN(X)(1 + scale_f) + shift_f) W_f^T + b_f -> [R, p*p*out_ch]."""
    sh, sc = final_modulation(W, t_emb, dt)
    return modulate(layer_norm(X), sh, sc) @ _f(W["fin_w"], dt).T + _f(W["fin_b"], dt)


def eps_from_output(out, p: int, out_ch: int, latent_ch: int):
    """Noise prediction per token as [R, latent_ch, p, p]: output column
    (pi*p + qi)*out_ch + c holds channel c of pixel (pi, qi) of the patch; the
    first latent_ch channels are the noise, the rest the learned variance."""
    R = out.shape[0]
    o = out.reshape(R, p, p, out_ch)
    return o[..., :latent_ch].transpose(0, 3, 1, 2)


def alphas_cumprod(n: int = 1000, beta_start: float = 1e-4, beta_end: float = 0.02):
    """DDPM linear-beta schedule, cumulative product of (1 - beta)."""
    betas = np.linspace(beta_start, beta_end, n, dtype=np.float64)
    return np.cumprod(1.0 - betas)


def ddim_update(x, eps, abar_t: float, abar_next: float):
    """Deterministic DDIM step (eta = 0):
    x0 = (x - sqrt(1 - a_t) eps) / sqrt(a_t);  x' = sqrt(a') x0 + sqrt(1 - a') eps."""
    x0 = (x - math.sqrt(1.0 - abar_t) * eps) / math.sqrt(abar_t)
    return math.sqrt(abar_next) * x0 + math.sqrt(1.0 - abar_next) * eps


def _abar_pair(t: int, t_next: int):
    ac = alphas_cumprod()
    return float(ac[t]), (float(ac[t_next]) if t_next >= 0 else 1.0)


def latent_to_patches(latent, p):
    c, Hh, Ww = latent.shape
    gh, gw = Hh // p, Ww // p
    return latent.reshape(c, gh, p, gw, p).transpose(1, 3, 0, 2, 4).reshape(gh * gw, c, p, p)


def patches_to_latent(patches, gh, gw):
    N, c, p, _ = patches.shape
    return patches.reshape(gh, gw, c, p, p).transpose(2, 0, 3, 1, 4).reshape(c, gh * p, gw * p)


# ---------------------------------------------------------------------------
# whole denoising steps (one chain)
# ---------------------------------------------------------------------------

def dense_step(shape, W, latent, t: int, t_next: int, textKV, delta=None, dt=np.float64):
    """One dense denoising step of one chain (every token computed).  This is
    the step that builds the cache pool of Sec. 3.2.

    latent [c, H, W]; textKV: list over layers of (K_t, V_t) [M, H, D].
    Returns dict: K, V [L, H, N, D]; H [L, N, C]; latent_next; maps [N, n_delta]
    (sums over heads and layers) or None; eps [N, c, p, p]."""
    s = shape
    p = s.patch
    t_emb = timestep_embedding(W, t, dt)
    t0 = adaln_single(W, t_emb, dt)
    X = patch_embed(W, latent, s.grid_h, s.grid_w, p, dt)
    Ks, Vs, Hs = [], [], []
    maps = None
    for l, lw in enumerate(W["layers"]):
        mod = layer_modulation(lw, t0, dt)
        X, K, V, m = block_dense(lw, X, mod, textKV[l][0], textKV[l][1], s.heads, delta, dt)
        Ks.append(K); Vs.append(V); Hs.append(X.copy())
        if m is not None:
            maps = m if maps is None else maps + m
    out = final_layer(W, X, t_emb, dt)
    eps = eps_from_output(out, p, s.out_ch, s.latent_ch)
    a_t, a_n = _abar_pair(t, t_next)
    x_patches = latent_to_patches(_f(latent, dt), p)
    latent_next = patches_to_latent(ddim_update(x_patches, eps, a_t, a_n), s.grid_h, s.grid_w)
    return dict(K=np.stack(Ks), V=np.stack(Vs), H=np.stack(Hs), latent_next=latent_next,
                maps=maps, eps=eps)


def reuse_step(shape, W, latent, t: int, t_next: int, textKV, idx, cache,
               latent_cached_next, delta=None, dt=np.float64):
    """One region-reuse denoising step of one chain (Sec. 3.3).

    Only the active tokens `idx` (ascending) are embedded and run through the
    blocks; each block reads and updates the cache slot `cache` (dict of
    K, V [L, H, N, D] and H [L, N, C] for this step).  After the last block
    the active tokens' noise prediction updates their patches of the latent;
    inactive patches take the cached trajectory's latent of the next step.

    Returns dict: K, V, H (the updated slot), X (active final hidden state),
    latent_next, maps (rows of inactive tokens are zero) and eps [R, c, p, p]."""
    s = shape
    p = s.patch
    idx = np.asarray(idx, dtype=np.int64)
    t_emb = timestep_embedding(W, t, dt)
    t0 = adaln_single(W, t_emb, dt)
    X = patch_embed(W, latent, s.grid_h, s.grid_w, p, dt)[idx]
    Ks, Vs, Hs = [], [], []
    maps = None
    for l, lw in enumerate(W["layers"]):
        mod = layer_modulation(lw, t0, dt)
        X, K, V, Hm, m = block_reuse(lw, X, idx, mod, textKV[l][0], textKV[l][1],
                                     cache["K"][l], cache["V"][l], cache["H"][l], s.heads, delta, dt)
        Ks.append(K); Vs.append(V); Hs.append(Hm)
        if m is not None:
            full = np.zeros((s.tokens, m.shape[1]), dtype=dt)
            full[idx] = m
            maps = full if maps is None else maps + full
    a_t, a_n = _abar_pair(t, t_next)
    lat_next = latent_to_patches(_f(latent_cached_next, dt), p).copy()
    eps = None
    if idx.size:
        out = final_layer(W, X, t_emb, dt)
        eps = eps_from_output(out, p, s.out_ch, s.latent_ch)
        x_patches = latent_to_patches(_f(latent, dt), p)[idx]
        lat_next[idx] = ddim_update(x_patches, eps, a_t, a_n)
    return dict(K=np.stack(Ks), V=np.stack(Vs), H=np.stack(Hs), X=X,
                latent_next=patches_to_latent(lat_next, s.grid_h, s.grid_w), maps=maps, eps=eps)


def guided_noise(eps_cond, eps_uncond, scale: float):
    """Classifier-free guidance of PixArt-alpha's sampler (not part of the
    method): eps_u + scale (eps_c - eps_u)."""
    return eps_uncond + scale * (eps_cond - eps_uncond)


def guided_latent(shape, latent, latent_cached_next, idx, eps_cond, eps_uncond, scale: float, t: int,
                  t_next: int, dt=np.float64):
    """Latent after one guided step of the tokens `idx`: their patches take the
    DDIM update with the guided noise of the two branches' predictions
    (eps [R, c, p, p] from reuse_step or dense_step); the other patches take
    the cached trajectory's next latent."""
    p = shape.patch
    idx = np.asarray(idx, dtype=np.int64)
    a_t, a_n = _abar_pair(t, t_next)
    lat_next = latent_to_patches(_f(latent_cached_next, dt), p).copy()
    if idx.size:
        x = latent_to_patches(_f(latent, dt), p)[idx]
        lat_next[idx] = ddim_update(x, guided_noise(eps_cond, eps_uncond, scale), a_t, a_n)
    return patches_to_latent(lat_next, shape.grid_h, shape.grid_w)


def _token_mode_mod(W, t_vec, dt):
    t0 = adaln_single(W, _f(t_vec, dt), dt)
    return layer_modulation(W["layers"][0], t0, dt)


def dense_block_tokens(shape, W, X, t_vec, text, delta=None, dt=np.float64):
    """Single-block form: hidden tokens X [N, C] in, block output out; the
    modulation comes from the given timestep vector through adaLN-single and
    the text tokens are already C-dimensional (no caption projection)."""
    lw = W["layers"][0]
    tk, tv = text_kv(lw, _f(text, dt), shape.heads, dt)
    return block_dense(lw, _f(X, dt), _token_mode_mod(W, t_vec, dt), tk, tv, shape.heads, delta, dt)


def reuse_block_tokens(shape, W, X_new, idx, t_vec, text, cacheK, cacheV, cacheH,
                       delta=None, dt=np.float64):
    """Single-block region-reuse form of `dense_block_tokens`; X_new [N, C] is
    the new turn's token set, of which rows `idx` are active."""
    lw = W["layers"][0]
    tk, tv = text_kv(lw, _f(text, dt), shape.heads, dt)
    Xa = _f(X_new, dt)[np.asarray(idx, dtype=np.int64)]
    return block_reuse(lw, Xa, idx, _token_mode_mod(W, t_vec, dt), tk, tv,
                       cacheK, cacheV, cacheH, shape.heads, delta, dt)


# ---------------------------------------------------------------------------
# localisation (Sec. 3.2)
# ---------------------------------------------------------------------------

def maps_from_logits(Z, delta, dt=np.float64):
    """Cross-attention maps from raw logits Z [L, H, N, M]: the softmax over the
    M text tokens, summed over heads and layers, at each delta column.
    Returns sums [N, n_delta] (divide by L*H for the mean)."""
    L, Hh, N, M = Z.shape
    acc = np.zeros((N, len(delta)), dtype=dt)
    cols = np.asarray(delta)
    for l in range(L):
        p = softmax(_f(Z[l], dt), axis=-1)  # [H, N, M]
        acc += p[:, :, cols].sum(axis=0)
    return acc


def dilate(mask2d, radius: int = 1):
    """Binary dilation by a (2r+1)x(2r+1) square, clipped at the border."""
    gh, gw = mask2d.shape
    out = np.zeros_like(mask2d, dtype=bool)
    for y in range(gh):
        for x in range(gw):
            y0, y1 = max(0, y - radius), min(gh, y + radius + 1)
            x0, x1 = max(0, x - radius), min(gw, x + radius + 1)
            out[y, x] = bool(mask2d[y0:y1, x0:x1].any())
    return out


def compact(masks):
    """Stable compaction of per-chain masks [B, N] into chain-local ascending
    token lists concatenated over chains, plus offsets [B+1]."""
    idx: List[int] = []
    offsets = [0]
    for b in range(masks.shape[0]):
        for i in range(masks.shape[1]):
            if masks[b, i]:
                idx.append(i)
        offsets.append(len(idx))
    return np.array(idx, dtype=np.int32), np.array(offsets, dtype=np.int32)


def localize(maps, gh: int, gw: int, n_avg: float = 1.0, theta: float = 0.3,
             radius: int = 1, return_scores: bool = False):
    """Edit region of Sec. 3.2 from the delta-token maps of one chain.

    a_j = maps[:, j] / n_avg is the spatial attention vector of delta token j.
    The threshold theta_j derived from a_j is a fraction theta of its range:
    token i belongs to the region of j when (a_j(i) - min a_j)/(max a_j - min
    a_j) >= theta (a constant a_j selects nothing).  The edit region is the
    union over j, dilated by `radius` tokens on the grid.
    Returns (mask u8 [N], idx i32 ascending[, scores [N, n_delta]])."""
    a = _f(maps) / n_avg
    N, J = a.shape
    sel = np.zeros(N, dtype=bool)
    scores = np.full((N, J), -np.inf)
    for j in range(J):
        lo, hi = a[:, j].min(), a[:, j].max()
        if hi > lo:
            scores[:, j] = (a[:, j] - lo) / (hi - lo)
            sel |= scores[:, j] >= theta
    m = dilate(sel.reshape(gh, gw), radius).reshape(-1)
    mask = m.astype(np.uint8)
    idx, _ = compact(mask[None, :])
    return (mask, idx, scores) if return_scores else (mask, idx)


# ---------------------------------------------------------------------------
# reuse schedule (Sec. 3.3, Eq. 1 and Eq. 2) -- host-side control
# ---------------------------------------------------------------------------

def cosine_similarity(e_before, e_after) -> float:
    """Eq. 1: s = cos(e(tau-), e(tau+))."""
    a, b = _f(e_before).ravel(), _f(e_after).ravel()
    return float(a @ b / (np.sqrt(a @ a) * np.sqrt(b @ b)))


def reuse_cutoff(T: int, s: float, tau_s: float, rho: float = 0.2) -> int:
    """Eq. 2: T_reuse = T when s >= tau_s, else floor(rho T)."""
    return T if s >= tau_s else int(math.floor(rho * T))


def step_plan(T: int, rho: float = 0.2, reading: str = "dense_then_reuse",
              s: Optional[float] = None, tau_s: float = 0.8) -> List[str]:
    """Per-step plan of one editing turn for the edited region.

    reading="dense_then_reuse": the first floor(rho T) steps run dense and the
    remaining steps run region reuse.
    reading="paper": Eq. 2 -- the region reuses the cache (its rows are copied
    unchanged, 'copy') for the first T_reuse steps and is recomputed with
    region reuse ('reuse') after that."""
    if reading == "dense_then_reuse":
        k = int(math.floor(rho * T))
        return ["dense"] * k + ["reuse"] * (T - k)
    if reading == "paper":
        tr = reuse_cutoff(T, 0.0 if s is None else s, tau_s, rho)
        return ["copy"] * tr + ["reuse"] * (T - tr)
    raise ValueError(reading)
