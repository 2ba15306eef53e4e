"""Seeded synthetic inputs for the region-reuse DiT step.

This module only *draws* inputs: weights, latents, text features, masks,
timestep grids and cache contents.  It holds none of the method's arithmetic
(no normalisation, attention, embedding or sampler math), so that both the
CPU oracle and the HIP path can consume the same inputs without sharing any
computation.

Shapes follow the PixArt-alpha backbone the paper evaluates on (Sec. 4.1):
hidden 1152, 16 heads x 72, MLP 4608, 120 text tokens, 2x2 patches over a
4-channel latent, 8 output channels (noise + variance).

Every stream is `numpy.random.default_rng([seed, stream_id])`, so one seed
fixes every tensor and changing one generator never shifts another.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np

# stream ids (one independent generator per kind of tensor)
_S_WEIGHTS, _S_PREV, _S_NEW, _S_TEXT, _S_MASK, _S_TVEC, _S_DELTA, _S_CACHE, _S_LOGITS = range(9)


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Model and workload shape.  `token_mode` is the single-block form that
    takes hidden tokens and a timestep vector directly (no patch embedding,
    caption projection, final layer or sampler)."""

    hidden: int = 1152
    heads: int = 16
    head_dim: int = 72
    mlp: int = 4608
    layers: int = 28
    text_len: int = 120
    text_dim: int = 4096
    grid_h: int = 32
    grid_w: int = 32
    latent_ch: int = 4
    patch: int = 2
    out_ch: int = 8
    dtype: str = "bf16"  # "f32" or "bf16": storage type of weights and cache
    token_mode: bool = False

    @property
    def tokens(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def latent_hw(self):
        return self.grid_h * self.patch, self.grid_w * self.patch


def shape_c1() -> ModelShape:
    """One fp32 block, 16x16 token grid, 1152-d text tokens."""
    return ModelShape(layers=1, text_dim=1152, grid_h=16, grid_w=16, dtype="f32", token_mode=True)


def shape_c2() -> ModelShape:
    """28 blocks at 512 px: latent 4x64x64 -> 32x32 tokens, bf16."""
    return ModelShape(layers=28, grid_h=32, grid_w=32, dtype="bf16")


def shape_c3() -> ModelShape:
    """28 blocks at 1024 px: latent 4x128x128 -> 64x64 tokens, bf16."""
    return ModelShape(layers=28, grid_h=64, grid_w=64, dtype="bf16")


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even) and return
    them as float32, so that the value handed to the GPU as bf16 and the value
    the oracle reads are the same number."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).reshape(a.shape)


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream)])


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    a = a.astype(np.float32, copy=False)
    return bf16_round(a) if dtype == "bf16" else a


LAYER_MATS = ("qkv_w", "proj_w", "xq_w", "xkv_w", "xproj_w", "fc1_w", "fc2_w")
LAYER_VECS = ("qkv_b", "proj_b", "xq_b", "xkv_b", "xproj_b", "fc1_b", "fc2_b")


def layer_weight_shapes(s: ModelShape) -> Dict[str, tuple]:
    C, F = s.hidden, s.mlp
    return {
        "qkv_w": (3 * C, C), "qkv_b": (3 * C,),
        "proj_w": (C, C), "proj_b": (C,),
        "xq_w": (C, C), "xq_b": (C,),
        "xkv_w": (2 * C, C), "xkv_b": (2 * C,),
        "xproj_w": (C, C), "xproj_b": (C,),
        "fc1_w": (F, C), "fc1_b": (F,),
        "fc2_w": (C, F), "fc2_b": (C,),
        "sst": (6, C),
    }


def global_weight_shapes(s: ModelShape) -> Dict[str, tuple]:
    C = s.hidden
    pin = s.latent_ch * s.patch * s.patch
    pout = s.out_ch * s.patch * s.patch
    return {
        "pe_w": (C, pin), "pe_b": (C,),
        "temb_w1": (C, 256), "temb_b1": (C,),
        "temb_w2": (C, C), "temb_b2": (C,),
        "tblock_w": (6 * C, C), "tblock_b": (6 * C,),
        "cap_w1": (C, s.text_dim), "cap_b1": (C,),
        "cap_w2": (C, C), "cap_b2": (C,),
        "fin_w": (pout, C), "fin_b": (pout,),
        "fin_sst": (2, C),
    }


def make_weights(s: ModelShape, seed: int = 0, std: float = 0.02,
                 stress: bool = False) -> Dict[str, object]:
    """Random-init weights ~N(0, std) for every matrix, bias and modulation
    table, stored as float32 holding bf16-exact values when `s.dtype` is bf16.

    `stress=True` draws a "peaky" variant: the self- and cross-attention query
    and key projections are scaled by 3 (attention logits with a standard
    deviation of about 4 instead of 0.5) and the gate rows of every modulation
    table are shifted by +1 (gates near 1), so that attention and every gated
    branch move the hidden state by O(1) rather than O(std)."""
    rng = _rng(seed, _S_WEIGHTS)
    C = s.hidden
    layers: List[Dict[str, np.ndarray]] = []
    for _ in range(s.layers):
        lw = {}
        for name, shp in layer_weight_shapes(s).items():
            a = rng.standard_normal(shp, dtype=np.float32) * np.float32(std)
            if stress and name == "qkv_w":
                a[: 2 * C] *= 3.0
            if stress and name in ("xq_w", "xkv_w"):
                a[:C] *= 3.0
            if stress and name == "sst":
                a[2] += 1.0
                a[5] += 1.0
            # matrices are handed to the GPU in the storage type, vectors and
            # modulation tables in float32; the values are the same either way
            lw[name] = _store(a, s.dtype)
        layers.append(lw)
    g = {}
    for name, shp in global_weight_shapes(s).items():
        a = rng.standard_normal(shp, dtype=np.float32) * np.float32(std)
        g[name] = _store(a, s.dtype)
    g["layers"] = layers
    return g


def rect_mask(gh: int, gw: int, rh: int, rw: int, y0: int, x0: int) -> np.ndarray:
    m = np.zeros((gh, gw), dtype=np.uint8)
    m[y0:y0 + rh, x0:x0 + rw] = 1
    return m.reshape(-1)


def random_aligned_rect_mask(gh: int, gw: int, count: int, rng: np.random.Generator,
                             align: int = 4) -> np.ndarray:
    """A rectangle of `count` tokens whose sides and origin are multiples of
    `align` tokens, drawn uniformly among the shapes that fit."""
    shapes = []
    for rh in range(align, gh + 1, align):
        if count % rh == 0:
            rw = count // rh
            if rw % align == 0 and rw <= gw:
                shapes.append((rh, rw))
    rh, rw = shapes[int(rng.integers(len(shapes)))]
    y0 = int(rng.integers((gh - rh) // align + 1)) * align
    x0 = int(rng.integers((gw - rw) // align + 1)) * align
    return rect_mask(gh, gw, rh, rw, y0, x0)


def blob_mask(gh: int, gw: int, frac: float, n_blobs: int, rng: np.random.Generator) -> np.ndarray:
    """`n_blobs` seeded ellipses; the active set is exactly the `round(frac*N)`
    tokens with the largest ellipse field max_b(1 - d_b^2), ties broken by
    lower token index, so the count is exact and seed-stable."""
    N = gh * gw
    yy, xx = np.meshgrid(np.arange(gh, dtype=np.float64), np.arange(gw, dtype=np.float64), indexing="ij")
    field = np.full((gh, gw), -np.inf)
    for _ in range(n_blobs):
        cy = rng.uniform(0.15, 0.85) * gh
        cx = rng.uniform(0.15, 0.85) * gw
        ry = rng.uniform(0.08, 0.25) * gh
        rx = rng.uniform(0.08, 0.25) * gw
        th = rng.uniform(0, math.pi)
        dy, dx = yy - cy, xx - cx
        u = (dx * math.cos(th) + dy * math.sin(th)) / rx
        v = (-dx * math.sin(th) + dy * math.cos(th)) / ry
        field = np.maximum(field, 1.0 - (u * u + v * v))
    k = int(round(frac * N))
    order = np.lexsort((np.arange(N), -field.reshape(-1)))
    m = np.zeros(N, dtype=np.uint8)
    m[order[:k]] = 1
    return m


def c3_edit_region(seed: int = 0, frac=None):
    """The 1024 px edit region of the benchmark workload: a seeded active
    fraction in [0.10, 0.20] (unless `frac` is given) spread over 1-3 seeded
    elliptical blobs of the 64 x 64 token grid.  Returns (mask, frac, n_blobs)."""
    rng = np.random.default_rng([seed, 4242])
    f = float(rng.uniform(0.10, 0.20))
    if frac is not None:
        f = float(frac)
    n_blobs = int(rng.integers(1, 4))
    return blob_mask(64, 64, f, n_blobs, rng), f, n_blobs


def sweep_regions(seed: int, frac: float, chains: int = 4):
    """Active token lists of the batch active-fraction workload at 1024 px:
    per chain a blob mask of 1-3 seeded blobs covering `frac` of the 64 x 64
    grid.  Returns a list of ascending index arrays."""
    rng = np.random.default_rng([seed, int(frac * 1000)])
    return [np.flatnonzero(blob_mask(64, 64, frac, int(rng.integers(1, 4)), rng)) for _ in range(chains)]


def resolution_region(seed: int, g: int, frac: float = 0.15):
    """Active token list of the resolution workload on a g x g token grid
    (g = 32, 64, 128 for 512, 1024, 2048 px): two seeded blobs covering
    `frac` of the grid."""
    rng = np.random.default_rng([seed, g * 16])
    return np.flatnonzero(blob_mask(g, g, frac, 2, rng))


def timestep_grid(T: int, t_max: int = 999) -> np.ndarray:
    """The sampler's integer timesteps, linearly spaced from t_max down to 0."""
    return np.round(np.linspace(t_max, 0, T)).astype(np.int64)


def make_c1(seed: int = 0) -> Dict[str, object]:
    """One fp32 block over 256 tokens: previous/new token sets, text tokens,
    a timestep vector, a 64-token 4-aligned rectangle mask and 3 delta
    columns."""
    s = shape_c1()
    N, C = s.tokens, s.hidden
    x_prev = _rng(seed, _S_PREV).standard_normal((N, C), dtype=np.float32)
    mask = random_aligned_rect_mask(s.grid_h, s.grid_w, 64, _rng(seed, _S_MASK))
    x_new = x_prev.copy()
    redraw = _rng(seed, _S_NEW).standard_normal((N, C), dtype=np.float32)
    x_new[mask.astype(bool)] = redraw[mask.astype(bool)]
    text = _rng(seed, _S_TEXT).standard_normal((s.text_len, C), dtype=np.float32)
    t_vec = _rng(seed, _S_TVEC).standard_normal((C,), dtype=np.float32)
    delta = np.sort(_rng(seed, _S_DELTA).choice(s.text_len, size=3, replace=False)).astype(np.int32)
    return dict(shape=s, weights=make_weights(s, seed), x_prev=x_prev, x_new=x_new,
                text=text, t_vec=t_vec, mask=mask, delta=delta)


def make_text(s: ModelShape, batch: int, seed: int, stream: int = _S_TEXT) -> np.ndarray:
    t = _rng(seed, stream).standard_normal((batch, s.text_len, s.text_dim), dtype=np.float32)
    return _store(t, s.dtype)


def edit_text(s: ModelShape, text: np.ndarray, n_delta: int, seed: int):
    """Redraw `n_delta` token rows of each prompt; return the new text and the
    sorted delta columns (shared by all chains)."""
    rng = _rng(seed, _S_DELTA)
    delta = np.sort(rng.choice(s.text_len, size=n_delta, replace=False)).astype(np.int32)
    new = text.copy()
    new[:, delta] = _store(rng.standard_normal((text.shape[0], n_delta, s.text_dim), dtype=np.float32), s.dtype)
    return new, delta


def make_latent(s: ModelShape, batch: int, seed: int, stream: int = _S_PREV) -> np.ndarray:
    H, W = s.latent_hw
    return _rng(seed, stream).standard_normal((batch, s.latent_ch, H, W), dtype=np.float32)


def redraw_masked_patches(s: ModelShape, latent: np.ndarray, masks: np.ndarray, seed: int) -> np.ndarray:
    """New-turn latent: the patches under each chain's mask redrawn, the rest
    kept (masks: [B, N] u8)."""
    out = latent.copy()
    fresh = _rng(seed, _S_NEW).standard_normal(latent.shape, dtype=np.float32)
    p = s.patch
    for b in range(latent.shape[0]):
        m = masks[b].reshape(s.grid_h, s.grid_w).astype(bool)
        pm = np.repeat(np.repeat(m, p, axis=0), p, axis=1)
        out[b][:, pm] = fresh[b][:, pm]
    return out


def make_cache_slot(s: ModelShape, batch: int, seed: int, stream_offset: int = 0,
                    kv_std: float = 1.0, h_std: float = 1.0) -> Dict[str, np.ndarray]:
    """A synthetic cache slot for one step: per layer K and V as [B,H,N,D] and
    the block-output hidden state as [B,N,C], drawn N(0, std) and rounded to
    the storage type.  Stands in for a previous turn's trajectory where
    computing that trajectory is not the point of a test."""
    rng = _rng(seed, _S_CACHE * 1000 + stream_offset)
    L, N, C, Hh, D = s.layers, s.tokens, s.hidden, s.heads, s.head_dim
    K = _store(rng.standard_normal((L, batch, Hh, N, D), dtype=np.float32) * np.float32(kv_std), s.dtype)
    V = _store(rng.standard_normal((L, batch, Hh, N, D), dtype=np.float32) * np.float32(kv_std), s.dtype)
    Hs = _store(rng.standard_normal((L, batch, N, C), dtype=np.float32) * np.float32(h_std), s.dtype)
    return dict(K=K, V=V, H=Hs)


def make_logits(n_layers: int, heads: int, tokens: int, text_len: int, gh: int, gw: int,
                n_delta: int, seed: int, boost: float = 3.0, frac: float = 0.1):
    """Localisation input: bf16-exact logits ~N(0,1) of shape
    [layers, heads, tokens, text_len], with `boost` added to the delta columns
    over one seeded elliptical blob.  Returns (logits f32, delta i32, blob u8)."""
    rng = _rng(seed, _S_LOGITS)
    Z = rng.standard_normal((n_layers, heads, tokens, text_len), dtype=np.float32)
    delta = np.sort(rng.choice(text_len, size=n_delta, replace=False)).astype(np.int32)
    blob = blob_mask(gh, gw, frac, 1, rng)
    sel = np.flatnonzero(blob)
    for j in delta:
        Z[:, :, sel, j] += np.float32(boost)
    return bf16_round(Z), delta, blob


def planted_maps(tokens: int, n_delta: int, gh: int, gw: int, seed: int, frac: float = 0.1):
    """Map sums [tokens, n_delta] with a seeded blob of high values per column."""
    rng = _rng(seed, _S_LOGITS + 100)
    maps = rng.uniform(0.0, 1.0, (tokens, n_delta)).astype(np.float32)
    blob = blob_mask(gh, gw, frac, 1, rng)
    maps[blob.astype(bool)] += 4.0
    return maps, blob
