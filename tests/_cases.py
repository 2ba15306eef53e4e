"""Shared set-up of GPU parity cases: draw inputs with `synth`, run the HIP
path through the C ABI, run the oracle on the same inputs, compare."""
from __future__ import annotations

import functools

import numpy as np
import torch

import oracle as O
import synth


@functools.lru_cache(maxsize=4)
def weights(shape, seed, stress=False):
    """Seeded weights, drawn once per session for each (shape, seed, stress)."""
    return synth.make_weights(shape, seed=seed, stress=stress)


def relerr(gpu, ref) -> float:
    """Normwise relative error max|gpu - ref| / max|ref|."""
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if r.size == 0:
        return 0.0
    return float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))


def tol(shape) -> float:
    return 2e-2 if shape.dtype == "bf16" else 1e-4


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def oracle_text_kv(shape, W, txt_b):
    if shape.token_mode:
        y = np.asarray(txt_b, np.float64)
    else:
        y = O.caption_projection(W, txt_b)
    return [O.text_kv(lw, y, shape.heads) for lw in W["layers"]]


def upload_slot(model, cache, t, slot):
    """slot: dict K, V [L, B, H, N, D]; H [L, B, N, C] (float32 arrays)."""
    L, B = slot["K"].shape[:2]
    for l in range(L):
        for b in range(B):
            cache.K(b, t, l).copy_(model.to_storage(slot["K"][l, b]))
            cache.V(b, t, l).copy_(model.to_storage(slot["V"][l, b]))
            cache.H(b, t, l).copy_(model.to_storage(slot["H"][l, b]))


def download_slot(cache, t, L, B):
    K = np.stack([np.stack([to_np(cache.K(b, t, l)) for b in range(B)]) for l in range(L)])
    V = np.stack([np.stack([to_np(cache.V(b, t, l)) for b in range(B)]) for l in range(L)])
    H = np.stack([np.stack([to_np(cache.H(b, t, l)) for b in range(B)]) for l in range(L)])
    return dict(K=K, V=V, H=H)


BF16_U = 2.0 ** -8  # unit roundoff of bf16 storage (8 significant bits, round to nearest)


def _block_errors(gH, X, X_in, gK, K, gV, V, storage_u):
    """Errors of one block: normwise H, K, V, and the per-block change
    dH = H_l - H_(l-1) with its measurement floor.  Both ends of the GPU's
    change are storage-rounded block outputs (the GPU's own block input was
    unrounded), so |dH_gpu - dH_true| carries up to u (|H_l| + |H_(l-1)|) of
    rounding that no kernel can remove; dH_floor is that bound relative to
    max |dH|."""
    d_ref = X - X_in
    return dict(H=relerr(gH, X), dH=relerr(gH - X_in, d_ref), K=relerr(gK, K), V=relerr(gV, V),
                dH_floor=storage_u * (np.abs(gH).max() + np.abs(X_in).max()) / max(np.abs(d_ref).max(), 1e-30))


def gate_failures(per_block, tl):
    """Blocks failing the per-block gate: H, K and V within `tl`, the
    per-block change within `tl` plus its storage-rounding floor."""
    bad = []
    for l, e in enumerate(per_block):
        if not (e["H"] < tl and e["K"] < tl and e["V"] < tl and e["dH"] < tl + e["dH_floor"]):
            bad.append((l, e))
    return bad


def summarize(per_block):
    """Worst value of each error over the blocks."""
    return {k: max(e[k] for e in per_block) for k in ("H", "dH", "K", "V", "dH_floor")}


def teacher_forced_reuse(shape, W, latent_b, t, tkv_o, idx, cache_b, got_b):
    """Per-block parity of a region-reuse step with re-synchronised inputs.

    Block l of the oracle takes as input the GPU's own output rows of block
    l-1 (its H slot at the active tokens; block 0 takes the oracle's
    embedding), so an error in one block does not compound through the
    later ones.  cache_b: the slot the step started from (K, V [L,H,N,D], H
    [L,N,C]); got_b: the slot the GPU left (same layout).  Returns, per
    block, the normwise errors of the active rows' block output H, their
    per-block change H_l - H_(l-1) (which a broken attention or gate moves
    by O(1) under the stress weights, even where H itself is dominated by the
    residual stream) with its storage floor, and their keys and values."""
    idx = np.asarray(idx, dtype=np.int64)
    u = BF16_U if shape.dtype == "bf16" else 2.0 ** -24
    t0 = O.adaln_single(W, O.timestep_embedding(W, t))
    X_in = O.patch_embed(W, latent_b, shape.grid_h, shape.grid_w, shape.patch)[idx]
    out = []
    for l, lw in enumerate(W["layers"]):
        mod = O.layer_modulation(lw, t0)
        X, K, V, _, _ = O.block_reuse(lw, X_in, idx, mod, tkv_o[l][0], tkv_o[l][1], cache_b["K"][l], cache_b["V"][l],
                                      cache_b["H"][l], shape.heads)
        gH = np.asarray(got_b["H"][l][idx], np.float64)
        out.append(_block_errors(gH, X, X_in, got_b["K"][l][:, idx], K[:, idx], got_b["V"][l][:, idx], V[:, idx],
                                 u if l > 0 else u / 2))
        X_in = gH
    return out


def teacher_forced_dense(shape, W, latent_b, t, tkv_o, got_b):
    """teacher_forced_reuse for a dense step: every token, blocks fed the
    GPU's previous block output (all N rows)."""
    u = BF16_U if shape.dtype == "bf16" else 2.0 ** -24
    t0 = O.adaln_single(W, O.timestep_embedding(W, t))
    X_in = O.patch_embed(W, latent_b, shape.grid_h, shape.grid_w, shape.patch)
    out = []
    for l, lw in enumerate(W["layers"]):
        mod = O.layer_modulation(lw, t0)
        X, K, V, _ = O.block_dense(lw, X_in, mod, tkv_o[l][0], tkv_o[l][1], shape.heads)
        gH = np.asarray(got_b["H"][l], np.float64)
        out.append(_block_errors(gH, X, X_in, got_b["K"][l], K, got_b["V"][l], V, u if l > 0 else u / 2))
        X_in = gH
    return out
