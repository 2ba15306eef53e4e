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
