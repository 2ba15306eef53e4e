"""Host control of multi-turn editing (Sec. 3.2 and Sec. 3.3): the sampler's
timestep grid, the prompt similarity of Eq. 1, the reuse cutoff of Eq. 2,
the per-step plan of a turn, and a driver that runs turns on the library's
four verbs (build cache, localise region, reuse step, update cache).

Plans (per step of a turn, for the edited region):

* ``"dense_then_reuse"``: the first floor(rho T) steps run dense (they rewrite
  the cache for those steps and the last of them emits the cross-attention
  maps of the delta tokens), the region is localised from the maps, and the
  remaining steps are region-reuse steps.
* ``"paper"``: Eq. 2 -- the region keeps the cached states ("copy": a reuse
  step with no active token, so every output is the cache) for the first
  T_reuse steps and is recomputed with region reuse after that.  No step of
  this plan runs dense, so the caller supplies the region.

Everything here is host arithmetic and orchestration; every computation on
tensors is a library call.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence

import numpy as np
import torch

from .runtime import ActiveSet, CacheBuffer, RegionCacheModel, compact_mask

__all__ = ["timestep_grid", "prompt_similarity", "delta_similarity", "reuse_cutoff", "step_plan", "EditSession"]


def timestep_grid(T: int) -> np.ndarray:
    """DDPM timesteps of a T-step sampler: 999 down to 0, evenly spaced, rounded."""
    return np.round(np.linspace(999, 0, T)).astype(np.int64)


def prompt_similarity(e_before, e_after) -> float:
    """Eq. 1: cosine similarity of the embeddings of the edited tokens before
    and after the edit."""
    a = np.asarray(e_before, np.float64).ravel()
    b = np.asarray(e_after, np.float64).ravel()
    return float(a @ b / (np.sqrt(a @ a) * np.sqrt(b @ b)))


def reuse_cutoff(T: int, s: float, tau_s: float, rho: float = 0.2) -> int:
    """Eq. 2: steps for which the cached states of the region are reused --
    all T when the edit is semantically consistent (s >= tau_s), otherwise the
    first floor(rho T)."""
    return T if s >= tau_s else int(math.floor(rho * T))


def step_plan(T: int, rho: float = 0.2, reading: str = "dense_then_reuse", s: Optional[float] = None,
              tau_s: float = 0.8) -> List[str]:
    """Per-step actions of one editing turn ("dense", "reuse" or "copy")."""
    if reading == "dense_then_reuse":
        k = int(math.floor(rho * T))
        return ["dense"] * k + ["reuse"] * (T - k)
    if reading == "paper":
        tr = reuse_cutoff(T, 0.0 if s is None else s, tau_s, rho)
        return ["copy"] * tr + ["reuse"] * (T - tr)
    raise ValueError(f"unknown reading {reading!r}")


def delta_similarity(txt_before: torch.Tensor, txt_after: torch.Tensor, delta_cols: Sequence[int]) -> List[float]:
    """Eq. 1 per chain: cosine similarity of the edited tokens' embeddings
    before and after the edit.  The embedding of the edited tokens is taken
    to be the prompt features at the delta columns (the text features the
    caption projection consumes), flattened over those columns.  Only these
    few rows are copied to the host."""
    cols = torch.as_tensor([int(c) for c in delta_cols], dtype=torch.long, device=txt_before.device)
    a = txt_before.index_select(1, cols).float().cpu().numpy()
    b = txt_after.index_select(1, cols).float().cpu().numpy()
    return [prompt_similarity(a[i], b[i]) for i in range(a.shape[0])]


class EditSession:
    """A batch of edit chains sharing one cache pool of T steps.

    ``first_turn`` generates from noise with T dense steps, which fills the
    pool; every ``edit_turn`` then runs the plan of its reading, keeping the
    pool equal to the latest turn's trajectory.  Under the "paper" reading
    each chain has its own reuse cutoff (Eq. 2 on its own Eq. 1 similarity):
    at step s a chain is active ("reuse") once s >= its cutoff and keeps the
    cache ("copy", no active token) before, all chains in one step call."""

    def __init__(self, model: RegionCacheModel, batch: int, T: int = 20, rho: float = 0.2, tau_s: float = 0.8,
                 reading: str = "dense_then_reuse", threshold: float = 0.3, radius: int = 1,
                 guidance: Optional[float] = None):
        """guidance: classifier-free guidance scale; the batch then holds
        (conditional, unconditional) chain pairs and the localised region of
        each conditional chain is used for its pair."""
        if reading not in ("dense_then_reuse", "paper"):
            raise ValueError(f"unknown reading {reading!r}")
        if guidance is not None and batch % 2:
            raise ValueError("guidance needs (conditional, unconditional) chain pairs")
        self.guidance = guidance
        self.model, self.batch, self.T = model, batch, T
        self.rho, self.tau_s, self.reading = rho, tau_s, reading
        self.threshold, self.radius = threshold, radius
        self.cache: CacheBuffer = model.alloc_cache(batch, T)
        self.tgrid = timestep_grid(T)
        self.turns = 0
        self.prev_txt: Optional[torch.Tensor] = None

    def _t_next(self, s: int) -> int:
        return int(self.tgrid[s + 1]) if s + 1 < self.T else -1

    def first_turn(self, txt: torch.Tensor, x_T: torch.Tensor) -> torch.Tensor:
        """T dense steps from the noise x_T [B, c, 2gh, 2gw] with the prompt
        features txt; returns the final latent."""
        m = self.model
        tkv = m.prepare_text(txt)
        x = x_T.contiguous()
        for s in range(self.T):
            nxt = torch.empty_like(x)
            m.build_cache(self.cache, s, x, int(self.tgrid[s]), self._t_next(s), tkv, latent_out=nxt,
                          guidance=self.guidance)
            x = nxt
        self.turns = 1
        self.prev_txt = txt
        return x

    def _chain_lists(self, act: ActiveSet) -> List[np.ndarray]:
        idx = act.idx[:max(act.total, 1)].cpu().numpy()[:act.total]
        off = [int(v) for v in act.host]
        return [idx[off[b]:off[b + 1]] for b in range(act.batch)]

    def edit_turn(self, txt: torch.Tensor, x_T: torch.Tensor, delta_cols: Sequence[int],
                  similarity=None, region: Optional[ActiveSet] = None) -> dict:
        """One editing turn with the new prompt features txt and the same
        initial noise x_T.  delta_cols are the text positions of the new or
        changed tokens.  similarity is Eq. 1's s for the "paper" reading: a
        number for every chain, one per chain, or None to compute it per
        chain from the previous turn's and this turn's features at the delta
        columns (delta_similarity).  region overrides the localised active
        set (required by the "paper" reading, which runs no dense step).
        Returns the final latent, chain 0's plan ("plan"), every chain's plan
        ("plans"), the similarities, the active set and (for
        "dense_then_reuse") the localisation mask."""
        if self.turns == 0:
            raise RuntimeError("edit_turn needs a first turn to fill the cache pool")
        m = self.model
        B = self.batch
        sims: Optional[List[float]] = None
        if self.reading == "paper":
            if similarity is None:
                sims = delta_similarity(self.prev_txt, txt, delta_cols)
            elif np.ndim(similarity) == 0:
                sims = [float(similarity)] * B
            else:
                sims = [float(v) for v in similarity]
            if self.guidance is not None:  # both branches of an image follow the conditional one
                sims = [sims[b - b % 2] for b in range(B)]
            plans = [step_plan(self.T, self.rho, "paper", sims[b], self.tau_s) for b in range(B)]
        else:
            plans = [step_plan(self.T, self.rho, self.reading)] * B
        n_dense = plans[0].count("dense")
        if region is None and n_dense == 0 and any("reuse" in p for p in plans):
            raise ValueError("this plan has no dense step to localise the region from: pass region")
        tkv = m.prepare_text(txt)
        x = x_T.contiguous()
        act, mask = region, None
        lists = self._chain_lists(region) if region is not None else None
        empty = np.zeros(0, np.int32)
        step_sets = {}
        for s in range(self.T):
            what = [p[s] for p in plans]
            nxt = torch.empty_like(x)
            t, tn = int(self.tgrid[s]), self._t_next(s)
            if what[0] == "dense":
                emit = region is None and s == n_dense - 1
                maps = torch.zeros((B, m.N, len(delta_cols)), device=x.device) if emit else None
                m.build_cache(self.cache, s, x, t, tn, tkv, list(delta_cols) if emit else None, maps, nxt,
                              guidance=self.guidance)
                if emit:
                    mask, act = m.localize(maps, len(delta_cols), self.threshold, self.radius)
                    if self.guidance is not None:  # the conditional branch's region for both branches
                        mask = mask[0::2].repeat_interleave(2, dim=0).contiguous()
                        act = compact_mask(mask)
                    lists = self._chain_lists(act)
            else:
                key = tuple(w == "reuse" for w in what)
                if key not in step_sets:
                    step_sets[key] = ActiveSet.from_lists([lists[b] if key[b] else empty for b in range(B)]) \
                        if any(key) else ActiveSet.from_lists([empty] * B)
                m.reuse_step(self.cache, s, step_sets[key], x, t, tn, tkv, latent_out=nxt, guidance=self.guidance)
            x = nxt
        self.turns += 1
        self.prev_txt = txt
        return dict(latent=x, plan=plans[0], plans=plans, similarity=sims, active=act, mask=mask)
