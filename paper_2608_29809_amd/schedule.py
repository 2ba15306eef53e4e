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

__all__ = ["timestep_grid", "prompt_similarity", "reuse_cutoff", "step_plan", "EditSession"]


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


class EditSession:
    """A batch of edit chains sharing one cache pool of T steps.

    ``first_turn`` generates from noise with T dense steps, which fills the
    pool; every ``edit_turn`` then runs the plan of its reading, keeping the
    pool equal to the latest turn's trajectory."""

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
        return x

    def edit_turn(self, txt: torch.Tensor, x_T: torch.Tensor, delta_cols: Sequence[int],
                  similarity: Optional[float] = None, region: Optional[ActiveSet] = None) -> dict:
        """One editing turn with the new prompt features txt and the same
        initial noise x_T.  delta_cols are the text positions of the new or
        changed tokens; similarity is Eq. 1's s for the "paper" reading;
        region overrides the localised active set (required by the "paper"
        reading).  Returns the final latent, the plan, the active set and (for
        "dense_then_reuse") the localisation mask."""
        if self.turns == 0:
            raise RuntimeError("edit_turn needs a first turn to fill the cache pool")
        m = self.model
        plan = step_plan(self.T, self.rho, self.reading, similarity, self.tau_s)
        n_dense = plan.count("dense")
        if region is None and n_dense == 0 and "reuse" in plan:
            raise ValueError("this plan has no dense step to localise the region from: pass region")
        tkv = m.prepare_text(txt)
        x = x_T.contiguous()
        act, mask = region, None
        empty = ActiveSet.from_lists([np.zeros(0, np.int32)] * self.batch)
        for s, what in enumerate(plan):
            nxt = torch.empty_like(x)
            t, tn = int(self.tgrid[s]), self._t_next(s)
            if what == "dense":
                emit = region is None and s == n_dense - 1
                maps = torch.zeros((self.batch, m.N, len(delta_cols)), device=x.device) if emit else None
                m.build_cache(self.cache, s, x, t, tn, tkv, list(delta_cols) if emit else None, maps, nxt,
                              guidance=self.guidance)
                if emit:
                    mask, act = m.localize(maps, len(delta_cols), self.threshold, self.radius)
                    if self.guidance is not None:  # the conditional branch's region for both branches
                        mask = mask[0::2].repeat_interleave(2, dim=0).contiguous()
                        act = compact_mask(mask)
            elif what == "copy":
                m.reuse_step(self.cache, s, empty, x, t, tn, tkv, latent_out=nxt, guidance=self.guidance)
            else:
                m.reuse_step(self.cache, s, act, x, t, tn, tkv, latent_out=nxt, guidance=self.guidance)
            x = nxt
        self.turns += 1
        return dict(latent=x, plan=plan, active=act, mask=mask)
