"""Device-memory plumbing around the C ABI, using PyTorch for allocation and
streams only.  Every computation is a call into libregioncache.so.

    model = RegionCacheModel(shape, weights)        # uploads the weights
    cache = model.alloc_cache(batch, steps)          # the cache pool
    tkv = model.prepare_text(txt)                    # per-turn text keys/values
    model.build_cache(cache, step, latent, t, t_next, tkv, latent_out=out)
    act = model.localize(maps, n_delta)              # or ActiveSet.from_mask(...)
    model.reuse_step(cache, step, act, latent, t, t_next, tkv, latent_out=out)
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import abi

GLOBAL_MATS = ("pe_w", "temb_w1", "temb_w2", "tblock_w", "cap_w1", "cap_w2", "fin_w")
LAYER_MATS = ("qkv_w", "proj_w", "xq_w", "xkv_w", "xproj_w", "fc1_w", "fc2_w")


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


class ActiveSet:
    """Active token set: device idx/offsets plus the host copy of the offsets."""

    def __init__(self, idx: torch.Tensor, offsets: torch.Tensor, offsets_host: Sequence[int]):
        self.idx = idx
        self.offsets = offsets
        self.batch = len(offsets_host) - 1
        self.host = (C.c_int32 * len(offsets_host))(*[int(v) for v in offsets_host])
        self.total = int(offsets_host[-1])
        self.counts = [int(offsets_host[b + 1] - offsets_host[b]) for b in range(self.batch)]

    @classmethod
    def from_lists(cls, per_chain: Sequence[np.ndarray], device="cuda"):
        offs = [0]
        for a in per_chain:
            offs.append(offs[-1] + len(a))
        flat = np.concatenate([np.asarray(a, np.int32) for a in per_chain]) if offs[-1] else np.zeros(1, np.int32)
        idx = torch.from_numpy(flat).to(device)
        return cls(idx, torch.tensor(offs, dtype=torch.int32, device=device), offs)

    def struct(self):
        return abi.rc_active_set(self.idx.data_ptr(), self.offsets.data_ptr(),
                                 C.cast(self.host, C.POINTER(C.c_int32)), self.batch)


class CacheBuffer:
    """The cache pool: device memory, or with host=True pinned host memory
    (the host-resident pool of the pipelined step; accessors then return
    host tensors)."""

    def __init__(self, model: "RegionCacheModel", batch: int, steps: int, host: bool = False):
        nbytes = abi.rc_cache_bytes(model.ctx, batch, steps)
        self.model = model
        self.host = host
        if host:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
        else:
            self.buf = torch.empty(nbytes, dtype=torch.uint8, device=model.device)
        self.view = abi.rc_cache_view(self.buf.data_ptr(), nbytes, batch, steps)
        self.batch, self.steps = batch, steps

    def _typed(self, off, n, dtype):
        esz = torch.empty(0, dtype=dtype).element_size()
        return self.buf[off:off + n * esz].view(dtype)

    def offsets(self, b, t, l):
        k, v, h = C.c_size_t(), C.c_size_t(), C.c_size_t()
        abi.rc_cache_offsets(self.model.ctx, C.byref(self.view), b, t, l, C.byref(k), C.byref(v), C.byref(h))
        return k.value, v.value, h.value

    def K(self, b, t, l):
        """Keys of slot (b, t, l) as [heads, N, 72]."""
        m = self.model
        return self._typed(self.offsets(b, t, l)[0], m.H * m.N * 72, m.dtype).view(m.H, m.N, 72)

    def V(self, b, t, l):
        """Values of slot (b, t, l) as [heads, N, 72] (token-major, like the keys)."""
        m = self.model
        return self._typed(self.offsets(b, t, l)[1], m.H * m.N * 72, m.dtype).view(m.H, m.N, 72)

    def H(self, b, t, l):
        """Block-output hidden state of slot (b, t, l): [N, C]."""
        m = self.model
        return self._typed(self.offsets(b, t, l)[2], m.N * m.C, m.dtype).view(m.N, m.C)

    def latent(self, b, t):
        m = self.model
        off = C.c_size_t()
        abi.rc_cache_latent_offset(m.ctx, C.byref(self.view), b, t, C.byref(off))
        Hl, Wl = m.shape.grid_h * 2, m.shape.grid_w * 2
        return self._typed(off.value, 4 * Hl * Wl, torch.float32).view(4, Hl, Wl)


class RegionCacheModel:
    """Uploads a weight dict (numpy float32 arrays as drawn by the input
    generators) to device memory and owns the library context."""

    def __init__(self, shape, weights: Dict, device: str = "cuda"):
        self.shape = shape
        self.device = device
        self.dtype = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        self.N = shape.grid_h * shape.grid_w
        self.C, self.H, self.F, self.L = shape.hidden, shape.heads, shape.mlp, shape.layers
        self._keep = []

        def mat(a):
            t = torch.as_tensor(np.ascontiguousarray(a)).to(device=device, dtype=self.dtype)
            self._keep.append(t)
            return t.data_ptr()

        def vec(a):
            t = torch.as_tensor(np.ascontiguousarray(a, dtype=np.float32)).to(device)
            self._keep.append(t)
            return t.data_ptr()

        layers = (abi.rc_layer_weights * shape.layers)()
        for i, lw in enumerate(weights["layers"]):
            for f in abi.LAYER_FIELDS:
                setattr(layers[i], f, mat(lw[f]) if f in LAYER_MATS else vec(lw[f]))
        self._layers = layers
        w = abi.rc_weights()
        w.layers = C.cast(layers, C.POINTER(abi.rc_layer_weights))
        for f in abi.GLOBAL_FIELDS:
            if shape.token_mode and f not in ("tblock_w", "tblock_b"):
                continue
            if f in weights:
                setattr(w, f, mat(weights[f]) if f in GLOBAL_MATS else vec(weights[f]))
        self._w = w
        cfg = abi.rc_model_config(shape.hidden, shape.heads, shape.head_dim, shape.mlp, shape.layers,
                                  shape.text_len, shape.text_dim, shape.grid_h, shape.grid_w, shape.latent_ch,
                                  shape.patch, shape.out_ch, abi.RC_BF16 if shape.dtype == "bf16" else abi.RC_F32,
                                  1 if shape.token_mode else 0, 1e-6)
        self._cfg = cfg
        ctx = C.c_void_p()
        abi.rc_create(C.byref(cfg), C.byref(w), C.byref(ctx))
        self.ctx = ctx
        self._ws = None

    def __del__(self):
        try:
            if getattr(self, "ctx", None):
                abi.rc_destroy(self.ctx)
                self.ctx = None
        except Exception:
            pass

    # ------------------------------------------------------------ buffers
    def alloc_cache(self, batch: int, steps: int, host: bool = False) -> CacheBuffer:
        return CacheBuffer(self, batch, steps, host)

    def staging(self, batch: int) -> torch.Tensor:
        """Device staging ring of the host-resident pool."""
        nbytes = abi.rc_staging_bytes(self.ctx, batch)
        if getattr(self, "_stage", None) is None or self._stage.numel() < nbytes:
            self._stage = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self._stage

    def workspace(self, max_rows: int, batch: int) -> torch.Tensor:
        nbytes = abi.rc_workspace_bytes(self.ctx, max_rows, batch)
        if self._ws is None or self._ws.numel() < nbytes:
            self._ws = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self._ws

    def to_storage(self, a) -> torch.Tensor:
        return torch.as_tensor(np.ascontiguousarray(a)).to(device=self.device, dtype=self.dtype)

    # ------------------------------------------------------------ calls
    def prepare_text(self, txt: torch.Tensor) -> torch.Tensor:
        B = txt.shape[0]
        tkv = torch.empty(abi.rc_text_kv_bytes(self.ctx, B), dtype=torch.uint8, device=self.device)
        ws = self.workspace(1, B)
        abi.rc_prepare_text(self.ctx, _ptr(txt), B, _ptr(tkv), _ptr(ws), ws.numel(), _stream())
        return tkv

    def _io(self, inp, timestep, timestep_next, tkv, delta, maps, latent_out, t_vec, text_valid=None,
            guidance=None):
        d = None
        n_delta = 0
        if delta is not None and len(delta):
            d = (C.c_int32 * len(delta))(*[int(x) for x in delta])
            n_delta = len(delta)
        io = abi.rc_step_io(inp.data_ptr(), None if t_vec is None else t_vec.data_ptr(), int(timestep),
                            int(timestep_next), tkv.data_ptr(),
                            None if d is None else C.cast(d, C.POINTER(C.c_int32)), n_delta,
                            None if maps is None else maps.data_ptr(),
                            None if latent_out is None else latent_out.data_ptr(),
                            None if text_valid is None else text_valid.data_ptr(),
                            0 if guidance is None else 1, 0.0 if guidance is None else float(guidance))
        return io, d

    def build_cache(self, cache: CacheBuffer, step: int, inp: torch.Tensor, timestep: int, timestep_next: int,
                    tkv: torch.Tensor, delta=None, maps=None, latent_out=None, t_vec=None, text_valid=None,
                    guidance=None):
        """text_valid: optional device int32 [batch] of unpadded prompt lengths.
        guidance: classifier-free guidance scale; chains 2p and 2p+1 are then
        the conditional and unconditional branch of one image."""
        io, keep = self._io(inp, timestep, timestep_next, tkv, delta, maps, latent_out, t_vec, text_valid,
                            guidance)
        ws = self.workspace(cache.batch * self.N, cache.batch)
        if cache.host:
            st = self.staging(cache.batch)
            abi.rc_build_cache_hosted(self.ctx, C.byref(cache.view), step, C.byref(io), _ptr(st), st.numel(),
                                      _ptr(ws), ws.numel(), _stream())
        else:
            abi.rc_build_cache(self.ctx, C.byref(cache.view), step, C.byref(io), _ptr(ws), ws.numel(), _stream())

    def reuse_step(self, cache: CacheBuffer, step: int, act: ActiveSet, inp: torch.Tensor, timestep: int,
                   timestep_next: int, tkv: torch.Tensor, delta=None, maps=None, latent_out=None, t_vec=None,
                   fuse: bool = True, active_hidden: Optional[torch.Tensor] = None, text_valid=None,
                   guidance=None, validate: bool = False):
        """validate: check the active set on the device first (RC_VALIDATE);
        an invalid set raises RcError (RC_ERR_INDEX) before any launch."""
        io, keep = self._io(inp, timestep, timestep_next, tkv, delta, maps, latent_out, t_vec, text_valid,
                            guidance)
        ws = self.workspace(max(act.total, 1), cache.batch)
        s = act.struct()
        if cache.host:
            if not fuse or active_hidden is not None:
                raise ValueError("a host-resident pool is updated in place (fuse=True, no active_hidden)")
            st = self.staging(cache.batch)
            abi.rc_reuse_step_hosted(self.ctx, C.byref(cache.view), step, C.byref(s), C.byref(io), _ptr(st),
                                     st.numel(), _ptr(ws), ws.numel(), _stream())
        else:
            flags = (abi.RC_FUSE_UPDATE if fuse else 0) | (abi.RC_VALIDATE if validate else 0)
            abi.rc_reuse_step(self.ctx, C.byref(cache.view), step, C.byref(s), C.byref(io), _ptr(active_hidden),
                              flags, _ptr(ws), ws.numel(), _stream())

    def validate_active(self, act: ActiveSet):
        """Device check of an active set (rc_validate_active); raises RcError
        with RC_ERR_INDEX if a chain's tokens are not strictly ascending in
        [0, N) or the device offsets differ from the host copy."""
        scratch = self.workspace(1, act.batch)
        s = act.struct()
        abi.rc_validate_active(self.ctx, C.byref(s), act.batch, _ptr(scratch), scratch.numel(), _stream())

    def update_cache(self, cache: CacheBuffer, step: int, act: ActiveSet, active_hidden: torch.Tensor):
        s = act.struct()
        abi.rc_update_cache(self.ctx, C.byref(cache.view), step, C.byref(s), _ptr(active_hidden), _stream())

    def localize(self, maps: torch.Tensor, n_delta: int, threshold: float = 0.3, radius: int = 1):
        B = maps.shape[0]
        mask = torch.empty((B, self.N), dtype=torch.uint8, device=self.device)
        idx = torch.empty(B * self.N, dtype=torch.int32, device=self.device)
        offs = torch.empty(B + 1, dtype=torch.int32, device=self.device)
        host = (C.c_int32 * (B + 1))()
        abi.rc_localize_region(self.ctx, _ptr(maps), B, n_delta, threshold, radius, _ptr(mask), _ptr(idx),
                               _ptr(offs), C.cast(host, C.POINTER(C.c_int32)), _stream())
        return mask, ActiveSet(idx, offs, list(host))

    def set_kernel_timing(self, enable: bool):
        abi.rc_set_kernel_timing(self.ctx, 1 if enable else 0)

    def kernel_timing(self, cls: int):
        ms, n = C.c_double(), C.c_int64()
        abi.rc_get_kernel_timing(self.ctx, cls, C.byref(ms), C.byref(n))
        return ms.value, n.value


def compact_mask(mask: torch.Tensor) -> ActiveSet:
    B, N = mask.shape
    idx = torch.empty(B * N, dtype=torch.int32, device=mask.device)
    offs = torch.empty(B + 1, dtype=torch.int32, device=mask.device)
    host = (C.c_int32 * (B + 1))()
    abi.rc_compact_mask(_ptr(mask), B, N, _ptr(idx), _ptr(offs), C.cast(host, C.POINTER(C.c_int32)), _stream())
    return ActiveSet(idx, offs, list(host))


def maps_from_logits(logits_bf16: torch.Tensor, delta: Sequence[int]) -> torch.Tensor:
    """Sum over (layer, head) of the softmax probability of each delta column;
    logits [L, H, N, M] bf16 on the device -> maps [N, n_delta] float32."""
    L, Hh, N, M = logits_bf16.shape
    nd = len(delta)
    out = torch.empty((N, nd), dtype=torch.float32, device=logits_bf16.device)
    nbytes = abi.rc_maps_from_logits_scratch_bytes(L, N, nd)
    scratch = torch.empty(nbytes, dtype=torch.uint8, device=logits_bf16.device)
    d = (C.c_int32 * nd)(*[int(x) for x in delta])
    abi.rc_maps_from_logits(_ptr(logits_bf16), L, Hh, N, M, C.cast(d, C.POINTER(C.c_int32)), nd, _ptr(out),
                            _ptr(scratch), nbytes, _stream())
    return out
