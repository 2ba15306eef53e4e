"""ctypes binding of libregioncache.so (include/regioncache.h).

Argument marshalling only: every function here forwards to the C function of
the same name and raises RcError on a negative status.  Nothing is computed
in Python.  The library must have been built (paper_2608_29809_amd/build.py);
importing this module without it raises immediately.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libregioncache.so")

RC_OK = 0
STATUS = {0: "RC_OK", -1: "RC_ERR_INVALID_ARG", -2: "RC_ERR_SHAPE", -3: "RC_ERR_ALIGN",
          -4: "RC_ERR_INDEX", -5: "RC_ERR_CAPACITY", -6: "RC_ERR_NO_DEVICE", -7: "RC_ERR_HIP",
          -8: "RC_ERR_UNSUPPORTED"}
RC_F32, RC_BF16 = 0, 1
RC_FUSE_UPDATE = 1
RC_VALIDATE = 2
RC_STATIC_SCRATCH_BYTES = 16 << 20
(RC_KC_GEMM, RC_KC_ATTN_SELF, RC_KC_ATTN_CROSS, RC_KC_ATTN_COMBINE, RC_KC_NORM, RC_KC_EMBED,
 RC_KC_FINAL, RC_KC_COND, RC_KC_MISC, RC_KC_GEMM_QKV, RC_KC_GEMM_FC1, RC_KC_GEMM_FC2, RC_KC_GEMM_PROJ,
 RC_KC_GEMM_XQ, RC_KC_GEMM_XPROJ, RC_KC_SPLIT_FINISH) = range(16)
RC_KC_COUNT = 16
KERNEL_CLASSES = ["gemm", "attn_self", "attn_cross", "attn_combine", "norm", "embed", "final",
                  "cond", "misc", "gemm_qkv", "gemm_fc1", "gemm_fc2", "gemm_proj",
                  "gemm_xq", "gemm_xproj", "split_finish"]


class RcError(RuntimeError):
    def __init__(self, status, func, msg):
        super().__init__(f"{func} -> {STATUS.get(status, status)}: {msg}")
        self.status = status


class rc_model_config(C.Structure):
    _fields_ = [("hidden", C.c_int32), ("heads", C.c_int32), ("head_dim", C.c_int32), ("mlp", C.c_int32),
                ("layers", C.c_int32), ("text_len", C.c_int32), ("text_dim", C.c_int32),
                ("grid_h", C.c_int32), ("grid_w", C.c_int32), ("latent_ch", C.c_int32), ("patch", C.c_int32),
                ("out_ch", C.c_int32), ("dtype", C.c_int32), ("token_mode", C.c_int32), ("ln_eps", C.c_float)]


LAYER_FIELDS = ["qkv_w", "proj_w", "xq_w", "xkv_w", "xproj_w", "fc1_w", "fc2_w",
                "qkv_b", "proj_b", "xq_b", "xkv_b", "xproj_b", "fc1_b", "fc2_b", "sst"]


class rc_layer_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in LAYER_FIELDS]


GLOBAL_FIELDS = ["pe_w", "pe_b", "temb_w1", "temb_b1", "temb_w2", "temb_b2", "tblock_w", "tblock_b",
                 "cap_w1", "cap_b1", "cap_w2", "cap_b2", "fin_w", "fin_b", "fin_sst"]


class rc_weights(C.Structure):
    _fields_ = [("layers", C.POINTER(rc_layer_weights))] + [(n, C.c_void_p) for n in GLOBAL_FIELDS]


class rc_cache_view(C.Structure):
    _fields_ = [("base", C.c_void_p), ("bytes", C.c_size_t), ("batch", C.c_int32), ("steps", C.c_int32)]


class rc_active_set(C.Structure):
    _fields_ = [("idx", C.c_void_p), ("offsets", C.c_void_p), ("offsets_host", C.POINTER(C.c_int32)),
                ("batch", C.c_int32)]


class rc_step_io(C.Structure):
    _fields_ = [("input", C.c_void_p), ("t_vec", C.c_void_p), ("timestep", C.c_int32),
                ("timestep_next", C.c_int32), ("text_kv", C.c_void_p),
                ("delta_cols_host", C.POINTER(C.c_int32)), ("n_delta", C.c_int32), ("maps", C.c_void_p),
                ("latent_out", C.c_void_p), ("text_valid", C.c_void_p), ("guided", C.c_int32),
                ("guidance_scale", C.c_float)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2608_29809_amd/build.py "
                          "(or __graft_entry__.build())")
    lib = C.CDLL(LIB_PATH)
    P, S, I32, U32 = C.c_void_p, C.c_size_t, C.c_int32, C.c_uint32
    pI32 = C.POINTER(C.c_int32)
    sig = {
        "rc_last_error": (C.c_char_p, []),
        "rc_create": (C.c_int, [C.POINTER(rc_model_config), C.POINTER(rc_weights), C.POINTER(P)]),
        "rc_destroy": (None, [P]),
        "rc_cache_bytes": (S, [P, I32, I32]),
        "rc_text_kv_bytes": (S, [P, I32]),
        "rc_workspace_bytes": (S, [P, I32, I32]),
        "rc_cache_offsets": (C.c_int, [P, C.POINTER(rc_cache_view), I32, I32, I32, C.POINTER(S),
                                       C.POINTER(S), C.POINTER(S)]),
        "rc_cache_latent_offset": (C.c_int, [P, C.POINTER(rc_cache_view), I32, I32, C.POINTER(S)]),
        "rc_prepare_text": (C.c_int, [P, P, I32, P, P, S, P]),
        "rc_build_cache": (C.c_int, [P, C.POINTER(rc_cache_view), I32, C.POINTER(rc_step_io), P, S, P]),
        "rc_reuse_step": (C.c_int, [P, C.POINTER(rc_cache_view), I32, C.POINTER(rc_active_set),
                                    C.POINTER(rc_step_io), P, U32, P, S, P]),
        "rc_update_cache": (C.c_int, [P, C.POINTER(rc_cache_view), I32, C.POINTER(rc_active_set), P, P]),
        "rc_validate_active": (C.c_int, [P, C.POINTER(rc_active_set), I32, P, S, P]),
        "rc_staging_bytes": (S, [P, I32]),
        "rc_reuse_step_hosted": (C.c_int, [P, C.POINTER(rc_cache_view), I32, C.POINTER(rc_active_set),
                                           C.POINTER(rc_step_io), P, S, P, S, P]),
        "rc_build_cache_hosted": (C.c_int, [P, C.POINTER(rc_cache_view), I32, C.POINTER(rc_step_io), P, S, P, S,
                                            P]),
        "rc_localize_region": (C.c_int, [P, P, I32, I32, C.c_float, I32, P, P, P, pI32, P]),
        "rc_maps_from_logits_scratch_bytes": (S, [I32, I32, I32]),
        "rc_maps_from_logits": (C.c_int, [P, I32, I32, I32, I32, pI32, I32, P, P, S, P]),
        "rc_maps_from_logits_noalloc": (C.c_int, [P, I32, I32, I32, I32, pI32, I32, P, P]),
        "rc_compact_mask": (C.c_int, [P, I32, I32, P, P, pI32, P]),
        "rc_sync": (C.c_int, [P]),
        "rc_set_kernel_timing": (C.c_int, [P, I32]),
        "rc_get_kernel_timing": (C.c_int, [P, I32, C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


LIB = _load()


def rc_last_error() -> str:
    return LIB.rc_last_error().decode()


def _chk(name, st):
    if st != RC_OK:
        raise RcError(st, name, rc_last_error())
    return st


def _wrap(name):
    f = getattr(LIB, name)

    def call(*args):
        return _chk(name, f(*args))

    call.__name__ = name
    call.__doc__ = f"Forwards to the C function {name} (include/regioncache.h); raises RcError on failure."
    return call


for _n in ["rc_create", "rc_cache_offsets", "rc_cache_latent_offset", "rc_prepare_text", "rc_build_cache",
           "rc_reuse_step", "rc_update_cache", "rc_validate_active", "rc_reuse_step_hosted", "rc_build_cache_hosted",
           "rc_localize_region", "rc_maps_from_logits", "rc_maps_from_logits_noalloc", "rc_compact_mask", "rc_sync", "rc_set_kernel_timing",
           "rc_get_kernel_timing"]:
    globals()[_n] = _wrap(_n)

rc_destroy = LIB.rc_destroy
rc_cache_bytes = LIB.rc_cache_bytes
rc_text_kv_bytes = LIB.rc_text_kv_bytes
rc_workspace_bytes = LIB.rc_workspace_bytes
rc_staging_bytes = LIB.rc_staging_bytes
rc_maps_from_logits_scratch_bytes = LIB.rc_maps_from_logits_scratch_bytes
