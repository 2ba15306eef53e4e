"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, sizes its buffers as documented, and rejects invalid
arguments before any launch.  Nothing here executes GPU code: where a call
would pass validation it is only made when no GPU is present (it must then
return RC_ERR_NO_DEVICE)."""
import ctypes as C
import os
import re

import pytest
import torch

from paper_2608_29809_amd import abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "regioncache.h")
NO_GPU = torch.cuda.device_count() == 0
FAKE = 1 << 20  # an aligned non-null address; never dereferenced by these tests


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rc_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 19
    for n in names:
        assert hasattr(abi.LIB, n), n


def cfg(**over):
    d = dict(hidden=1152, heads=16, head_dim=72, mlp=4608, layers=2, text_len=120, text_dim=4096,
             grid_h=32, grid_w=32, latent_ch=4, patch=2, out_ch=8, dtype=abi.RC_BF16, token_mode=0, ln_eps=1e-6)
    d.update(over)
    return abi.rc_model_config(*[d[f] for f, _ in abi.rc_model_config._fields_])


def weights(layers=2):
    L = (abi.rc_layer_weights * layers)()
    for i in range(layers):
        for f in abi.LAYER_FIELDS:
            setattr(L[i], f, FAKE)
    w = abi.rc_weights()
    w.layers = C.cast(L, C.POINTER(abi.rc_layer_weights))
    for f in abi.GLOBAL_FIELDS:
        setattr(w, f, FAKE)
    return w, L


def create(c, w):
    ctx = C.c_void_p()
    st = abi.LIB.rc_create(C.byref(c), C.byref(w), C.byref(ctx))
    return st, ctx


def test_create_validation():
    w, keep = weights()
    assert create(cfg(head_dim=64, hidden=1024), w)[0] == -8
    assert create(cfg(hidden=1140), w)[0] == -2
    assert create(cfg(grid_h=5, grid_w=5), w)[0] == -8
    assert create(cfg(text_len=200), w)[0] == -8
    assert create(cfg(dtype=7), w)[0] == -1
    w.layers[1].fc2_w = None
    assert create(cfg(), w)[0] == -1
    assert "layer 1" in abi.rc_last_error()
    w.layers[1].fc2_w = FAKE + 8
    assert create(cfg(), w)[0] == -3
    w.layers[1].fc2_w = FAKE
    st, ctx = create(cfg(), w)
    assert st == 0 and ctx.value
    abi.rc_destroy(ctx)


@pytest.fixture
def ctx():
    w, keep = weights()
    st, c = create(cfg(), w)
    assert st == 0
    yield c
    abi.rc_destroy(c)


def test_buffer_sizes(ctx):
    N, C_, L = 1024, 1152, 2
    slot = 3 * N * C_ * 2
    slots = 3 * 5 * L * slot
    lat = 3 * 6 * 4 * 64 * 64 * 4
    assert abi.rc_cache_bytes(ctx, 3, 5) == ((slots + 255) // 256) * 256 + lat
    assert abi.rc_text_kv_bytes(ctx, 3) == L * 3 * 2 * 16 * 128 * 72 * 2
    assert abi.rc_workspace_bytes(ctx, 500, 1) > 500 * (4 * C_ + 3 * 2 * C_ + 2 * 4608)
    assert abi.rc_cache_bytes(ctx, 0, 5) == 0
    view = abi.rc_cache_view(FAKE, abi.rc_cache_bytes(ctx, 3, 5), 3, 5)
    k, v, h = C.c_size_t(), C.c_size_t(), C.c_size_t()
    abi.rc_cache_offsets(ctx, C.byref(view), 2, 4, 1, C.byref(k), C.byref(v), C.byref(h))
    base = ((2 * 5 + 4) * L + 1) * slot
    assert (k.value, v.value, h.value) == (base, base + 16 * N * 72 * 2, base + 2 * 16 * N * 72 * 2)
    off = C.c_size_t()
    abi.rc_cache_latent_offset(ctx, C.byref(view), 1, 5, C.byref(off))
    assert off.value == ((slots + 255) // 256) * 256 + (1 * 6 + 5) * 4 * 64 * 64 * 4
    with pytest.raises(abi.RcError):
        abi.rc_cache_offsets(ctx, C.byref(view), 3, 0, 0, C.byref(k), C.byref(v), C.byref(h))


def _io(**over):
    d = dict(input=FAKE, t_vec=None, timestep=500, timestep_next=450, text_kv=FAKE, delta_cols_host=None,
             n_delta=0, maps=None, latent_out=FAKE, text_valid=None, guided=0, guidance_scale=0.0)
    d.update(over)
    return abi.rc_step_io(*[d[f] for f, _ in abi.rc_step_io._fields_])


def test_step_validation(ctx):
    nb = abi.rc_cache_bytes(ctx, 1, 4)
    view = abi.rc_cache_view(FAKE, nb, 1, 4)
    ws = abi.rc_workspace_bytes(ctx, 1024, 1)
    build = abi.LIB.rc_build_cache
    assert build(ctx, C.byref(view), 4, C.byref(_io()), FAKE, ws, None) == -2           # step out of range
    small = abi.rc_cache_view(FAKE, nb - 1, 1, 4)
    assert build(ctx, C.byref(small), 0, C.byref(_io()), FAKE, ws, None) == -5         # cache too small
    mis = abi.rc_cache_view(FAKE + 4, nb, 1, 4)
    assert build(ctx, C.byref(mis), 0, C.byref(_io()), FAKE, ws, None) == -3           # misaligned
    assert build(ctx, C.byref(view), 0, C.byref(_io(timestep=1000)), FAKE, ws, None) == -1
    bad = (C.c_int32 * 2)(5, 120)
    io = _io(delta_cols_host=C.cast(bad, C.POINTER(C.c_int32)), n_delta=2, maps=FAKE)
    assert build(ctx, C.byref(view), 0, C.byref(io), FAKE, ws, None) == -4           # delta column range
    assert build(ctx, C.byref(view), 0, C.byref(_io(n_delta=9)), FAKE, ws, None) == -1
    assert build(ctx, C.byref(view), 0, C.byref(_io(latent_out=None)), FAKE, ws, None) == -1
    if NO_GPU:
        assert build(ctx, C.byref(view), 0, C.byref(_io()), FAKE, ws, None) == -6    # valid, no device


def test_reuse_validation(ctx):
    nb = abi.rc_cache_bytes(ctx, 2, 4)
    view = abi.rc_cache_view(FAKE, nb, 2, 4)
    ws = abi.rc_workspace_bytes(ctx, 1024, 2)
    step = abi.LIB.rc_reuse_step

    def aset(offs, batch=2):
        h = (C.c_int32 * len(offs))(*offs)
        return abi.rc_active_set(FAKE, FAKE, C.cast(h, C.POINTER(C.c_int32)), batch), h

    a, k1 = aset([0, 10, 5])                                                             # not monotone
    assert step(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), None, 1, FAKE, ws, None) == -4
    a, k2 = aset([1, 10, 20])                                                            # offsets[0] != 0
    assert step(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), None, 1, FAKE, ws, None) == -4
    a, k3 = aset([0, 2000, 2010])                                                        # R_b > N
    assert step(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), None, 1, FAKE, ws, None) == -4
    a, k4 = aset([0, 10, 20], batch=3)                                                   # batch mismatch
    assert step(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), None, 1, FAKE, ws, None) == -2
    a, k5 = aset([0, 10, 20])
    assert step(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), None, 4, FAKE, ws, None) == -1  # flags
    # RC_VALIDATE is a known flag; it needs the workspace for its verdict
    fv = abi.RC_FUSE_UPDATE | abi.RC_VALIDATE
    assert step(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), None, fv, None, ws, None) == -1
    assert step(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), None, fv, FAKE, 8, None) == -1
    if NO_GPU:
        assert step(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), None, 1, FAKE, ws, None) == -6
        assert step(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), None, fv, FAKE, ws, None) == -6


def test_validate_active_plumbing(ctx):
    """rc_validate_active: host-side counts checked first (as for a step),
    then the scratch, then the device."""
    val = abi.LIB.rc_validate_active

    def aset(offs, batch=2):
        h = (C.c_int32 * len(offs))(*offs)
        return abi.rc_active_set(FAKE, FAKE, C.cast(h, C.POINTER(C.c_int32)), batch), h

    a, k = aset([0, 10, 20])
    assert val(None, C.byref(a), 2, FAKE, 16, None) == -1
    assert val(ctx, None, 2, FAKE, 16, None) == -1
    assert val(ctx, C.byref(a), 3, FAKE, 16, None) == -2        # batch differs from the set's
    assert val(ctx, C.byref(a), 0, FAKE, 16, None) == -2
    b, k2 = aset([0, 10, 5])
    assert val(ctx, C.byref(b), 2, FAKE, 16, None) == -4        # not monotone on the host
    b, k3 = aset([0, 2000, 2001])
    assert val(ctx, C.byref(b), 2, FAKE, 16, None) == -4        # more tokens than the grid
    assert val(ctx, C.byref(a), 2, None, 16, None) == -1
    assert val(ctx, C.byref(a), 2, FAKE, 8, None) == -1
    assert val(ctx, C.byref(a), 2, FAKE + 4, 16, None) == -1
    if NO_GPU:
        assert val(ctx, C.byref(a), 2, FAKE, 16, None) == -6


def test_guidance_validation(ctx):
    """Guided steps pair chains 2p / 2p+1: odd batches and unequal pair counts
    are refused before any launch."""
    view1 = abi.rc_cache_view(FAKE, abi.rc_cache_bytes(ctx, 1, 4), 1, 4)
    view2 = abi.rc_cache_view(FAKE, abi.rc_cache_bytes(ctx, 2, 4), 2, 4)
    ws = abi.rc_workspace_bytes(ctx, 2048, 2)
    build, step = abi.LIB.rc_build_cache, abi.LIB.rc_reuse_step
    g = _io(guided=1, guidance_scale=4.5)
    assert build(ctx, C.byref(view1), 0, C.byref(g), FAKE, ws, None) == -2           # odd batch
    assert build(ctx, C.byref(view2), 0, C.byref(_io(guided=2)), FAKE, ws, None) == -1
    assert build(ctx, C.byref(view2), 0, C.byref(_io(guided=1, guidance_scale=float("nan"))), FAKE, ws,
                 None) == -1
    h = (C.c_int32 * 3)(0, 10, 19)
    a = abi.rc_active_set(FAKE, FAKE, C.cast(h, C.POINTER(C.c_int32)), 2)
    assert step(ctx, C.byref(view2), 1, C.byref(a), C.byref(g), None, 1, FAKE, ws, None) == -4  # 10 vs 9
    if NO_GPU:
        assert build(ctx, C.byref(view2), 0, C.byref(g), FAKE, ws, None) == -6


def test_localize_and_logits_validation(ctx):
    loc = abi.LIB.rc_localize_region
    assert loc(ctx, FAKE, 1, 0, 0.3, 1, FAKE, FAKE, FAKE, None, None) == -1
    assert loc(ctx, FAKE, 1, 3, 0.3, 5, FAKE, FAKE, FAKE, None, None) == -1
    assert loc(ctx, None, 1, 3, 0.3, 1, FAKE, FAKE, FAKE, None, None) == -1
    d = (C.c_int32 * 2)(1, 2)
    dp = C.cast(d, C.POINTER(C.c_int32))
    sb = abi.rc_maps_from_logits_scratch_bytes(28, 4096, 2)
    assert sb == 28 * 4096 * 2 * 4
    ml = abi.LIB.rc_maps_from_logits
    assert ml(FAKE, 28, 16, 4096, 121, dp, 2, FAKE, FAKE, sb, None) == -8
    assert ml(FAKE, 28, 16, 4000, 120, dp, 2, FAKE, FAKE, sb, None) == -8
    assert ml(FAKE, 28, 16, 4096, 120, dp, 2, FAKE, FAKE, sb - 4, None) == -5
    bad = (C.c_int32 * 2)(1, 120)
    assert ml(FAKE, 28, 16, 4096, 120, C.cast(bad, C.POINTER(C.c_int32)), 2, FAKE, FAKE, sb, None) == -4
    if NO_GPU:
        assert ml(FAKE, 28, 16, 4096, 120, dp, 2, FAKE, FAKE, sb, None) == -6
        assert abi.LIB.rc_sync(None) == -6
    # the allocation-free variant: same argument checks, and problems beyond
    # its 16 MiB static scratch refused before any device call
    na = abi.LIB.rc_maps_from_logits_noalloc
    assert abi.RC_STATIC_SCRATCH_BYTES == 16 << 20
    assert na(FAKE, 28, 16, 4096, 121, dp, 2, FAKE, None) == -8
    assert na(None, 28, 16, 4096, 120, dp, 2, FAKE, None) == -1
    assert na(FAKE, 28, 16, 4096, 120, C.cast(bad, C.POINTER(C.c_int32)), 2, FAKE, None) == -4
    d8 = (C.c_int32 * 8)(*range(8))
    d8p = C.cast(d8, C.POINTER(C.c_int32))
    assert 33 * 16384 * 8 * 4 > abi.RC_STATIC_SCRATCH_BYTES >= 32 * 16384 * 8 * 4
    assert na(FAKE, 33, 16, 16384, 120, d8p, 8, FAKE, None) == -5
    if NO_GPU:
        assert na(FAKE, 28, 16, 16384, 120, d8p, 8, FAKE, None) == -6


def test_text_and_update_validation(ctx):
    assert abi.LIB.rc_prepare_text(ctx, None, 1, FAKE, FAKE, 1 << 30, None) == -1
    assert abi.LIB.rc_prepare_text(ctx, FAKE, 0, FAKE, FAKE, 1 << 30, None) == -2
    nb = abi.rc_cache_bytes(ctx, 1, 2)
    view = abi.rc_cache_view(FAKE, nb, 1, 2)
    h = (C.c_int32 * 2)(0, 7)
    a = abi.rc_active_set(FAKE, FAKE, C.cast(h, C.POINTER(C.c_int32)), 1)
    assert abi.LIB.rc_update_cache(ctx, C.byref(view), 0, C.byref(a), None, None) == -1
    assert abi.LIB.rc_update_cache(ctx, C.byref(view), 2, C.byref(a), FAKE, None) == -2


def test_hosted_pool_validation(ctx):
    """Host-resident pool: the staging ring holds three entries of every
    chain's slot; the hosted steps validate like the device ones before any
    device call, and refuse fp32 storage."""
    N, C_ = 1024, 1152
    assert abi.rc_staging_bytes(ctx, 2) == 3 * 2 * 3 * N * C_ * 2
    assert abi.rc_staging_bytes(ctx, 0) == 0
    nb = abi.rc_cache_bytes(ctx, 1, 4)
    view = abi.rc_cache_view(FAKE, nb, 1, 4)
    ws = abi.rc_workspace_bytes(ctx, 1024, 1)
    sb = abi.rc_staging_bytes(ctx, 1)
    h = (C.c_int32 * 2)(0, 7)
    a = abi.rc_active_set(FAKE, FAKE, C.cast(h, C.POINTER(C.c_int32)), 1)
    reuse, build = abi.LIB.rc_reuse_step_hosted, abi.LIB.rc_build_cache_hosted
    assert reuse(None, C.byref(view), 1, C.byref(a), C.byref(_io()), FAKE, sb, FAKE, ws, None) == -1
    assert reuse(ctx, C.byref(view), 4, C.byref(a), C.byref(_io()), FAKE, sb, FAKE, ws, None) == -2
    bad = (C.c_int32 * 2)(0, 2000)
    ab = abi.rc_active_set(FAKE, FAKE, C.cast(bad, C.POINTER(C.c_int32)), 1)
    assert reuse(ctx, C.byref(view), 1, C.byref(ab), C.byref(_io()), FAKE, sb, FAKE, ws, None) == -4
    assert build(ctx, C.byref(view), 0, C.byref(_io(timestep=1000)), FAKE, sb, FAKE, ws, None) == -1
    if NO_GPU:
        assert reuse(ctx, C.byref(view), 1, C.byref(a), C.byref(_io()), FAKE, sb, FAKE, ws, None) == -6
        assert build(ctx, C.byref(view), 0, C.byref(_io()), FAKE, sb, FAKE, ws, None) == -6


def test_kernel_timing_classes(ctx):
    abi.rc_set_kernel_timing(ctx, 1)
    ms, n = C.c_double(), C.c_int64()
    abi.rc_get_kernel_timing(ctx, abi.RC_KC_ATTN_SELF, C.byref(ms), C.byref(n))
    assert n.value == 0 and ms.value == 0.0
    with pytest.raises(abi.RcError):
        abi.rc_get_kernel_timing(ctx, abi.RC_KC_COUNT, C.byref(ms), C.byref(n))
    abi.rc_set_kernel_timing(ctx, 0)


def test_kernel_class_table_matches_header():
    """The binding's kernel-class constants and names follow the header's enum."""
    import re
    hdr = open(os.path.join(ROOT, "include", "regioncache.h")).read()
    vals = {k: int(v) for k, v in re.findall(r"(RC_KC_\w+)\s*=\s*(\d+)", hdr)}
    assert vals["RC_KC_COUNT"] == abi.RC_KC_COUNT == len(abi.KERNEL_CLASSES)
    for k, v in vals.items():
        assert getattr(abi, k) == v, k
