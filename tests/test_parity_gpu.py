"""Parity of the HIP path (through the C ABI) with the CPU oracle, and the
method's invariants measured on the GPU.

Tolerances: normwise relative error <= 2e-2 for bf16 storage and <= 1e-4 for
fp32 storage against the float64 oracle; index lists bit-exact; derived masks
equal except for tokens whose normalised score lies within 1e-3 of the
threshold (and their dilation neighbourhoods)."""
import sys

import numpy as np
import pytest
import torch

import oracle as O
import synth
from _cases import (download_slot, gate_failures, oracle_text_kv, relerr, summarize, teacher_forced_dense,
                    teacher_forced_reuse, to_np, tol, upload_slot, weights)

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2608_29809_amd.runtime import ActiveSet, RegionCacheModel, compact_mask, maps_from_logits


def _say(*a):
    print(*a, flush=True, file=sys.stderr)


# --------------------------------------------------------------------------- index work (bit-exact)

@pytest.mark.parametrize("B,N", [(1, 256), (3, 1024), (2, 4096)])
def test_compact_bit_exact(B, N):
    _say("compact", B, N)
    rng = np.random.default_rng(N + B)
    masks = (rng.random((B, N)) < rng.uniform(0.02, 0.6, size=(B, 1))).astype(np.uint8)
    masks[0, :] = 0 if B > 1 else masks[0, :]
    if B > 2:
        masks[2, :] = 1
    act = compact_mask(torch.from_numpy(masks).cuda())
    torch.cuda.synchronize()
    idx_ref, off_ref = O.compact(masks)
    assert list(act.host) == off_ref.tolist()
    assert np.array_equal(to_np(act.idx[:off_ref[-1]]).astype(np.int32), idx_ref)


def _excused(scores, theta, gh, gw, band=1e-3):
    near = (np.abs(scores - theta) < band).any(axis=1)
    return O.dilate(near.reshape(gh, gw), 1).reshape(-1)


def test_localize_maps_vs_oracle():
    _say("localize maps")
    s = synth.shape_c3()
    gh, gw = s.grid_h, s.grid_w
    B, nd = 3, 5
    maps = np.stack([synth.planted_maps(gh * gw, nd, gh, gw, seed=b)[0] for b in range(B)])
    maps[2] = np.random.default_rng(9).uniform(0, 1, maps[2].shape)  # no planted region
    model = _tiny_model_for_grid(gh, gw)
    mask, act = model.localize(torch.from_numpy(maps).cuda(), nd, 0.3, 1)
    torch.cuda.synchronize()
    mask = to_np(mask).astype(np.uint8)
    for b in range(B):
        m_ref, i_ref, sc = O.localize(maps[b], gh, gw, return_scores=True)
        ok = (mask[b] == m_ref) | _excused(sc, 0.3, gh, gw)
        assert ok.all(), b
        g_idx = to_np(act.idx[act.host[b]:act.host[b + 1]]).astype(np.int32)
        assert np.array_equal(g_idx, np.flatnonzero(mask[b]))
        if not _excused(sc, 0.3, gh, gw).any():
            assert np.array_equal(g_idx, i_ref)


def _tiny_model_for_grid(gh, gw):
    shp = synth.ModelShape(layers=1, grid_h=gh, grid_w=gw, dtype="bf16")
    return RegionCacheModel(shp, synth.make_weights(shp, seed=0))


def test_maps_from_logits_small():
    _say("maps_from_logits small")
    Z, delta, blob = synth.make_logits(2, 4, 256, 120, 16, 16, n_delta=4, seed=1)
    g = maps_from_logits(torch.from_numpy(Z).cuda().to(torch.bfloat16), delta)
    torch.cuda.synchronize()
    ref = O.maps_from_logits(Z, delta)
    assert relerr(to_np(g), ref) < 1e-5


def test_localize_logits_full_size():
    """The 1024 px localisation workload: logits [28, 16, 4096, 120] bf16 with
    +3 on the delta columns over a blob -> mask + index list."""
    _say("localize logits full")
    s = synth.shape_c3()
    gh, gw = s.grid_h, s.grid_w
    Z, delta, blob = synth.make_logits(28, 16, gh * gw, 120, gh, gw, n_delta=6, seed=3, frac=0.12)
    Zt = torch.from_numpy(Z).to(torch.bfloat16).cuda()
    g = maps_from_logits(Zt, delta)
    model = _tiny_model_for_grid(gh, gw)
    mask, act = model.localize(g[None].contiguous(), len(delta), 0.3, 1)
    torch.cuda.synchronize()
    ref = O.maps_from_logits(Z, delta)
    assert relerr(to_np(g), ref) < 1e-4
    m_ref, i_ref, sc = O.localize(ref, gh, gw, n_avg=28 * 16, return_scores=True)
    assert not _excused(sc, 0.3, gh, gw).any()
    assert np.array_equal(to_np(mask[0]).astype(np.uint8), m_ref)
    assert np.array_equal(to_np(act.idx[:act.total]).astype(np.int32), i_ref)
    assert np.array_equal(m_ref.astype(bool), O.dilate(blob.reshape(gh, gw).astype(bool), 1).reshape(-1))


# --------------------------------------------------------------------------- single fp32 block (token mode)

@pytest.mark.parametrize("stress", [False, True])
def test_c1_block_fp32(stress):
    """One fp32 block over 256 tokens: dense build, then region reuse over the
    4-aligned rectangle, each against the oracle at 1e-4."""
    _say("c1 fp32 stress", stress)
    case = synth.make_c1(0)
    s = case["shape"]
    W = synth.make_weights(s, seed=0, stress=stress) if stress else case["weights"]
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(1, 1)
    tkv = model.prepare_text(model.to_storage(case["text"][None]))
    tvec = torch.from_numpy(case["t_vec"]).cuda()
    delta = case["delta"]
    maps = torch.zeros((1, s.tokens, len(delta)), device="cuda")
    model.build_cache(cache, 0, model.to_storage(case["x_prev"][None]), 0, -1, tkv, delta, maps, t_vec=tvec)
    torch.cuda.synchronize()
    Xd, Kd, Vd, md = O.dense_block_tokens(s, W, case["x_prev"], case["t_vec"], case["text"], delta)
    got = download_slot(cache, 0, 1, 1)
    assert relerr(got["H"][0, 0], Xd) < 1e-4
    assert relerr(got["K"][0, 0], Kd) < 1e-4
    assert relerr(got["V"][0, 0], Vd) < 1e-4
    assert relerr(to_np(maps[0]), md) < 1e-4
    # reuse over the rectangle, starting from the oracle's own dense cache
    upload_slot(model, cache, 0, dict(K=Kd[None, None].astype(np.float32), V=Vd[None, None].astype(np.float32),
                                      H=Xd[None, None].astype(np.float32)))
    idx = np.flatnonzero(case["mask"])
    act = ActiveSet.from_lists([idx])
    maps.zero_()
    model.reuse_step(cache, 0, act, model.to_storage(case["x_new"][None]), 0, -1, tkv, delta, maps, t_vec=tvec)
    torch.cuda.synchronize()
    Xr, Kr, Vr, Hr, mr = O.reuse_block_tokens(s, W, case["x_new"], idx, case["t_vec"], case["text"], Kd, Vd, Xd,
                                              delta)
    got = download_slot(cache, 0, 1, 1)
    assert relerr(got["H"][0, 0], Hr) < 1e-4
    assert relerr(got["K"][0, 0], Kr) < 1e-4
    assert relerr(got["V"][0, 0], Vr) < 1e-4
    # per-block delta of the active rows is also within tolerance
    assert relerr(got["H"][0, 0][idx] - case["x_new"][idx], Hr[idx] - case["x_new"][idx]) < 1e-4
    full_maps = np.zeros_like(md)
    full_maps[idx] = mr
    assert relerr(to_np(maps[0]), full_maps) < 1e-4
    inactive = np.setdiff1d(np.arange(s.tokens), idx)
    assert np.array_equal(got["H"][0, 0][inactive], Xd[inactive].astype(np.float32))


# --------------------------------------------------------------------------- full-model steps (patch mode)

def _reuse_case(shape, seed, per_chain_idx, t=500, t_next=450, stress=False, delta=(3, 17, 64), step=1,
                steps=2, fuse=True):
    W = weights(shape, seed, stress)
    B = len(per_chain_idx)
    txt = synth.make_text(shape, B, seed)
    lat = synth.make_latent(shape, B, seed)
    lat_next_cached = synth.make_latent(shape, B, seed, stream=77)
    slot = synth.make_cache_slot(shape, B, seed)
    model = RegionCacheModel(shape, W)
    cache = model.alloc_cache(B, steps)
    upload_slot(model, cache, step, slot)
    for b in range(B):
        cache.latent(b, step + 1).copy_(torch.from_numpy(lat_next_cached[b]))
    tkv = model.prepare_text(model.to_storage(txt))
    act = ActiveSet.from_lists(per_chain_idx)
    maps = torch.zeros((B, shape.tokens, len(delta)), device="cuda")
    lat_out = torch.empty(lat.shape, device="cuda")
    lat_in = torch.from_numpy(lat).cuda()
    hid = None
    if not fuse:
        hid = torch.empty((shape.layers, max(act.total, 1), shape.hidden), dtype=model.dtype, device="cuda")
    model.reuse_step(cache, step, act, lat_in, t, t_next, tkv, list(delta), maps, lat_out, fuse=fuse,
                     active_hidden=hid)
    if not fuse:
        model.update_cache(cache, step, act, hid)
    torch.cuda.synchronize()
    got = download_slot(cache, step, shape.layers, B)
    got["latent_next"] = to_np(lat_out)
    got["maps"] = to_np(maps)
    got["traj_next"] = np.stack([to_np(cache.latent(b, step + 1)) for b in range(B)])
    refs, tkvs = [], []
    for b in range(B):
        tkv_o = oracle_text_kv(shape, W, txt[b])
        tkvs.append(tkv_o)
        cs = dict(K=slot["K"][:, b], V=slot["V"][:, b], H=slot["H"][:, b])
        refs.append(O.reuse_step(shape, W, lat[b], t, t_next, tkv_o, per_chain_idx[b], cs, lat_next_cached[b],
                                 np.array(delta)))
    return got, refs, dict(slot=slot, lat_next_cached=lat_next_cached, model=model, cache=cache, W=W, lat=lat,
                           tkv_o=tkvs, t=t)


def _check_teacher_forced(shape, got, per_chain_idx, ctx):
    """Per-block gate with re-synchronised inputs (tests/_cases.py): each
    block of the oracle is fed the GPU's previous block output; block
    outputs, keys and values of the active rows within the bf16 tolerance in
    every block, and their per-block change within it plus the rounding
    floor of its measurement from the storage-rounded block outputs."""
    tl = tol(shape)
    for b, idx in enumerate(per_chain_idx):
        idx = np.asarray(idx)
        if idx.size == 0:
            continue
        cache_b = {k: ctx["slot"][k][:, b] for k in ("K", "V", "H")}
        got_b = {k: got[k][:, b] for k in ("K", "V", "H")}
        per = teacher_forced_reuse(shape, ctx["W"], ctx["lat"][b], ctx["t"], ctx["tkv_o"][b], idx, cache_b, got_b)
        w = summarize(per)
        _say(f"chain {b} R={idx.size} per block (re-synchronised), worst: " +
             " ".join(f"{k} {v:.2e}" for k, v in w.items()))
        _say(f"chain {b} per block, median: " +
             " ".join(f"{k} {np.median([e[k] for e in per]):.2e}" for k in ("H", "dH", "K", "V")))
        bad = gate_failures(per, tl)
        assert not bad, (b, bad[:3])


def _check_reuse(shape, got, refs, per_chain_idx, ctx, tolerance=None):
    tl = tolerance or tol(shape)
    for b, r in enumerate(refs):
        idx = np.asarray(per_chain_idx[b])
        inact = np.setdiff1d(np.arange(shape.tokens), idx)
        # inactive rows: the cache, bit for bit
        assert np.array_equal(got["H"][:, b][:, inact], ctx["slot"]["H"][:, b][:, inact]), b
        assert np.array_equal(got["K"][:, b][:, :, inact], ctx["slot"]["K"][:, b][:, :, inact]), b
        assert np.array_equal(got["V"][:, b][:, :, inact], ctx["slot"]["V"][:, b][:, :, inact]), b
        if idx.size == 0:
            assert np.array_equal(got["latent_next"][b], ctx["lat_next_cached"][b])
            continue
        e_h = relerr(got["H"][:, b][:, idx], r["H"][:, idx])
        e_k = relerr(got["K"][:, b][:, :, idx], r["K"][:, :, idx])
        e_v = relerr(got["V"][:, b][:, :, idx], r["V"][:, :, idx])
        e_l = relerr(got["latent_next"][b], r["latent_next"])
        e_m = relerr(got["maps"][b], r["maps"])
        _say(f"chain {b} R={idx.size}: H {e_h:.2e} K {e_k:.2e} V {e_v:.2e} latent {e_l:.2e} maps {e_m:.2e}")
        assert e_h < tl and e_k < tl and e_v < tl and e_l < tl and e_m < tl
        assert np.array_equal(got["traj_next"][b], got["latent_next"][b])
        # inactive patches of the latent are the cached trajectory's
        lp = O.latent_to_patches(got["latent_next"][b], 2)
        cp = O.latent_to_patches(ctx["lat_next_cached"][b], 2)
        assert np.array_equal(lp[inact], cp[inact])


@pytest.mark.timeout(300)
@pytest.mark.parametrize("stress", [False, True])
def test_c2_reuse_step_full_model(stress):
    """512 px, 28 blocks, bf16, t = 500, a 15 % rectangle (11 x 14 tokens).
    With the stress weights (every branch moves the state by O(1)) each
    block is also gated with re-synchronised inputs."""
    _say("c2 reuse full, stress", stress)
    s = synth.shape_c2()
    idx = np.flatnonzero(synth.rect_mask(s.grid_h, s.grid_w, 11, 14, 9, 5))
    got, refs, ctx = _reuse_case(s, 0, [idx], stress=stress)
    if stress:
        _check_teacher_forced(s, got, [idx], ctx)
        _report_free_running(s, got, refs, [idx])
    else:
        _check_reuse(s, got, refs, [idx], ctx)


def _report_free_running(shape, got, refs, per_chain_idx):
    """Errors of the whole step against the free-running oracle (each side
    feeding its own blocks through all blocks), beside the per-block gate:
    within 2e-2 as well."""
    for b, r in enumerate(refs):
        idx = np.asarray(per_chain_idx[b])
        if idx.size == 0:
            continue
        e = dict(H=relerr(got["H"][:, b][:, idx], r["H"][:, idx]),
                 K=relerr(got["K"][:, b][:, :, idx], r["K"][:, :, idx]),
                 latent=relerr(got["latent_next"][b], r["latent_next"]), maps=relerr(got["maps"][b], r["maps"]))
        _say(f"chain {b} free-running whole step: " + " ".join(f"{k} {v:.2e}" for k, v in e.items()))
        assert max(e.values()) < tol(shape), (b, e)


@pytest.mark.parametrize("counts", [[1, 63, 0], [64, 65, 129], [127, 128, 1024]])
def test_ragged_multichain_stress(counts):
    """Several chains with unequal, ragged active counts (including 0 and N),
    peaky weights so every block moves the state by O(1)."""
    _say("ragged", counts)
    s = synth.ModelShape(layers=2, grid_h=32, grid_w=32, dtype="bf16")
    rng = np.random.default_rng(sum(counts))
    per = [np.sort(rng.choice(s.tokens, size=c, replace=False)) for c in counts]
    got, refs, ctx = _reuse_case(s, 5, per, stress=True, t=900, t_next=850)
    _check_reuse(s, got, refs, per, ctx)
    # with the stress weights every block moves the state by O(1), so the
    # per-block change of the active rows is gated too (the hidden state alone
    # is dominated by the residual stream)
    for b, r in enumerate(refs):
        idx = per[b]
        if idx.size == 0:
            continue
        dg = np.diff(got["H"][:, b][:, idx].astype(np.float64), axis=0)
        dr = np.diff(r["H"][:, idx].astype(np.float64), axis=0)
        e = relerr(dg, dr)
        _say(f"chain {b} per-block delta {e:.2e}")
        assert e < tol(s)


def test_reuse_unfused_update_matches_fused():
    s = synth.ModelShape(layers=2, grid_h=32, grid_w=32, dtype="bf16")
    idx = [np.arange(100, 300)]
    g1, _, _ = _reuse_case(s, 2, idx, fuse=True)
    g2, _, _ = _reuse_case(s, 2, idx, fuse=False)
    for k in ("H", "K", "V", "latent_next", "maps"):
        assert np.array_equal(g1[k], g2[k]), k


def test_dense_step_vs_oracle():
    """Build-cache (dense) step: every token, 4 blocks at 1024 tokens, and the
    all-active reuse step gives the same result bit for bit."""
    _say("dense step")
    s = synth.ModelShape(layers=4, grid_h=32, grid_w=32, dtype="bf16")
    W = synth.make_weights(s, seed=4, stress=True)
    txt = synth.make_text(s, 1, 4)
    lat = synth.make_latent(s, 1, 4)
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(1, 3)
    tkv = model.prepare_text(model.to_storage(txt))
    delta = [0, 50, 119]
    maps = torch.zeros((1, s.tokens, 3), device="cuda")
    out = torch.empty(lat.shape, device="cuda")
    model.build_cache(cache, 1, torch.from_numpy(lat).cuda(), 700, 650, tkv, delta, maps, out)
    torch.cuda.synchronize()
    got = download_slot(cache, 1, s.layers, 1)
    ref = O.dense_step(s, W, lat[0], 700, 650, oracle_text_kv(s, W, txt[0]), np.array(delta))
    for k in ("H", "K", "V"):
        e = relerr(got[k][:, 0], ref[k])
        _say(k, e)
        assert e < 2e-2
    assert relerr(to_np(out)[0], ref["latent_next"]) < 2e-2
    assert relerr(to_np(maps)[0], ref["maps"]) < 2e-2
    assert np.array_equal(to_np(cache.latent(0, 1)), lat[0])
    assert np.array_equal(to_np(cache.latent(0, 2)), to_np(out)[0])
    # all-active reuse == dense, bit for bit
    cache2 = model.alloc_cache(1, 3)
    cache2.buf.copy_(cache.buf)
    maps2 = torch.zeros_like(maps)
    out2 = torch.empty_like(out)
    model.reuse_step(cache2, 1, ActiveSet.from_lists([np.arange(s.tokens)]), torch.from_numpy(lat).cuda(), 700,
                     650, tkv, delta, maps2, out2)
    torch.cuda.synchronize()
    assert torch.equal(cache2.buf, cache.buf)
    assert torch.equal(out2, out) and torch.equal(maps2, maps)


@pytest.mark.timeout(300)
def test_dense_step_300_chains():
    """A dense step of 300 chains (more than one 256-thread block of chain
    offsets): one block on an 8 x 8 grid, 19200 rows.  Chains on both sides
    of 256 match the oracle, so every chain's row range was set."""
    _say("dense step, 300 chains")
    s = synth.ModelShape(layers=1, grid_h=8, grid_w=8, text_dim=128, dtype="bf16")
    B = 300
    W = synth.make_weights(s, seed=16, stress=True)
    txt = synth.make_text(s, B, 16)
    lat = synth.make_latent(s, B, 16)
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(B, 1)
    tkv = model.prepare_text(model.to_storage(txt))
    out = torch.empty(lat.shape, device="cuda")
    model.build_cache(cache, 0, torch.from_numpy(lat).cuda(), 600, 550, tkv, latent_out=out)
    torch.cuda.synchronize()
    o = to_np(out)
    assert np.isfinite(o).all()
    for b in (0, 1, 255, 256, 257, 299):
        ref = O.dense_step(s, W, lat[b], 600, 550, oracle_text_kv(s, W, txt[b]))
        e_h = relerr(to_np(cache.H(b, 0, 0)), ref["H"][0])
        e_l = relerr(o[b], ref["latent_next"])
        _say(f"chain {b}: H {e_h:.2e} latent {e_l:.2e}")
        assert e_h < 2e-2 and e_l < 2e-2


@pytest.mark.gpu
@pytest.mark.timeout(300)
def test_dense_step_two_chains():
    """Dense step of two chains at 1024 tokens each: 2048 rows per GEMM (the
    128-row tile plan for the wide projections), both chains vs the oracle."""
    _say("dense step, two chains")
    s = synth.ModelShape(layers=2, grid_h=32, grid_w=32, dtype="bf16")
    W = synth.make_weights(s, seed=6, stress=True)
    txt = synth.make_text(s, 2, 6)
    lat = synth.make_latent(s, 2, 6)
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(2, 2)
    tkv = model.prepare_text(model.to_storage(txt))
    out = torch.empty(lat.shape, device="cuda")
    model.build_cache(cache, 0, torch.from_numpy(lat).cuda(), 900, 850, tkv, latent_out=out)
    torch.cuda.synchronize()
    got = download_slot(cache, 0, s.layers, 2)
    for b in range(2):
        ref = O.dense_step(s, W, lat[b], 900, 850, oracle_text_kv(s, W, txt[b]))
        for k in ("H", "K", "V"):
            e = relerr(got[k][:, b], ref[k])
            _say(b, k, e)
            assert e < 2e-2
        assert relerr(to_np(out)[b], ref["latent_next"]) < 2e-2


@pytest.mark.gpu
@pytest.mark.timeout(400)
def test_dense_step_full_grid():
    """Build-cache (dense) step at 1024 px: 4096 tokens of one chain, two
    blocks, as the benchmark's dense step launches them (4096-row GEMMs on
    128 x 128 tiles two stages deep, the unsplit MLP-down GEMM, 4096-query
    self-attention) against the oracle, maps included."""
    _say("dense step, 4096 tokens")
    s = synth.ModelShape(layers=2, grid_h=64, grid_w=64, dtype="bf16")
    W = synth.make_weights(s, seed=9, stress=True)
    txt = synth.make_text(s, 1, 9)
    lat = synth.make_latent(s, 1, 9)
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(1, 2)
    tkv = model.prepare_text(model.to_storage(txt))
    delta = [2, 40, 77, 119]
    maps = torch.zeros((1, s.tokens, len(delta)), device="cuda")
    out = torch.empty(lat.shape, device="cuda")
    model.build_cache(cache, 0, torch.from_numpy(lat).cuda(), 950, 900, tkv, delta, maps, out)
    torch.cuda.synchronize()
    got = download_slot(cache, 0, s.layers, 1)
    ref = O.dense_step(s, W, lat[0], 950, 900, oracle_text_kv(s, W, txt[0]), np.array(delta))
    for k in ("H", "K", "V"):
        e = relerr(got[k][:, 0], ref[k])
        _say(k, e)
        assert e < 2e-2
    e_l, e_m = relerr(to_np(out)[0], ref["latent_next"]), relerr(to_np(maps)[0], ref["maps"])
    _say("latent", e_l, "maps", e_m)
    assert e_l < 2e-2 and e_m < 2e-2
    per = teacher_forced_dense(s, W, lat[0], 950, oracle_text_kv(s, W, txt[0]),
                               {k: got[k][:, 0] for k in ("K", "V", "H")})
    _say("per block (re-synchronised), worst: " + " ".join(f"{k} {v:.2e}" for k, v in summarize(per).items()))
    assert not gate_failures(per, 2e-2)


@pytest.mark.gpu
@pytest.mark.timeout(400)
def test_four_chains_mixed_fractions():
    """Four 1024 px chains whose edit regions cover about 5, 10, 25 and 50 % of
    their tokens (blob masks), two blocks: the batch-of-four workload's row
    count (over 3072 rows, so the large-row tile plans and the unsplit
    MLP-down GEMM run on the reuse path) and four chains' keys in one
    attention launch."""
    s = synth.ModelShape(layers=2, grid_h=64, grid_w=64, dtype="bf16")
    per = [np.flatnonzero(synth.blob_mask(64, 64, f, 2, np.random.default_rng(20 + i)))
           for i, f in enumerate((0.05, 0.10, 0.25, 0.50))]
    _say("four chains", [p.size for p in per])
    assert sum(p.size for p in per) > 3072
    got, refs, ctx = _reuse_case(s, 12, per, t=640, t_next=590, stress=True)
    _check_reuse(s, got, refs, per, ctx)
    _check_teacher_forced(s, got, per, ctx)


@pytest.mark.gpu
@pytest.mark.timeout(400)
@pytest.mark.parametrize("frac", [0.05, 0.10, 0.50])
def test_fraction_sweep_workloads(frac):
    """The batch active-fraction workload (four 1024 px chains with the masks
    the benchmark's sweep draws: 820, 1640 and 8192 rows) in its launch
    configuration, two blocks, against the oracle."""
    s = synth.ModelShape(layers=2, grid_h=64, grid_w=64, dtype="bf16")
    per = synth.sweep_regions(0, frac)
    _say("fraction sweep", frac, [p.size for p in per])
    got, refs, ctx = _reuse_case(s, 13, per, t=700, t_next=650, stress=True)
    _check_reuse(s, got, refs, per, ctx)
    _check_teacher_forced(s, got, per, ctx)


@pytest.mark.gpu
@pytest.mark.timeout(400)
def test_all_active_four_chains_equals_dense():
    """The 100 % point of the batch sweep at full size: four 1024 px chains,
    28 blocks, every token active (16384 rows).  The region step over a slot
    whose keys, values and hidden states were poisoned equals the dense step
    bit for bit (slot, maps, latents)."""
    _say("all-active, four chains, 28 blocks")
    s = synth.shape_c3()
    B = 4
    W = synth.make_weights(s, seed=14)
    txt = synth.make_text(s, B, 14)
    lat = torch.from_numpy(synth.make_latent(s, B, 14)).cuda()
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(B, 2)
    tkv = model.prepare_text(model.to_storage(txt))
    delta = [1, 60, 118]
    maps = torch.zeros((B, s.tokens, 3), device="cuda")
    out = torch.empty_like(lat)
    model.build_cache(cache, 0, lat, 920, 870, tkv, delta, maps, out)
    cache2 = model.alloc_cache(B, 2)
    cache2.buf.copy_(cache.buf)
    for b in range(B):
        for l in range(s.layers):
            cache2.K(b, 0, l).fill_(float("nan"))
            cache2.V(b, 0, l).fill_(float("nan"))
            cache2.H(b, 0, l).fill_(float("nan"))
    maps2 = torch.zeros_like(maps)
    out2 = torch.empty_like(out)
    model.reuse_step(cache2, 0, ActiveSet.from_lists([np.arange(s.tokens)] * B), lat, 920, 870, tkv, delta, maps2,
                     out2)
    torch.cuda.synchronize()
    assert torch.equal(cache2.buf, cache.buf)
    assert torch.equal(out2, out) and torch.equal(maps2, maps)
    assert torch.isfinite(out).all() and bool((maps > 0).all())


def test_empty_mask_and_poison():
    """No active token: slot unchanged and latent = cached trajectory.  Then
    NaN in the stale cached rows of the active tokens never reaches an output."""
    s = synth.ModelShape(layers=2, grid_h=32, grid_w=32, dtype="bf16")
    W = synth.make_weights(s, seed=6)
    txt = synth.make_text(s, 1, 6)
    lat = synth.make_latent(s, 1, 6)
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(1, 2)
    upload_slot(model, cache, 0, synth.make_cache_slot(s, 1, 6))
    cache.latent(0, 1).copy_(torch.from_numpy(synth.make_latent(s, 1, 7)[0]))
    before = cache.buf.clone()
    tkv = model.prepare_text(model.to_storage(txt))
    out = torch.empty(lat.shape, device="cuda")
    model.reuse_step(cache, 0, ActiveSet.from_lists([np.zeros(0, np.int32)]), torch.from_numpy(lat).cuda(), 500,
                     450, tkv, latent_out=out)
    torch.cuda.synchronize()
    assert torch.equal(cache.buf, before)
    assert torch.equal(out[0], cache.latent(0, 1))
    # poison
    idx = np.arange(200, 260)
    for l in range(s.layers):
        cache.K(0, 0, l)[:, idx] = float("nan")
        cache.V(0, 0, l)[:, idx] = float("nan")
        cache.H(0, 0, l)[idx] = float("nan")
    model.reuse_step(cache, 0, ActiveSet.from_lists([idx]), torch.from_numpy(lat).cuda(), 500, 450, tkv,
                     latent_out=out)
    torch.cuda.synchronize()
    for l in range(s.layers):
        assert torch.isfinite(cache.K(0, 0, l).float()).all()
        assert torch.isfinite(cache.V(0, 0, l).float()).all()
        assert torch.isfinite(cache.H(0, 0, l).float()).all()
    assert torch.isfinite(out).all()


def test_determinism():
    s = synth.ModelShape(layers=2, grid_h=64, grid_w=64, dtype="bf16")
    idx = [np.flatnonzero(synth.blob_mask(64, 64, 0.15, 2, np.random.default_rng(1)))]
    g1, _, _ = _reuse_case(s, 8, idx)
    g2, _, _ = _reuse_case(s, 8, idx)
    for k in ("H", "K", "V", "latent_next", "maps"):
        assert np.array_equal(g1[k], g2[k]), k


@pytest.mark.timeout(400)
@pytest.mark.parametrize("region", ["blob15", "bench"])
def test_c3_reuse_step_full_size(region):
    """1024 px (4096 tokens), 28 blocks, bf16, one reuse step: a 15 % two-blob
    mask (614 rows), and the benchmark's own edit region (seed 0, 723 rows),
    which runs every kernel in the launch configuration the benchmark times."""
    _say("c3 reuse full", region)
    s = synth.shape_c3()
    if region == "bench":
        idx = np.flatnonzero(synth.c3_edit_region(0)[0])
        assert idx.size == 723
    else:
        idx = np.flatnonzero(synth.blob_mask(64, 64, 0.15, 2, np.random.default_rng(0)))
    got, refs, ctx = _reuse_case(s, 0, [idx], t=842, t_next=789)
    _check_reuse(s, got, refs, [idx], ctx)


@pytest.mark.timeout(600)
def test_c3_reuse_step_full_size_stress():
    """The benchmark's own 1024 px region (723 rows, 4096 keys per head, five
    key splits plus the combine, 28 blocks) with the stress weights: every
    block gated with re-synchronised inputs (block outputs, their per-block
    change, keys and values of the active rows), so a wrong self-attention
    in the launch configuration the benchmark times cannot hide behind the
    residual stream."""
    _say("c3 reuse full, stress, bench region")
    s = synth.shape_c3()
    idx = np.flatnonzero(synth.c3_edit_region(0)[0])
    assert idx.size == 723
    got, refs, ctx = _reuse_case(s, 0, [idx], t=842, t_next=789, stress=True)
    _check_teacher_forced(s, got, [idx], ctx)
    _report_free_running(s, got, refs, [idx])
    # outside the region the slot is the cache, bit for bit
    inact = np.setdiff1d(np.arange(s.tokens), idx)
    assert np.array_equal(got["H"][:, 0][:, inact], ctx["slot"]["H"][:, 0][:, inact])
    assert np.array_equal(got["K"][:, 0][:, :, inact], ctx["slot"]["K"][:, 0][:, :, inact])


@pytest.mark.gpu
@pytest.mark.timeout(400)
@pytest.mark.parametrize("region", ["blob10", "bench15"])
def test_reuse_step_2048px(region):
    """2048 px (128 x 128 = 16384 tokens), two blocks: a 10 % blob region and
    the benchmark's resolution-workload region (15 %, 2458 rows): the largest
    grid the library takes, keys of all 16384 tokens per head."""
    _say("2048 px reuse", region)
    s = synth.ModelShape(layers=2, grid_h=128, grid_w=128, dtype="bf16")
    if region == "bench15":
        idx = synth.resolution_region(0, 128)
        assert idx.size == 2458
    else:
        idx = np.flatnonzero(synth.blob_mask(128, 128, 0.10, 2, np.random.default_rng(3)))
    got, refs, ctx = _reuse_case(s, 3, [idx], t=600, t_next=550, stress=True)
    _check_reuse(s, got, refs, [idx], ctx)
    _check_teacher_forced(s, got, [idx], ctx)


@pytest.mark.gpu
@pytest.mark.timeout(400)
def test_dense_step_2048px_sampled_rows():
    """Dense step at 2048 px (16384 tokens, two blocks), as the resolution
    workload launches it: the first block's keys and values of 256 sampled
    tokens against the oracle evaluated row by row (patch and position
    embedding, LayerNorm, modulation, QKV projection), and the all-active
    region step over a poisoned slot equal to the dense step bit for bit."""
    _say("2048 px dense, sampled rows")
    s = synth.ModelShape(layers=2, grid_h=128, grid_w=128, dtype="bf16")
    W = synth.make_weights(s, seed=15)
    txt = synth.make_text(s, 1, 15)
    lat = synth.make_latent(s, 1, 15)
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(1, 2)
    tkv = model.prepare_text(model.to_storage(txt))
    lat_d = torch.from_numpy(lat).cuda()
    out = torch.empty_like(lat_d)
    model.build_cache(cache, 0, lat_d, 810, 760, tkv, latent_out=out)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(15).choice(s.tokens, 256, replace=False))
    C, H, D = s.hidden, s.heads, s.head_dim
    t0 = O.adaln_single(W, O.timestep_embedding(W, 810))
    lw = W["layers"][0]
    mod = O.layer_modulation(lw, t0)
    X = O.patch_embed(W, lat[0], s.grid_h, s.grid_w, s.patch)[rows]
    qkv = O.modulate(O.layer_norm(X), mod[0], mod[1]) @ lw["qkv_w"].astype(np.float64).T + lw["qkv_b"]
    k_ref = qkv[:, C:2 * C].reshape(-1, H, D).transpose(1, 0, 2)
    v_ref = qkv[:, 2 * C:].reshape(-1, H, D).transpose(1, 0, 2)
    e_k = relerr(to_np(cache.K(0, 0, 0))[:, rows], k_ref)
    e_v = relerr(to_np(cache.V(0, 0, 0))[:, rows], v_ref)
    _say(f"block 0 sampled rows: K {e_k:.2e} V {e_v:.2e}")
    assert e_k < 2e-2 and e_v < 2e-2
    cache2 = model.alloc_cache(1, 2)
    cache2.buf.copy_(cache.buf)
    for l in range(s.layers):
        cache2.K(0, 0, l).fill_(float("nan"))
        cache2.V(0, 0, l).fill_(float("nan"))
        cache2.H(0, 0, l).fill_(float("nan"))
    out2 = torch.empty_like(out)
    model.reuse_step(cache2, 0, ActiveSet.from_lists([np.arange(s.tokens)]), lat_d, 810, 760, tkv, latent_out=out2)
    torch.cuda.synchronize()
    assert torch.equal(cache2.buf, cache.buf) and torch.equal(out2, out)


@pytest.mark.gpu
@pytest.mark.timeout(300)
def test_padded_prompts_per_chain():
    """Prompts of different lengths in one batch (padding masked per chain):
    the reuse step and the dense step equal the oracle run on each chain's
    unpadded prompt, maps included."""
    _say("padded prompts")
    s = synth.ModelShape(layers=2, grid_h=32, grid_w=32, dtype="bf16")
    W = weights(s, 8, True)
    B, valid, delta = 3, [57, 120, 1], (0, 17, 40)
    txt = synth.make_text(s, B, 8)
    lat = synth.make_latent(s, B, 8)
    lat_next_cached = synth.make_latent(s, B, 8, stream=77)
    slot = synth.make_cache_slot(s, B, 8)
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(B, 2)
    upload_slot(model, cache, 1, slot)
    for b in range(B):
        cache.latent(b, 2).copy_(torch.from_numpy(lat_next_cached[b]))
    tkv = model.prepare_text(model.to_storage(txt))
    tv = torch.tensor(valid, dtype=torch.int32, device="cuda")
    rng = np.random.default_rng(8)
    per = [np.sort(rng.choice(s.tokens, n, replace=False)) for n in (150, 64, 300)]
    act = ActiveSet.from_lists(per)
    maps = torch.zeros((B, s.tokens, len(delta)), device="cuda")
    out = torch.empty(lat.shape, device="cuda")
    model.reuse_step(cache, 1, act, torch.from_numpy(lat).cuda(), 500, 450, tkv, list(delta), maps, out,
                     text_valid=tv)
    torch.cuda.synchronize()
    got = download_slot(cache, 1, s.layers, B)
    for b in range(B):
        L = valid[b]
        tkv_o = oracle_text_kv(s, W, txt[b][:L])
        d_ok = [d for d in delta if d < L]
        cs = dict(K=slot["K"][:, b], V=slot["V"][:, b], H=slot["H"][:, b])
        ref = O.reuse_step(s, W, lat[b], 500, 450, tkv_o, per[b], cs, lat_next_cached[b], np.array(d_ok))
        for k in ("H", "K", "V"):
            e = relerr(got[k][:, b][:, per[b]] if k == "H" else got[k][:, b][:, :, per[b]],
                       ref[k][:, per[b]] if k == "H" else ref[k][:, :, per[b]])
            _say(b, L, k, e)
            assert e < 2e-2
        assert relerr(to_np(out)[b], ref["latent_next"]) < 2e-2
        m = to_np(maps)[b]
        for j, d in enumerate(delta):
            if d < L:
                assert relerr(m[per[b], j], ref["maps"][per[b], d_ok.index(d)]) < 2e-2
            else:
                assert np.all(m[:, j] == 0.0)
    # dense step, same prompts
    out2 = torch.empty_like(out)
    model.build_cache(cache, 0, torch.from_numpy(lat).cuda(), 700, 650, tkv, latent_out=out2, text_valid=tv)
    torch.cuda.synchronize()
    got = download_slot(cache, 0, s.layers, B)
    for b in range(B):
        ref = O.dense_step(s, W, lat[b], 700, 650, oracle_text_kv(s, W, txt[b][:valid[b]]))
        assert relerr(got["H"][:, b], ref["H"]) < 2e-2
        assert relerr(to_np(out2)[b], ref["latent_next"]) < 2e-2


@pytest.mark.gpu
@pytest.mark.timeout(300)
def test_guided_pair_reuse_and_dense():
    """Classifier-free guidance: chains 0/1 are the conditional and null-prompt
    branches of one image (own caches, same latent, same region).  Both get
    the DDIM update of eps_u + 4.5 (eps_c - eps_u); each branch's cache
    matches its own unguided oracle step."""
    _say("guided pair")
    s = synth.ModelShape(layers=2, grid_h=32, grid_w=32, dtype="bf16")
    W = weights(s, 9, True)
    g = 4.5
    txt = synth.make_text(s, 2, 9)
    txt[1] = 0.0  # null prompt features
    lat1 = synth.make_latent(s, 1, 9)
    lat = np.concatenate([lat1, lat1])
    lnc1 = synth.make_latent(s, 1, 9, stream=77)
    lnc = np.concatenate([lnc1, lnc1])
    slot = synth.make_cache_slot(s, 2, 9)
    model = RegionCacheModel(s, W)
    cache = model.alloc_cache(2, 2)
    upload_slot(model, cache, 1, slot)
    for b in range(2):
        cache.latent(b, 2).copy_(torch.from_numpy(lnc[b]))
    tkv = model.prepare_text(model.to_storage(txt))
    idx = np.sort(np.random.default_rng(9).choice(s.tokens, 200, replace=False))
    act = ActiveSet.from_lists([idx, idx])
    out = torch.empty(lat.shape, device="cuda")
    model.reuse_step(cache, 1, act, torch.from_numpy(lat).cuda(), 500, 450, tkv, latent_out=out, guidance=g)
    torch.cuda.synchronize()
    got = download_slot(cache, 1, s.layers, 2)
    o = to_np(out)
    assert np.array_equal(o[0], o[1])
    assert np.array_equal(to_np(cache.latent(0, 2)), to_np(cache.latent(1, 2)))
    refs = []
    for b in range(2):
        cs = dict(K=slot["K"][:, b], V=slot["V"][:, b], H=slot["H"][:, b])
        refs.append(O.reuse_step(s, W, lat[b], 500, 450, oracle_text_kv(s, W, txt[b]), idx, cs, lnc[b]))
        for k in ("H", "K", "V"):
            e = relerr(got[k][:, b][:, idx] if k == "H" else got[k][:, b][:, :, idx],
                       refs[b][k][:, idx] if k == "H" else refs[b][k][:, :, idx])
            assert e < 2e-2, (b, k, e)
    ref_lat = O.guided_latent(s, lat1[0], lnc1[0], idx, refs[0]["eps"], refs[1]["eps"], g, 500, 450)
    e = relerr(o[0], ref_lat)
    _say("guided latent", e)
    assert e < 2e-2
    # the unguided result differs: guidance is applied
    assert relerr(o[0], refs[0]["latent_next"]) > 1e-3
    # dense step of the pair
    out2 = torch.empty_like(out)
    model.build_cache(cache, 0, torch.from_numpy(lat).cuda(), 700, 650, tkv, latent_out=out2, guidance=g)
    torch.cuda.synchronize()
    dc = O.dense_step(s, W, lat1[0], 700, 650, oracle_text_kv(s, W, txt[0]))
    du = O.dense_step(s, W, lat1[0], 700, 650, oracle_text_kv(s, W, txt[1]))
    ref2 = O.guided_latent(s, lat1[0], lat1[0], np.arange(s.tokens), dc["eps"], du["eps"], g, 700, 650)
    o2 = to_np(out2)
    assert np.array_equal(o2[0], o2[1])
    assert relerr(o2[0], ref2) < 2e-2

