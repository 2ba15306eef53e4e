"""Pins of the CPU oracle against things other than itself: library routines,
closed forms, special cases that collapse the block to a hand-checkable
expression, brute force on tiny inputs, invariants of the method, and the
values the paper prints (tests/golden)."""
import json
import math
import os

import numpy as np
import pytest
import scipy.ndimage
import scipy.special
import torch
import torch.nn.functional as F

import oracle as O
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

# a tiny model with a non-square token grid so that row/column swaps show up
TINY = synth.ModelShape(hidden=64, heads=4, head_dim=16, mlp=256, layers=2, text_len=8,
                        text_dim=32, grid_h=6, grid_w=5, dtype="f32")


def _tiny_weights(seed=0, stress=True):
    return synth.make_weights(TINY, seed=seed, std=0.2, stress=stress)


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# --------------------------------------------------------------------------- library special cases

def test_layer_norm_matches_torch():
    x = np.random.default_rng(1).standard_normal((7, 33)) * 3 + 1
    ref = F.layer_norm(torch.from_numpy(x), (33,), eps=1e-6).numpy()
    assert _rel(O.layer_norm(x), ref) < 1e-13


def test_gelu_silu_match_torch():
    x = np.linspace(-8, 8, 1001)
    assert _rel(O.gelu_tanh(x), F.gelu(torch.from_numpy(x), approximate="tanh").numpy()) < 1e-13
    assert _rel(O.silu(x), F.silu(torch.from_numpy(x)).numpy()) < 1e-13


def test_softmax_matches_scipy():
    s = np.random.default_rng(2).standard_normal((5, 120)) * 10
    assert _rel(O.softmax(s), scipy.special.softmax(s, axis=-1)) < 1e-13


def test_attention_matches_torch_sdpa():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((9, 4, 16))
    k = rng.standard_normal((23, 4, 16))
    v = rng.standard_normal((23, 4, 16))
    ref = F.scaled_dot_product_attention(torch.from_numpy(q).permute(1, 0, 2),
                                         torch.from_numpy(k).permute(1, 0, 2),
                                         torch.from_numpy(v).permute(1, 0, 2)).permute(1, 0, 2).numpy()
    assert _rel(O.attention(q, k, v), ref) < 1e-12


def test_attention_brute_force_loops():
    """Triple loop over queries, keys and dims in float64 (P5)."""
    rng = np.random.default_rng(4)
    R, N, H, D = 3, 11, 2, 5
    q, k, v = rng.standard_normal((R, H, D)), rng.standard_normal((N, H, D)), rng.standard_normal((N, H, D))
    out = np.zeros((R, H, D))
    for h in range(H):
        for r in range(R):
            s = [sum(q[r, h, d] * k[n, h, d] for d in range(D)) / math.sqrt(D) for n in range(N)]
            mx = max(s)
            w = [math.exp(x - mx) for x in s]
            z = sum(w)
            for d in range(D):
                out[r, h, d] = sum(w[n] * v[n, h, d] for n in range(N)) / z
    assert _rel(O.attention(q, k, v), out) < 1e-13


def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(5)
    _, p = O.attention(rng.standard_normal((6, 3, 8)) * 5, rng.standard_normal((40, 3, 8)) * 5,
                       rng.standard_normal((40, 3, 8)), return_probs=True)
    assert np.allclose(p.sum(-1), 1.0, atol=1e-14, rtol=0)


def test_dilate_matches_scipy():
    rng = np.random.default_rng(6)
    for shape in [(6, 5), (16, 16), (9, 13)]:
        m = rng.random(shape) < 0.08
        ref = scipy.ndimage.binary_dilation(m, structure=np.ones((3, 3), bool))
        assert np.array_equal(O.dilate(m, 1), ref)
        ref2 = scipy.ndimage.binary_dilation(m, structure=np.ones((5, 5), bool))
        assert np.array_equal(O.dilate(m, 2), ref2)


def test_compact_matches_flatnonzero():
    rng = np.random.default_rng(7)
    masks = (rng.random((3, 50)) < 0.3).astype(np.uint8)
    masks[1] = 0
    idx, off = O.compact(masks)
    assert off[0] == 0 and off[-1] == idx.size
    for b in range(3):
        assert np.array_equal(idx[off[b]:off[b + 1]], np.flatnonzero(masks[b]))


def test_patch_embed_matches_conv2d():
    """Token embedding without the position table == a stride-p convolution."""
    rng = np.random.default_rng(8)
    s = TINY
    W = {"pe_w": rng.standard_normal((s.hidden, 16)), "pe_b": rng.standard_normal(s.hidden)}
    lat = rng.standard_normal((4, s.grid_h * 2, s.grid_w * 2))
    x = O.patch_embed(W, lat, s.grid_h, s.grid_w, 2) - O.pos_embed_2d(s.grid_h, s.grid_w, s.hidden)
    ref = F.conv2d(torch.from_numpy(lat)[None], torch.from_numpy(W["pe_w"]).reshape(s.hidden, 4, 2, 2),
                   torch.from_numpy(W["pe_b"]), stride=2)[0]          # [C, gh, gw]
    ref = ref.permute(1, 2, 0).reshape(-1, s.hidden).numpy()           # tokens row-major
    assert _rel(x, ref) < 1e-13


def test_eps_layout_matches_unpatchify_einsum():
    """Output column (pi*p+qi)*c_out + c is pixel (pi, qi) of channel c."""
    rng = np.random.default_rng(9)
    gh, gw, p, co = 3, 4, 2, 8
    out = rng.standard_normal((gh * gw, p * p * co))
    img = torch.einsum("nhwpqc->nchpwq", torch.from_numpy(out).reshape(1, gh, gw, p, p, co))
    img = img.reshape(co, gh * p, gw * p).numpy()
    eps = O.eps_from_output(out, p, co, 4)                             # [N, 4, p, p]
    lat = O.patches_to_latent(eps, gh, gw)
    assert np.array_equal(lat, img[:4])


def test_patchify_inverse():
    rng = np.random.default_rng(10)
    lat = rng.standard_normal((4, 12, 10))
    assert np.array_equal(O.patches_to_latent(O.latent_to_patches(lat, 2), 6, 5), lat)


# --------------------------------------------------------------------------- closed forms

def test_timestep_sinusoid_closed_form():
    e0 = O.timestep_sinusoid(0.0)
    assert np.array_equal(e0, np.r_[np.ones(128), np.zeros(128)])
    t = 37.0
    e = O.timestep_sinusoid(t)
    assert abs(e[0] - math.cos(t)) < 1e-15 and abs(e[128] - math.sin(t)) < 1e-15
    f_last = 10000.0 ** (-127 / 128)
    assert abs(e[127] - math.cos(t * f_last)) < 1e-14


def test_pos_embed_structure():
    gh = gw = 7
    P = O.pos_embed_2d(gh, gw, 64)
    assert np.array_equal(P[0], np.r_[np.zeros(16), np.ones(16), np.zeros(16), np.ones(16)])
    # first half depends on the column only, second half on the row only;
    # token (y, x)'s column half equals token (x, y)'s row half
    for y in range(gh):
        for x in range(gw):
            assert np.array_equal(P[y * gw + x, :32], P[x, :32])
            assert np.array_equal(P[y * gw + x, 32:], P[y * gw, 32:])
            assert np.array_equal(P[y * gw + x, :32], P[x * gw + y, 32:])
    # non-square grids: row coordinate must not leak into the column half
    P2 = O.pos_embed_2d(3, 5, 64)
    assert np.array_equal(P2[5 * 2 + 1, :32], P2[1, :32])
    assert abs(P2[5 * 2 + 1, 32] - math.sin(2.0)) < 1e-15


def test_pos_embed_matches_library_routine():
    """The position table equals an independent library implementation of
    the 2-D sin-cos table (the OmDet-Turbo encoder's in transformers, float64):
    frequency ladder, sin/cos order and which half holds which coordinate.
    The library lists tokens column-major (x * gh + y); the oracle row-major
    (y * gw + x).  Non-square grids, so swapping the coordinates fails."""
    import torch
    from transformers.models.omdet_turbo.modeling_omdet_turbo import OmDetTurboHybridEncoder as Enc
    for gh, gw, C in ((5, 7, 64), (3, 11, 1152), (32, 32, 1152)):
        lib = Enc.build_2d_sincos_position_embedding(gw, gh, C, 10000.0, dtype=torch.float64)[0].numpy()
        P = O.pos_embed_2d(gh, gw, C)
        ys, xs = np.divmod(np.arange(gh * gw), gw)
        assert np.abs(P - lib[xs * gh + ys]).max() < 1e-12, (gh, gw, C)


def test_pos_embed_frequency_ladder():
    """Frequencies read back from the table (atan2 of the sin and cos columns
    at x = 1, unambiguous since every frequency is <= 1 < pi) form the
    geometric ladder from 1 down to 10^-4 * 10^(4/q) over q = C/4 columns."""
    C = 1152
    q = C // 4
    P = O.pos_embed_2d(2, 3, C)
    w = np.arctan2(P[1, :q], P[1, q:2 * q])  # token (y=0, x=1)
    assert abs(w[0] - 1.0) < 1e-14
    ratio = w[1:] / w[:-1]
    assert np.abs(ratio - ratio[0]).max() < 1e-12
    assert abs(w[-1] * 1e4 - 1e4 ** (1.0 / q)) < 1e-9
    # the row half carries the same ladder in y: token (y=1, x=0)
    wy = np.arctan2(P[3, C // 2:C // 2 + q], P[3, C // 2 + q:])
    assert np.abs(wy - w).max() < 1e-14


def test_alphas_cumprod_and_ddim_roundtrip():
    ac = O.alphas_cumprod()
    betas = np.linspace(1e-4, 0.02, 1000)
    assert abs(ac[0] - (1 - 1e-4)) < 1e-16
    assert abs(ac[-1] - math.exp(np.log1p(-betas).sum())) < 1e-15
    rng = np.random.default_rng(11)
    x0, eps = rng.standard_normal(50), rng.standard_normal(50)
    a, an = ac[700], ac[650]
    xt = math.sqrt(a) * x0 + math.sqrt(1 - a) * eps
    assert _rel(O.ddim_update(xt, eps, a, an), math.sqrt(an) * x0 + math.sqrt(1 - an) * eps) < 1e-13
    assert _rel(O.ddim_update(xt, eps, a, 1.0), x0) < 1e-12
    # zero noise prediction only rescales
    assert _rel(O.ddim_update(xt, 0 * eps, a, an), math.sqrt(an / a) * xt) < 1e-14


# --------------------------------------------------------------------------- block special cases

def _mod(C, rng, **over):
    names = ["sh1", "sc1", "g1", "sh2", "sc2", "g2"]
    m = {n: rng.standard_normal(C) * 0.3 for n in names}
    m.update(over)
    return tuple(m[n] for n in names)


def _tiny_block_inputs(seed=12):
    W = _tiny_weights(seed)
    lw = {k: v.astype(np.float64) for k, v in W["layers"][0].items()}
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((TINY.tokens, TINY.hidden))
    y = rng.standard_normal((TINY.text_len, TINY.hidden))
    tk, tv = O.text_kv(lw, y, TINY.heads)
    return lw, X, tk, tv, rng


def test_block_identity_when_branches_closed():
    lw, X, tk, tv, rng = _tiny_block_inputs()
    C = TINY.hidden
    lw["xproj_w"][:] = 0
    lw["xproj_b"][:] = 0
    mod = _mod(C, rng, g1=np.zeros(C), g2=np.zeros(C))
    out, _, _, _ = O.block_dense(lw, X, mod, tk, tv, TINY.heads)
    assert np.array_equal(out, X)


def test_block_self_attention_branch_closed_form():
    """scale_1 = -1 makes every normalised row equal shift_1, so all queries,
    keys and values coincide and attention returns that value row."""
    lw, X, tk, tv, rng = _tiny_block_inputs()
    C = TINY.hidden
    lw["xproj_w"][:] = 0
    lw["xproj_b"][:] = 0
    sh1, g1 = rng.standard_normal(C), rng.standard_normal(C)
    mod = _mod(C, rng, sh1=sh1, sc1=-np.ones(C), g1=g1, g2=np.zeros(C))
    out, K, V, _ = O.block_dense(lw, X, mod, tk, tv, TINY.heads)
    v_row = lw["qkv_w"][2 * C:] @ sh1 + lw["qkv_b"][2 * C:]
    expect = X + g1 * (lw["proj_w"] @ v_row + lw["proj_b"])
    assert _rel(out, expect) < 1e-12
    k_row = lw["qkv_w"][C:2 * C] @ sh1 + lw["qkv_b"][C:2 * C]
    assert _rel(K.transpose(1, 0, 2).reshape(TINY.tokens, C), np.tile(k_row, (TINY.tokens, 1))) < 1e-12


def test_block_cross_attention_branch_closed_form_and_maps():
    """Zero query projection -> uniform cross-attention: the branch adds
    mean(V_text) W_xp^T + b_xp and every delta map entry is heads/M."""
    lw, X, tk, tv, rng = _tiny_block_inputs()
    C = TINY.hidden
    lw["xq_w"][:] = 0
    lw["xq_b"][:] = 0
    mod = _mod(C, rng, g1=np.zeros(C), g2=np.zeros(C))
    delta = np.array([1, 5])
    out, _, _, maps = O.block_dense(lw, X, mod, tk, tv, TINY.heads, delta=delta)
    expect = X + lw["xproj_w"] @ tv.reshape(TINY.text_len, C).mean(0) + lw["xproj_b"]
    assert _rel(out, expect) < 1e-12
    assert np.allclose(maps, TINY.heads / TINY.text_len, atol=1e-15, rtol=0)


def test_maps_sum_over_all_columns_is_heads():
    lw, X, tk, tv, rng = _tiny_block_inputs()
    mod = _mod(TINY.hidden, rng)
    _, _, _, maps = O.block_dense(lw, X, mod, tk, tv, TINY.heads, delta=np.arange(TINY.text_len))
    assert np.allclose(maps.sum(1), TINY.heads, atol=1e-12, rtol=0)
    assert maps.min() >= 0 and maps.max() <= TINY.heads


def test_block_mlp_branch_closed_form():
    """scale_2 = -1 with the other branches closed: X + g2 (gelu(sh2 W1^T + b1) W2^T + b2)."""
    lw, X, tk, tv, rng = _tiny_block_inputs()
    C = TINY.hidden
    lw["xproj_w"][:] = 0
    lw["xproj_b"][:] = 0
    sh2, g2 = rng.standard_normal(C), rng.standard_normal(C)
    mod = _mod(C, rng, g1=np.zeros(C), sh2=sh2, sc2=-np.ones(C), g2=g2)
    out, _, _, _ = O.block_dense(lw, X, mod, tk, tv, TINY.heads)
    hid = lw["fc1_w"] @ sh2 + lw["fc1_b"]
    hid = 0.5 * hid * (1 + np.tanh(math.sqrt(2 / math.pi) * (hid + 0.044715 * hid ** 3)))
    expect = X + g2 * (lw["fc2_w"] @ hid + lw["fc2_b"])
    assert _rel(out, expect) < 1e-12


def test_layer_modulation_order():
    """Rows of the per-block table map to (shift1, scale1, gate1, shift2, scale2, gate2)."""
    C = 8
    lw = {"sst": np.arange(6 * C, dtype=np.float64).reshape(6, C)}
    t0 = np.zeros((6, C))
    mod = O.layer_modulation(lw, t0)
    for i in range(6):
        assert np.array_equal(mod[i], np.arange(i * C, (i + 1) * C))


# --------------------------------------------------------------------------- method invariants

def _tiny_step_inputs(seed=20):
    s = TINY
    W = _tiny_weights(seed)
    rng = np.random.default_rng(seed)
    lat = rng.standard_normal((4, s.grid_h * 2, s.grid_w * 2))
    txt = rng.standard_normal((s.text_len, s.text_dim))
    y = O.caption_projection(W, txt)
    tkv = [O.text_kv(lw, y, s.heads) for lw in W["layers"]]
    cache = dict(K=rng.standard_normal((s.layers, s.heads, s.tokens, s.head_dim)),
                 V=rng.standard_normal((s.layers, s.heads, s.tokens, s.head_dim)),
                 H=rng.standard_normal((s.layers, s.tokens, s.hidden)))
    lat_next_cached = rng.standard_normal(lat.shape)
    return W, lat, tkv, cache, lat_next_cached, rng


def test_all_active_equals_dense():
    """P1: with every token active, the reuse step is the dense step, whatever
    the cache held."""
    s = TINY
    W, lat, tkv, cache, lnc, _ = _tiny_step_inputs()
    delta = np.array([0, 3, 7])
    d = O.dense_step(s, W, lat, 600, 550, tkv, delta)
    r = O.reuse_step(s, W, lat, 600, 550, tkv, np.arange(s.tokens), cache, lnc, delta)
    for k in ("K", "V", "H", "latent_next", "maps"):
        assert _rel(r[k], d[k]) < 1e-12, k


def test_empty_mask_returns_cache():
    """P2: with no active token the slot is unchanged and the latent is the
    cached trajectory's."""
    s = TINY
    W, lat, tkv, cache, lnc, _ = _tiny_step_inputs()
    r = O.reuse_step(s, W, lat, 600, 550, tkv, np.zeros(0, np.int64), cache, lnc)
    for k in ("K", "V", "H"):
        assert np.array_equal(r[k], cache[k])
    assert np.array_equal(r["latent_next"], lnc)


def test_cache_consistency_any_mask():
    """P3: when the cache was built by a dense step on the same input, a reuse
    step over any active set reproduces the dense step."""
    s = TINY
    W, lat, tkv, _, _, rng = _tiny_step_inputs()
    d = O.dense_step(s, W, lat, 400, 350, tkv)
    cache = dict(K=d["K"], V=d["V"], H=d["H"])
    for trial in range(4):
        idx = np.flatnonzero(rng.random(s.tokens) < [0.1, 0.3, 0.6, 0.9][trial])
        r = O.reuse_step(s, W, lat, 400, 350, tkv, idx, cache, d["latent_next"])
        for k in ("K", "V", "H", "latent_next"):
            assert _rel(r[k], d[k]) < 1e-12, (trial, k)


def test_locality_and_poison():
    """P4: stale cached K/V/H of active rows (NaN) never reach an output;
    inactive rows of K/V/H and inactive latent patches are the cache's,
    bit for bit; cached H of inactive rows is never read."""
    s = TINY
    W, lat, tkv, cache, lnc, rng = _tiny_step_inputs()
    idx = np.array([1, 2, 7, 8, 12, 29])
    act = np.zeros(s.tokens, bool)
    act[idx] = True
    pois = {k: v.copy() for k, v in cache.items()}
    pois["K"][:, :, idx] = np.nan
    pois["V"][:, :, idx] = np.nan
    pois["H"][:, idx] = np.nan
    r = O.reuse_step(s, W, lat, 500, 450, tkv, idx, pois, lnc, np.array([2]))
    for k in ("K", "V", "H", "latent_next", "maps", "X"):
        assert np.all(np.isfinite(r[k])), k
    assert np.array_equal(r["K"][:, :, ~act], cache["K"][:, :, ~act])
    assert np.array_equal(r["H"][:, ~act], cache["H"][:, ~act])
    assert np.all(r["maps"][~act] == 0)
    lp = O.latent_to_patches(r["latent_next"], 2)
    assert np.array_equal(lp[~act], O.latent_to_patches(lnc, 2)[~act])
    # changing the cached hidden state of inactive rows changes no active output
    alt = {k: v.copy() for k, v in cache.items()}
    alt["H"][:, ~act] += 5.0
    r2 = O.reuse_step(s, W, lat, 500, 450, tkv, idx, alt, lnc)
    assert np.array_equal(r2["X"], O.reuse_step(s, W, lat, 500, 450, tkv, idx, cache, lnc)["X"])


def test_gathered_rows_equal_dense_attention_over_merged_kv():
    """P5 on a block: a reuse block's active outputs equal a dense block run on
    inputs whose inactive rows are chosen so that their K/V are the cached ones
    -- checked here by feeding the dense block the merged K/V directly through
    brute force attention."""
    lw, X, tk, tv, rng = _tiny_block_inputs(30)
    C, Hh, D = TINY.hidden, TINY.heads, TINY.head_dim
    mod = _mod(C, rng)
    idx = np.array([0, 4, 5, 17])
    cK = rng.standard_normal((Hh, TINY.tokens, D))
    cV = rng.standard_normal((Hh, TINY.tokens, D))
    cH = rng.standard_normal((TINY.tokens, C))
    out, K, V, Hm, _ = O.block_reuse(lw, X[idx], idx, mod, tk, tv, cK, cV, cH, Hh)
    # recompute the attention branch by brute force over the merged K/V
    h = O.modulate(O.layer_norm(X[idx]), mod[0], mod[1])
    qkv = (h @ lw["qkv_w"].T + lw["qkv_b"]).reshape(len(idx), 3, Hh, D)
    o = np.zeros((len(idx), Hh, D))
    for r in range(len(idx)):
        for hh in range(Hh):
            s = np.array([qkv[r, 0, hh] @ K[hh, n] for n in range(TINY.tokens)]) / math.sqrt(D)
            w = np.exp(s - s.max())
            o[r, hh] = (w[:, None] * V[hh]).sum(0) / w.sum()
    # merged K/V: fresh at idx, cached elsewhere
    assert np.array_equal(np.delete(K, idx, axis=1), np.delete(cK, idx, axis=1))
    assert _rel(K[:, idx].transpose(1, 0, 2), qkv[:, 1]) < 1e-14
    x1 = X[idx] + mod[2] * (o.reshape(len(idx), C) @ lw["proj_w"].T + lw["proj_b"])
    x_ref, _ = O.cross_and_mlp(lw, x1, mod, tk, tv, Hh, None, np.float64)
    assert _rel(out, x_ref) < 1e-12
    assert np.array_equal(Hm[idx], out)


def test_fp32_oracle_agrees_with_fp64():
    """P10: the same step in float32 and float64 agree to 1e-5 normwise."""
    s = TINY
    W = synth.make_weights(s, seed=3, std=0.05)
    rng = np.random.default_rng(3)
    lat = rng.standard_normal((4, s.grid_h * 2, s.grid_w * 2))
    txt = rng.standard_normal((s.text_len, s.text_dim))
    outs = {}
    for dt in (np.float32, np.float64):
        y = O.caption_projection(W, txt, dt)
        tkv = [O.text_kv(lw, y, s.heads, dt) for lw in W["layers"]]
        outs[dt] = O.dense_step(s, W, lat, 700, 650, tkv, dt=dt)
    for k in ("H", "K", "latent_next"):
        assert _rel(outs[np.float32][k], outs[np.float64][k]) < 1e-5


def test_token_mode_reuse_all_active_equals_dense():
    s = synth.ModelShape(hidden=64, heads=4, head_dim=16, mlp=128, layers=1, text_len=8,
                         text_dim=64, grid_h=4, grid_w=6, dtype="f32", token_mode=True)
    W = synth.make_weights(s, seed=5, std=0.2, stress=True)
    rng = np.random.default_rng(5)
    X = rng.standard_normal((s.tokens, s.hidden))
    txt = rng.standard_normal((s.text_len, s.hidden))
    tv = rng.standard_normal(s.hidden)
    d = O.dense_block_tokens(s, W, X, tv, txt, delta=np.array([2]))
    cK, cV = rng.standard_normal((2, s.heads, s.tokens, s.head_dim))
    cH = rng.standard_normal((s.tokens, s.hidden))
    r = O.reuse_block_tokens(s, W, X, np.arange(s.tokens), tv, txt, cK, cV, cH, delta=np.array([2]))
    assert _rel(r[0], d[0]) < 1e-12 and _rel(r[1], d[1]) < 1e-12 and _rel(r[4], d[3]) < 1e-12


# --------------------------------------------------------------------------- localisation

def test_localize_planted_region():
    """P7: boosted delta columns over a blob are recovered exactly: the
    pre-dilation mask is the blob and the output is its 3x3 dilation."""
    gh = gw = 24
    Z, delta, blob = synth.make_logits(2, 4, gh * gw, 120, gh, gw, n_delta=3, seed=0, frac=0.1)
    maps = O.maps_from_logits(Z, delta)
    mask, idx, scores = O.localize(maps, gh, gw, n_avg=8, return_scores=True)
    pre = (scores >= 0.3).any(1)
    assert np.array_equal(pre, blob.astype(bool))
    ref = scipy.ndimage.binary_dilation(blob.reshape(gh, gw).astype(bool), np.ones((3, 3), bool))
    assert np.array_equal(mask.astype(bool), ref.reshape(-1))
    assert np.array_equal(idx, np.flatnonzero(ref))
    # no score inside the 1e-3 band around the threshold
    assert np.min(np.abs(scores - 0.3)) > 1e-3


def test_maps_from_logits_is_mean_softmax():
    rng = np.random.default_rng(13)
    Z = rng.standard_normal((3, 2, 5, 7))
    delta = np.array([0, 6])
    ref = scipy.special.softmax(Z, axis=-1)[..., delta].sum(axis=(0, 1))
    assert _rel(O.maps_from_logits(Z, delta), ref) < 1e-13


def test_localize_scale_invariance_and_degenerate():
    """P9: positive affine changes of the maps leave the region unchanged; a
    constant map selects nothing."""
    gh, gw = 10, 12
    maps, blob = synth.planted_maps(gh * gw, 4, gh, gw, seed=3)
    m1, i1 = O.localize(maps, gh, gw)
    m2, i2 = O.localize(maps * 7.5 + 3.0, gh, gw, n_avg=2.0)
    assert np.array_equal(m1, m2) and np.array_equal(i1, i2)
    const = np.ones((gh * gw, 2))
    m3, i3 = O.localize(const, gh, gw)
    assert m3.sum() == 0 and i3.size == 0


def test_localize_threshold_inclusive():
    """Sec. 3.2 includes tokens whose response equals the threshold."""
    maps = np.zeros((9, 1))
    maps[4, 0] = 1.0
    maps[0, 0] = 0.3          # normalised score exactly 0.3
    mask, _ = O.localize(maps, 3, 3, radius=0)
    assert mask[0] == 1 and mask[4] == 1 and mask.sum() == 2


# --------------------------------------------------------------------------- schedule (paper values)

def test_reuse_cutoff_golden():
    g = json.load(open(os.path.join(GOLDEN, "reuse_cutoff.json")))
    for c in g["cases"]:
        s = 0.9 if c["similar"] else 0.1
        assert O.reuse_cutoff(c["T"], s, tau_s=0.5, rho=g["rho"]) == c["T_reuse"]


def test_step_plans():
    assert O.step_plan(20) == ["dense"] * 4 + ["reuse"] * 16
    assert O.step_plan(20, reading="paper", s=0.1, tau_s=0.8) == ["copy"] * 4 + ["reuse"] * 16
    assert O.step_plan(20, reading="paper", s=0.95, tau_s=0.8) == ["copy"] * 20


def test_cosine_similarity():
    assert abs(O.cosine_similarity([1, 0], [0, 1])) < 1e-15
    assert abs(O.cosine_similarity([1, 2, 3], [2, 4, 6]) - 1) < 1e-15
    assert abs(O.cosine_similarity([1, 0], [1, 1]) - math.sqrt(0.5)) < 1e-15


# --------------------------------------------------------------------------- projections against torch.nn modules

def _linear(w, b):
    m = torch.nn.Linear(w.shape[1], w.shape[0], dtype=torch.float64)
    with torch.no_grad():
        m.weight.copy_(torch.from_numpy(np.asarray(w, np.float64)))
        m.bias.copy_(torch.from_numpy(np.asarray(b, np.float64)))
    return m


def test_caption_projection_matches_torch_mlp():
    W = _tiny_weights(40)
    txt = np.random.default_rng(40).standard_normal((TINY.text_len, TINY.text_dim))
    mlp = torch.nn.Sequential(_linear(W["cap_w1"], W["cap_b1"]), torch.nn.GELU(approximate="tanh"),
                              _linear(W["cap_w2"], W["cap_b2"]))
    ref = mlp(torch.from_numpy(txt)).detach().numpy()
    assert _rel(O.caption_projection(W, txt), ref) < 1e-13


def test_timestep_embedding_and_adaln_match_torch():
    W = _tiny_weights(41)
    t = 613.0
    e = torch.from_numpy(O.timestep_sinusoid(t))
    mlp = torch.nn.Sequential(_linear(W["temb_w1"], W["temb_b1"]), torch.nn.SiLU(), _linear(W["temb_w2"], W["temb_b2"]))
    temb_ref = mlp(e).detach().numpy()
    temb = O.timestep_embedding(W, t)
    assert _rel(temb, temb_ref) < 1e-13
    blk = torch.nn.Sequential(torch.nn.SiLU(), _linear(W["tblock_w"], W["tblock_b"]))
    t0_ref = blk(torch.from_numpy(temb_ref)).detach().numpy().reshape(6, -1)
    assert _rel(O.adaln_single(W, temb), t0_ref) < 1e-13


def test_text_kv_matches_torch_linear():
    W = _tiny_weights(42)
    lw = W["layers"][1]
    y = np.random.default_rng(42).standard_normal((TINY.text_len, TINY.hidden))
    kv = _linear(lw["xkv_w"], lw["xkv_b"])(torch.from_numpy(y)).detach()
    k_ref, v_ref = kv.view(TINY.text_len, 2, TINY.heads, TINY.head_dim).unbind(1)
    k, v = O.text_kv(lw, y, TINY.heads)
    assert _rel(k, k_ref.numpy()) < 1e-13 and _rel(v, v_ref.numpy()) < 1e-13


def test_final_layer_matches_torch():
    W = _tiny_weights(43)
    rng = np.random.default_rng(43)
    X = rng.standard_normal((7, TINY.hidden)) * 2 + 0.5
    temb = rng.standard_normal(TINY.hidden)
    ln = torch.nn.LayerNorm(TINY.hidden, eps=1e-6, elementwise_affine=False, dtype=torch.float64)
    sh = torch.from_numpy(W["fin_sst"][0].astype(np.float64) + temb)
    sc = torch.from_numpy(W["fin_sst"][1].astype(np.float64) + temb)
    h = ln(torch.from_numpy(X)) * (1 + sc) + sh
    ref = _linear(W["fin_w"], W["fin_b"])(h).detach().numpy()
    assert _rel(O.final_layer(W, X, temb), ref) < 1e-13


def test_guided_latent_special_cases():
    """Classifier-free guidance: scale 1 is the conditional step and scale 0
    the unconditional step (each the oracle's own unguided reuse step);
    the guided noise is affine in the scale."""
    s = TINY
    W, lat, tkv_c, cache, lnc, rng = _tiny_step_inputs(31)
    y_u = O.caption_projection(W, np.zeros((s.text_len, s.text_dim)))
    tkv_u = [O.text_kv(lw, y_u, s.heads) for lw in W["layers"]]
    idx = np.flatnonzero(rng.random(s.tokens) < 0.4)
    rc = O.reuse_step(s, W, lat, 500, 450, tkv_c, idx, cache, lnc)
    ru = O.reuse_step(s, W, lat, 500, 450, tkv_u, idx, cache, lnc)
    g1 = O.guided_latent(s, lat, lnc, idx, rc["eps"], ru["eps"], 1.0, 500, 450)
    g0 = O.guided_latent(s, lat, lnc, idx, rc["eps"], ru["eps"], 0.0, 500, 450)
    assert _rel(g1, rc["latent_next"]) < 1e-12 and _rel(g0, ru["latent_next"]) < 1e-12
    e2 = O.guided_noise(rc["eps"], ru["eps"], 2.0)
    assert _rel(e2, 2.0 * rc["eps"] - ru["eps"]) < 1e-12
    # the dense step's noise prediction plugs in the same way
    dc = O.dense_step(s, W, lat, 500, 450, tkv_c)
    assert _rel(O.guided_latent(s, lat, lnc, np.arange(s.tokens), dc["eps"], dc["eps"], 4.5, 500, 450),
                dc["latent_next"]) < 1e-12
