"""Multi-turn editing driver (Sec. 3.2, Sec. 3.3, Eq. 1, Eq. 2).

CPU: the host schedule arithmetic against the oracle's (which is pinned to
the paper's printed cutoff in test_oracle_pins).  GPU: two-turn runs of the
driver and the invariants the method fixes -- the first turn against the
oracle's chained dense steps, patches outside the edited region carried over
bit for bit, the cache of unchanged tokens untouched, and a fully reused turn
reproducing the previous one."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2608_29809_amd import schedule as S
from tests._cases import download_slot, oracle_text_kv, relerr, to_np


def test_timestep_grid_matches_inputs_and_oracle_reading():
    for T in (1, 2, 5, 20, 50):
        assert np.array_equal(S.timestep_grid(T), synth.timestep_grid(T))
    assert list(S.timestep_grid(20)[:3]) == [999, 946, 894] and S.timestep_grid(20)[-1] == 0


def test_similarity_and_cutoff_match_oracle():
    rng = np.random.default_rng(0)
    for _ in range(20):
        a, b = rng.standard_normal(64), rng.standard_normal(64)
        assert abs(S.prompt_similarity(a, b) - O.cosine_similarity(a, b)) < 1e-12
    assert abs(S.prompt_similarity(a, 3 * a) - 1.0) < 1e-12
    for T in (10, 20, 25, 50):
        for s in (-1.0, 0.0, 0.5, 0.79, 0.8, 0.81, 1.0):
            for tau in (0.5, 0.8):
                assert S.reuse_cutoff(T, s, tau) == O.reuse_cutoff(T, s, tau)


def test_step_plans_match_oracle():
    for T in (5, 20, 25):
        assert S.step_plan(T) == O.step_plan(T)
        for s in (0.1, 0.9):
            assert S.step_plan(T, reading="paper", s=s) == O.step_plan(T, reading="paper", s=s)
    assert S.step_plan(20)[:5] == ["dense"] * 4 + ["reuse"]
    with pytest.raises(ValueError):
        S.step_plan(20, reading="other")


def _setup(T=5, B=2, seed=11):
    from paper_2608_29809_amd.runtime import RegionCacheModel
    s = synth.ModelShape(layers=2, grid_h=16, grid_w=16, dtype="bf16")
    W = synth.make_weights(s, seed=seed, stress=True)
    model = RegionCacheModel(s, W)
    txt0 = synth.make_text(s, B, seed)
    txt1, delta = synth.edit_text(s, txt0, 3, seed + 1)
    delta = [int(d) for d in delta]
    x_T = synth.make_latent(s, B, seed)
    return s, W, model, txt0, txt1, delta, x_T


@pytest.mark.gpu
@pytest.mark.timeout(300)
def test_first_turn_vs_oracle_and_edit_turn_invariants():
    s, W, model, txt0, txt1, delta, x_T = _setup()
    T, B = 5, 2
    sess = S.EditSession(model, B, T=T)
    xT = torch.from_numpy(x_T).cuda()
    x0 = sess.first_turn(model.to_storage(txt0), xT)
    torch.cuda.synchronize()
    # the first turn: T chained dense steps of the oracle
    tg = S.timestep_grid(T)
    for b in range(B):
        tkv = oracle_text_kv(s, W, txt0[b])
        x = x_T[b]
        for k in range(T):
            x = O.dense_step(s, W, x, int(tg[k]), int(tg[k + 1]) if k + 1 < T else -1, tkv)["latent_next"]
        e = relerr(to_np(x0)[b], x)
        print(f"first turn chain {b}: latent {e:.2e}", flush=True)
        assert e < 3e-2
    slots0 = [download_slot(sess.cache, k, s.layers, B) for k in range(T)]
    # second turn, dense-then-reuse: 1 dense step emitting maps, localisation, 4 reuse steps
    out = sess.edit_turn(model.to_storage(txt1), xT, delta)
    torch.cuda.synchronize()
    assert out["plan"] == ["dense"] + ["reuse"] * 4
    act, mask = out["active"], to_np(out["mask"]).astype(bool)
    assert act.total == int(mask.sum())
    x1 = to_np(out["latent"])
    gh, gw = s.grid_h, s.grid_w
    for b in range(B):
        inact = ~mask[b].reshape(gh, gw)
        pix = np.repeat(np.repeat(inact, 2, axis=0), 2, axis=1)  # 2x2 latent patch per token
        # patches outside the region end where the previous turn ended
        assert np.array_equal(x1[b][:, pix], to_np(x0)[b][:, pix]), b
        # the cache of tokens outside the region is untouched in the reuse steps
        tok = np.flatnonzero(~mask[b])
        for k in range(1, T):
            got = download_slot(sess.cache, k, s.layers, B)
            for key in ("K", "V", "H"):
                ax = 2 if key != "H" else 1
                assert np.array_equal(np.take(got[key][:, b], tok, axis=ax),
                                      np.take(slots0[k][key][:, b], tok, axis=ax)), (b, k, key)


@pytest.mark.gpu
@pytest.mark.timeout(300)
def test_paper_plan_copy_and_region_reuse():
    s, W, model, txt0, txt1, delta, x_T = _setup(seed=12)
    T, B = 5, 2
    sess = S.EditSession(model, B, T=T, reading="paper", tau_s=0.8)
    xT = torch.from_numpy(x_T).cuda()
    x0 = sess.first_turn(model.to_storage(txt0), xT)
    torch.cuda.synchronize()
    before = sess.cache.buf.clone()
    # a consistent edit (s >= tau_s): the region reuses the cache for all T
    # steps, so the turn reproduces the previous one and leaves the pool as is
    out = sess.edit_turn(model.to_storage(txt1), xT, delta, similarity=0.95)
    torch.cuda.synchronize()
    assert out["plan"] == ["copy"] * T
    assert torch.equal(out["latent"], x0)
    assert torch.equal(sess.cache.buf, before)
    # a semantic change (s < tau_s): copy for floor(0.2 T) = 1 step, then the
    # given region is recomputed; patches outside it end as before
    from paper_2608_29809_amd.runtime import ActiveSet
    region = [np.arange(40, 90), np.arange(0, 32)]
    out = sess.edit_turn(model.to_storage(txt1), xT, delta, similarity=0.2, region=ActiveSet.from_lists(region))
    torch.cuda.synchronize()
    assert out["plan"] == ["copy"] + ["reuse"] * 4
    x1 = to_np(out["latent"])
    for b in range(B):
        inact = np.ones(s.tokens, bool)
        inact[region[b]] = False
        pix = np.repeat(np.repeat(inact.reshape(s.grid_h, s.grid_w), 2, axis=0), 2, axis=1)
        assert np.array_equal(x1[b][:, pix], to_np(x0)[b][:, pix])
        assert not np.array_equal(x1[b][:, ~pix], to_np(x0)[b][:, ~pix])
    with pytest.raises(ValueError):
        sess.edit_turn(model.to_storage(txt1), xT, delta, similarity=0.2)


@pytest.mark.gpu
@pytest.mark.timeout(300)
def test_guided_session_pairs_stay_in_step():
    """With guidance the two branches of an image share latents and region:
    both chains of each pair end every turn with identical latents, and the
    localised region of the conditional branch is used for both."""
    s, W, model, txt0, txt1, delta, x_T = _setup(seed=13, B=2)
    txt0[1] = 0.0
    txt1[1] = 0.0
    x_T[1] = x_T[0]
    sess = S.EditSession(model, 2, T=5, guidance=4.5)
    xT = torch.from_numpy(x_T).cuda()
    x0 = sess.first_turn(model.to_storage(txt0), xT)
    out = sess.edit_turn(model.to_storage(txt1), xT, delta)
    torch.cuda.synchronize()
    assert torch.equal(x0[0], x0[1])
    assert torch.equal(out["latent"][0], out["latent"][1])
    m = to_np(out["mask"])
    assert np.array_equal(m[0], m[1])
    assert out["active"].counts[0] == out["active"].counts[1] == int(m[0].sum())

