"""Multi-turn editing driver (Sec. 3.2, Sec. 3.3, Eq. 1, Eq. 2).

CPU: the host schedule arithmetic against the oracle's (which is pinned to
the paper's printed cutoff in test_oracle_pins) and Eq. 1 on the prompt
features.  GPU: whole turns of the driver -- dense steps emitting the delta
maps, in-pipeline localisation, region-reuse and copy steps -- compared
step by step with the oracle run of the same plan, each step fed the GPU's
own inputs (re-synchronised) and gated at 2e-2; the free-running drift over
turns is reported; a five-turn chain."""
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


def test_delta_similarity_is_eq1_on_the_delta_rows():
    """Eq. 1 from the prompt features: the cosine of the delta rows before
    and after the edit, per chain (host arithmetic on a few rows)."""
    rng = np.random.default_rng(3)
    a = torch.from_numpy(rng.standard_normal((2, 10, 16)).astype(np.float32))
    b = a.clone()
    b[1, [2, 7]] = torch.from_numpy(rng.standard_normal((2, 16)).astype(np.float32))
    sims = S.delta_similarity(a, b, [2, 7])
    assert abs(sims[0] - 1.0) < 1e-12
    ref = O.cosine_similarity(a[1, [2, 7]].numpy(), b[1, [2, 7]].numpy())
    assert abs(sims[1] - ref) < 1e-12


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


# With random-init weights the delta-token maps are noise, and the range
# threshold 0.3 plus the one-token dilation selects (nearly) the whole 16 x 16
# grid; the session tests use a stricter threshold so that the regions are
# partial (46-80 of 256 tokens at these seeds) and the region-reuse steps
# have inactive tokens.  The 0.3 rule itself is tested on planted regions in
# test_parity_gpu.py.
LOC_THRESHOLD = 0.9


def _snapshot(sess, s, B):
    """The pool after a turn: every step's slot and the latent trajectory."""
    slots = [download_slot(sess.cache, k, s.layers, B) for k in range(sess.T)]
    traj = np.stack([np.stack([to_np(sess.cache.latent(b, k)) for k in range(sess.T + 1)]) for b in range(B)])
    return slots, traj


def _excused(scores, theta, gh, gw, band=1e-3):
    near = (np.abs(scores - theta) < band).any(axis=1)
    return O.dilate(near.reshape(gh, gw), 1).reshape(-1)


def _check_turn(s, W, txt, x_T, plans, before, after, lists, delta=None, maps=None, mask=None, tol=2e-2):
    """Per-step parity of one turn with re-synchronised inputs: step k of
    the oracle takes the GPU's own latent entering the step (trajectory
    entry k of this turn; x_T for step 0) and, for a region-reuse step, the
    slot and next latent the previous turn left, and follows the chain's
    plan.  Dense steps: every token's keys, values and hidden states and the
    latent within tol; the emitting step's maps within tol and the
    localised mask equal to the oracle's localisation of the same maps
    (tokens within 1e-3 of the threshold excused), the index list then
    bit-exact.  Region steps: the active rows within tol, everything else
    the previous turn's bit for bit.  Copy steps: the previous turn's slot
    and latent bit for bit.  Returns the worst error over the turn."""
    T = len(plans[0])
    tg = S.timestep_grid(T)
    slots0, traj0 = before
    slots1, traj1 = after
    worst = 0.0
    for b, plan in enumerate(plans):
        tkv = oracle_text_kv(s, W, txt[b])
        for k, what in enumerate(plan):
            t, tn = int(tg[k]), (int(tg[k + 1]) if k + 1 < T else -1)
            x_in = x_T[b] if k == 0 else traj1[b][k]
            got = {key: slots1[k][key][:, b] for key in ("K", "V", "H")}
            old = {key: slots0[k][key][:, b] for key in ("K", "V", "H")}
            if what == "dense":
                emit = maps is not None and k == plan.count("dense") - 1
                r = O.dense_step(s, W, x_in, t, tn, tkv, np.array(delta) if emit else None)
                errs = [relerr(got[key], r[key]) for key in ("K", "V", "H")] + [relerr(traj1[b][k + 1], r["latent_next"])]
                if emit:
                    errs.append(relerr(maps[b], r["maps"]))
                    m_ref, i_ref, sc = O.localize(maps[b], s.grid_h, s.grid_w, theta=LOC_THRESHOLD, return_scores=True)
                    exc = _excused(sc, LOC_THRESHOLD, s.grid_h, s.grid_w)
                    assert ((mask[b] == m_ref) | exc).all(), (b, k)
                    if not exc.any():
                        assert np.array_equal(lists[b], i_ref), (b, k)
            elif what == "reuse":
                idx = np.asarray(lists[b])
                r = O.reuse_step(s, W, x_in, t, tn, tkv, idx, old, traj0[b][k + 1])
                inact = np.setdiff1d(np.arange(s.tokens), idx)
                for key in ("K", "V"):
                    assert np.array_equal(got[key][:, :, inact], old[key][:, :, inact]), (b, k, key)
                assert np.array_equal(got["H"][:, inact], old["H"][:, inact]), (b, k)
                errs = [relerr(got["K"][:, :, idx], r["K"][:, :, idx]), relerr(got["V"][:, :, idx], r["V"][:, :, idx]),
                        relerr(got["H"][:, idx], r["H"][:, idx]), relerr(traj1[b][k + 1], r["latent_next"])]
            else:  # copy: the region keeps the cached states
                for key in ("K", "V", "H"):
                    assert np.array_equal(got[key], old[key]), (b, k, key)
                assert np.array_equal(traj1[b][k + 1], traj0[b][k + 1]), (b, k)
                errs = [0.0]
            e = max(errs)
            print(f"chain {b} step {k} {what}: {e:.2e}", flush=True)
            assert e < tol, (b, k, what, errs)
            worst = max(worst, e)
    return worst


def _free_running(s, W, txts, x_T, T, plans_per_turn, regions_per_turn, b):
    """The oracle's own run of the same turns (its own cache, no
    re-synchronisation): the final latent of the last turn."""
    tg = S.timestep_grid(T)
    cache = None
    x = None
    for turn, txt in enumerate(txts):
        tkv = oracle_text_kv(s, W, txt[b])
        plan = plans_per_turn[turn][b]
        new_cache, x, traj = [], x_T[b], [x_T[b]]
        for k, what in enumerate(plan):
            t, tn = int(tg[k]), (int(tg[k + 1]) if k + 1 < T else -1)
            if what == "dense":
                r = O.dense_step(s, W, x, t, tn, tkv)
                new_cache.append(dict(K=r["K"], V=r["V"], H=r["H"]))
                x = r["latent_next"]
            elif what == "reuse":
                r = O.reuse_step(s, W, x, t, tn, tkv, regions_per_turn[turn][b], cache[0][k], cache[1][k + 1])
                new_cache.append(dict(K=r["K"], V=r["V"], H=r["H"]))
                x = r["latent_next"]
            else:
                new_cache.append(cache[0][k])
                x = cache[1][k + 1]
            traj.append(x)
        cache = (new_cache, traj)
    return x


@pytest.mark.gpu
@pytest.mark.timeout(300)
def test_first_and_edit_turn_stepwise_vs_oracle():
    """dense_then_reuse: a first turn of T dense steps, then an edit turn
    (1 dense step emitting the delta maps, localisation, 4 region-reuse
    steps), every step against the oracle with re-synchronised inputs at
    2e-2; the free-running drift of the whole edit turn is reported."""
    s, W, model, txt0, txt1, delta, x_T = _setup()
    T, B = 5, 2
    sess = S.EditSession(model, B, T=T, threshold=LOC_THRESHOLD)
    xT = torch.from_numpy(x_T).cuda()
    empty = _snapshot_empty(s, B, T)
    sess.first_turn(model.to_storage(txt0), xT)
    torch.cuda.synchronize()
    snap0 = _snapshot(sess, s, B)
    w0 = _check_turn(s, W, txt0, x_T, [["dense"] * T] * B, empty, snap0, None)
    print(f"first turn, worst per-step error {w0:.2e}", flush=True)
    # the edit turn; its maps are read back from the emitting dense step
    maps_box = {}
    orig_localize = model.localize

    def spy(maps, *a, **k):
        maps_box["maps"] = to_np(maps)
        return orig_localize(maps, *a, **k)

    model.localize = spy
    out = sess.edit_turn(model.to_storage(txt1), xT, delta)
    model.localize = orig_localize
    torch.cuda.synchronize()
    assert out["plan"] == ["dense"] + ["reuse"] * 4
    mask = to_np(out["mask"]).astype(np.uint8)
    act = out["active"]
    lists = [to_np(act.idx[act.host[b]:act.host[b + 1]]).astype(np.int64) for b in range(B)]
    for b in range(B):
        assert np.array_equal(lists[b], np.flatnonzero(mask[b]))
        assert 0 < lists[b].size < s.tokens
    snap1 = _snapshot(sess, s, B)
    w1 = _check_turn(s, W, txt1, x_T, out["plans"], snap0, snap1, lists, delta, maps_box["maps"], mask)
    print(f"edit turn, worst per-step error {w1:.2e}", flush=True)
    for b in range(B):
        x_free = _free_running(s, W, [txt0, txt1], x_T, T, [[["dense"] * T] * B, out["plans"]], [None, lists], b)
        print(f"chain {b}: free-running drift of the final latent after two turns "
              f"{relerr(snap1[1][b][T], x_free):.2e}", flush=True)


def _snapshot_empty(s, B, T):
    """Stand-in 'previous turn' for the first turn (dense steps read no cache)."""
    z = dict(K=np.zeros((s.layers, B, s.heads, s.tokens, s.head_dim), np.float32),
             V=np.zeros((s.layers, B, s.heads, s.tokens, s.head_dim), np.float32),
             H=np.zeros((s.layers, B, s.tokens, s.hidden), np.float32))
    return [z] * T, np.zeros((B, T + 1, s.latent_ch) + s.latent_hw, np.float32)


@pytest.mark.gpu
@pytest.mark.timeout(300)
def test_paper_plan_eq1_per_chain_stepwise_vs_oracle():
    """The paper's reading of Eq. 2 with Eq. 1 computed from the prompt
    features: chain 0's delta tokens are only doubled (s = 1 >= tau_s: the
    region keeps the cache for all T steps), chain 1's are redrawn (s ~ 0:
    copy for floor(0.2 T) = 1 step, then region reuse), in one batch; every
    step against the oracle with re-synchronised inputs."""
    s, W, model, txt0, txt1, delta, x_T = _setup(seed=12)
    T, B = 5, 2
    txt1 = txt1.copy()
    txt1[0] = txt0[0]
    txt1[0][delta] = txt0[0][delta] * np.float32(2.0)  # same direction, exact in bf16
    sess = S.EditSession(model, B, T=T, reading="paper", tau_s=0.8)
    xT = torch.from_numpy(x_T).cuda()
    sess.first_turn(model.to_storage(txt0), xT)
    torch.cuda.synchronize()
    snap0 = _snapshot(sess, s, B)
    from paper_2608_29809_amd.runtime import ActiveSet
    region = [np.arange(40, 90), np.arange(0, 32)]
    out = sess.edit_turn(model.to_storage(txt1), xT, delta, region=ActiveSet.from_lists(region))
    torch.cuda.synchronize()
    sims = out["similarity"]
    assert abs(sims[0] - 1.0) < 1e-6 and sims[1] < 0.5, sims
    assert out["plans"][0] == ["copy"] * T
    assert out["plans"][1] == ["copy"] + ["reuse"] * (T - 1)
    snap1 = _snapshot(sess, s, B)
    w = _check_turn(s, W, txt1, x_T, out["plans"], snap0, snap1, region)
    print(f"paper-plan turn, worst per-step error {w:.2e}", flush=True)
    with pytest.raises(ValueError):
        sess.edit_turn(model.to_storage(txt1), xT, delta, similarity=0.2)


@pytest.mark.gpu
@pytest.mark.timeout(600)
def test_five_turn_chain_stepwise_vs_oracle():
    """One chain pair through five turns (a first turn and four edits, each
    with freshly redrawn delta tokens), dense_then_reuse: every step of
    every turn against the oracle with re-synchronised inputs at 2e-2; the
    pool after each turn is that turn's trajectory."""
    s, W, model, txt0, _, _, x_T = _setup(seed=14)
    T, B = 5, 2
    sess = S.EditSession(model, B, T=T, threshold=LOC_THRESHOLD)
    xT = torch.from_numpy(x_T).cuda()
    sess.first_turn(model.to_storage(txt0), xT)
    torch.cuda.synchronize()
    snap = _snapshot(sess, s, B)
    txt = txt0
    worst = 0.0
    for turn in range(1, 5):
        txt, delta = synth.edit_text(s, txt, 3, 100 + turn)
        delta = [int(d) for d in delta]
        maps_box = {}
        orig = model.localize

        def spy(maps, *a, **k):
            maps_box["maps"] = to_np(maps)
            return orig(maps, *a, **k)

        model.localize = spy
        out = sess.edit_turn(model.to_storage(txt), xT, delta)
        model.localize = orig
        torch.cuda.synchronize()
        act = out["active"]
        lists = [to_np(act.idx[act.host[b]:act.host[b + 1]]).astype(np.int64) for b in range(B)]
        new = _snapshot(sess, s, B)
        w = _check_turn(s, W, txt, x_T, out["plans"], snap, new, lists, delta, maps_box["maps"],
                        to_np(out["mask"]).astype(np.uint8))
        print(f"turn {turn}: region sizes {[len(x) for x in lists]}, worst per-step error {w:.2e}", flush=True)
        assert all(0 < len(x) < s.tokens for x in lists)
        worst = max(worst, w)
        snap = new
    assert sess.turns == 5
    print(f"five turns, worst per-step error {worst:.2e}", flush=True)


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

