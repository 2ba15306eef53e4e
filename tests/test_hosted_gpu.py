"""Host-resident cache pool (pipelined execution, Sec. 3.4): the same step on
a pool in pinned host memory and on a device pool of identical contents
gives bit-identical results -- every slot of every block and chain, the
latent, the trajectory and the maps -- for a region-reuse step and a dense
step, and both match the oracle (whole step within 2e-2, and every block
with re-synchronised inputs).  Five blocks, so the three-entry staging ring
wraps around; three ragged chains, one of them with no active token."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from paper_2608_29809_amd.runtime import ActiveSet, RegionCacheModel
from _cases import (download_slot, gate_failures, oracle_text_kv, relerr, summarize, teacher_forced_dense,
                    teacher_forced_reuse, to_np, upload_slot, weights)

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[hosted]", *a, flush=True)


def _pools(model, shape, B, steps, seed):
    slot = synth.make_cache_slot(shape, B, seed)
    lat_next = synth.make_latent(shape, B, seed, stream=77)
    pools = []
    for host in (False, True):
        cache = model.alloc_cache(B, steps, host=host)
        cache.buf.zero_()
        upload_slot(model, cache, 1, slot)
        for b in range(B):
            cache.latent(b, 2).copy_(torch.from_numpy(lat_next[b]))
        pools.append(cache)
    torch.cuda.synchronize()
    return pools


def _compare(dev, host, t, L, B):
    a, b = download_slot(dev, t, L, B), download_slot(host, t, L, B)
    for k in ("K", "V", "H"):
        assert np.array_equal(a[k], b[k]), k
    for c in range(B):
        for e in range(dev.steps + 1):
            assert np.array_equal(to_np(dev.latent(c, e)), to_np(host.latent(c, e))), (c, e)


@pytest.mark.timeout(300)
def test_hosted_pool_matches_device_pool():
    shape = synth.ModelShape(layers=5, grid_h=32, grid_w=32, dtype="bf16")
    W = weights(shape, 11, True)
    B, steps = 3, 3
    model = RegionCacheModel(shape, W)
    dev, host = _pools(model, shape, B, steps, 11)
    txt = synth.make_text(shape, B, 11)
    tkv = model.prepare_text(model.to_storage(txt))
    rng = np.random.default_rng(11)
    per = [np.sort(rng.choice(shape.tokens, size=c, replace=False)) for c in (123, 0, 300)]
    act = ActiveSet.from_lists(per)
    lat = torch.from_numpy(synth.make_latent(shape, B, 11)).cuda()
    delta = [2, 40, 97]
    outs = []
    for cache in (dev, host):
        _say("reuse step, host pool" if cache.host else "reuse step, device pool")
        maps = torch.zeros((B, shape.tokens, len(delta)), device="cuda")
        out = torch.empty(lat.shape, device="cuda")
        model.reuse_step(cache, 1, act, lat, 700, 650, tkv, delta, maps, out)
        torch.cuda.synchronize()
        outs.append((to_np(out), to_np(maps)))
    assert np.array_equal(outs[0][0], outs[1][0])
    assert np.array_equal(outs[0][1], outs[1][1])
    _compare(dev, host, 1, shape.layers, B)
    # the rows the step computed did change (the comparison is not vacuous)
    before = synth.make_cache_slot(shape, B, 11)
    got = download_slot(host, 1, shape.layers, B)
    assert not np.array_equal(got["H"][:, 0][:, per[0]], before["H"][:, 0][:, per[0]])
    # and the hosted step is the method's step: against the oracle
    lat_np = to_np(lat)
    lat_next = synth.make_latent(shape, B, 11, stream=77)
    tkv_o = [oracle_text_kv(shape, W, txt[b]) for b in range(B)]
    for b in range(B):
        cs = dict(K=before["K"][:, b], V=before["V"][:, b], H=before["H"][:, b])
        r = O.reuse_step(shape, W, lat_np[b], 700, 650, tkv_o[b], per[b], cs, lat_next[b], np.array(delta))
        e = dict(latent=relerr(outs[1][0][b], r["latent_next"]), maps=relerr(outs[1][1][b], r["maps"]))
        if per[b].size:
            e.update(H=relerr(got["H"][:, b][:, per[b]], r["H"][:, per[b]]),
                     K=relerr(got["K"][:, b][:, :, per[b]], r["K"][:, :, per[b]]),
                     V=relerr(got["V"][:, b][:, :, per[b]], r["V"][:, :, per[b]]))
            pb = teacher_forced_reuse(shape, W, lat_np[b], 700, tkv_o[b], per[b], cs,
                                      {k: got[k][:, b] for k in ("K", "V", "H")})
            assert not gate_failures(pb, 2e-2), b
            e["per_block_worst_dH"] = summarize(pb)["dH"]
        _say(f"hosted reuse step vs oracle, chain {b} R={per[b].size}: " + " ".join(f"{k} {v:.2e}" for k, v in e.items()))
        assert e["latent"] < 2e-2 and e["maps"] < 2e-2 and e.get("H", 0) < 2e-2 and e.get("K", 0) < 2e-2
        assert e.get("V", 0) < 2e-2

    outs = []
    for cache in (dev, host):
        _say("dense step, host pool" if cache.host else "dense step, device pool")
        out = torch.empty(lat.shape, device="cuda")
        model.build_cache(cache, 0, lat, 999, 700, tkv, latent_out=out)
        torch.cuda.synchronize()
        outs.append(to_np(out))
    assert np.array_equal(outs[0], outs[1])
    _compare(dev, host, 0, shape.layers, B)
    got = download_slot(host, 0, shape.layers, B)
    for b in range(B):
        r = O.dense_step(shape, W, lat_np[b], 999, 700, tkv_o[b])
        e = dict(latent=relerr(outs[1][b], r["latent_next"]), H=relerr(got["H"][:, b], r["H"]),
                 K=relerr(got["K"][:, b], r["K"]), V=relerr(got["V"][:, b], r["V"]))
        pb = teacher_forced_dense(shape, W, lat_np[b], 999, tkv_o[b], {k: got[k][:, b] for k in ("K", "V", "H")})
        _say(f"hosted dense step vs oracle, chain {b}: " + " ".join(f"{k} {v:.2e}" for k, v in e.items()))
        assert max(e.values()) < 2e-2 and not gate_failures(pb, 2e-2), b
