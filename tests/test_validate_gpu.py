"""Device check of active sets (rc_validate_active and RC_VALIDATE on the
reuse step; the active token set of Sec. 3.3 must be a strictly ascending
list of tokens of the grid per chain).

Invalid lists are only ever handed to the check itself.  The step with
RC_VALIDATE is given in-range lists only (a duplicate, a descending pair),
which could not write outside the slot even if the check missed them; it
must refuse them before any launch and leave the pool and outputs as they
were."""
import sys

import numpy as np
import pytest
import torch

import synth
from _cases import upload_slot, weights

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2608_29809_amd import abi
    from paper_2608_29809_amd.runtime import ActiveSet, RegionCacheModel


def _say(*a):
    print("[validate]", *a, flush=True, file=sys.stderr)


SHAPE = synth.ModelShape(layers=1, grid_h=16, grid_w=16, dtype="bf16")


@pytest.fixture(scope="module")
def model():
    return RegionCacheModel(SHAPE, weights(SHAPE, 21))


def _raw(idx, offs_dev, offs_host):
    """An active set from raw lists (the device offsets may differ from the host copy)."""
    t_idx = torch.tensor(np.asarray(idx, np.int64), dtype=torch.int32, device="cuda")
    t_off = torch.tensor(offs_dev, dtype=torch.int32, device="cuda")
    return ActiveSet(t_idx, t_off, offs_host)


def test_valid_sets_pass(model):
    N = SHAPE.tokens
    for per in ([np.arange(N)], [np.zeros(0, int), np.array([0, 5, N - 1])],
                [np.array([10, 200]), np.array([3, 4, 5])],   # chain 1 may start below chain 0's last token
                [np.zeros(0, int)] * 3):
        _say("valid", [len(p) for p in per])
        model.validate_active(ActiveSet.from_lists(per))


@pytest.mark.parametrize("case", ["token_N", "negative", "beyond_16_bits", "duplicate", "descending",
                                  "device_offsets_differ", "last_chain"])
def test_invalid_sets_refused(model, case):
    N = SHAPE.tokens
    idx, offs = {
        "token_N": ([1, 2, N], [0, 3]),
        "negative": ([-1, 2, 3], [0, 3]),
        "beyond_16_bits": ([1, 65536 + 5], [0, 2]),
        "duplicate": ([4, 9, 9, 20], [0, 4]),
        "descending": ([4, 30, 20], [0, 3]),
        "device_offsets_differ": ([1, 2, 3, 4], [0, 2, 4]),
        "last_chain": ([1, 2, 3, 7, 7], [0, 3, 5]),
    }[case]
    host = list(offs)
    dev = list(offs)
    if case == "device_offsets_differ":
        dev = [0, 3, 4]
    _say("invalid", case)
    with pytest.raises(abi.RcError) as ei:
        model.validate_active(_raw(idx, dev, host))
    assert ei.value.status == -4, ei.value
    msg = str(ei.value)
    assert ("chain" in msg) or ("offsets" in msg), msg
    if case == "last_chain":
        assert "chain 1" in msg, msg


def _step_setup(model, per):
    B = len(per)
    cache = model.alloc_cache(B, 2)
    upload_slot(model, cache, 1, synth.make_cache_slot(SHAPE, B, 21))
    for b in range(B):
        cache.latent(b, 2).copy_(torch.from_numpy(synth.make_latent(SHAPE, B, 21, stream=77)[b]))
    tkv = model.prepare_text(model.to_storage(synth.make_text(SHAPE, B, 21)))
    lat = torch.from_numpy(synth.make_latent(SHAPE, B, 21)).cuda()
    return cache, tkv, lat


def test_reuse_step_with_validate_flag(model):
    per = [np.array([3, 17, 18, 100]), np.arange(40, 90)]
    cache, tkv, lat = _step_setup(model, per)
    ref = cache.buf.clone()
    out_a = torch.full(lat.shape, float("nan"), device="cuda")
    model.reuse_step(cache, 1, ActiveSet.from_lists(per), lat, 500, 450, tkv, latent_out=out_a)
    after_a = cache.buf.clone()
    cache.buf.copy_(ref)
    out_b = torch.full(lat.shape, float("nan"), device="cuda")
    model.reuse_step(cache, 1, ActiveSet.from_lists(per), lat, 500, 450, tkv, latent_out=out_b, validate=True)
    torch.cuda.synchronize()
    assert torch.equal(after_a, cache.buf) and torch.equal(out_a, out_b)
    # in-range but invalid lists: refused before any launch, nothing written
    for bad in ([np.array([3, 17, 17, 100]), np.arange(40, 90)], [np.array([3, 17, 18, 100]), np.arange(90, 40, -1)]):
        cache.buf.copy_(ref)
        out = torch.full(lat.shape, float("nan"), device="cuda")
        torch.cuda.synchronize()
        with pytest.raises(abi.RcError) as ei:
            model.reuse_step(cache, 1, ActiveSet.from_lists(bad), lat, 500, 450, tkv, latent_out=out, validate=True)
        torch.cuda.synchronize()
        assert ei.value.status == -4
        assert torch.equal(cache.buf, ref)
        assert torch.isnan(out).all()
