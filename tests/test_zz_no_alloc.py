"""The allocation-free maps call (rc_maps_from_logits_noalloc): through the C
ABI, its maps equal those of rc_maps_from_logits with a caller-owned scratch
buffer, bit for bit, on two calls in a row -- the full 1024 px localisation
logits, then a smaller problem -- and both agree with the oracle on the
small one.  The library-owned scratch keeps the first call's partial maps;
the second call must not read them."""
import ctypes as C
import sys

import numpy as np
import pytest
import torch

import oracle as O
import synth
from _cases import relerr, to_np

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[no-alloc]", *a, flush=True, file=sys.stderr)


def _both(Zt, delta):
    from paper_2608_29809_amd import abi
    L, Hh, N, M = Zt.shape
    nd = len(delta)
    d = (C.c_int32 * nd)(*[int(x) for x in delta])
    dp = C.cast(d, C.POINTER(C.c_int32))
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    ref = torch.full((N, nd), float("nan"), dtype=torch.float32, device="cuda")
    got = torch.full((N, nd), float("nan"), dtype=torch.float32, device="cuda")
    nbytes = abi.rc_maps_from_logits_scratch_bytes(L, N, nd)
    scratch = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    abi.rc_maps_from_logits(C.c_void_p(Zt.data_ptr()), L, Hh, N, M, dp, nd, C.c_void_p(ref.data_ptr()),
                            C.c_void_p(scratch.data_ptr()), nbytes, stream)
    abi.rc_maps_from_logits_noalloc(C.c_void_p(Zt.data_ptr()), L, Hh, N, M, dp, nd, C.c_void_p(got.data_ptr()),
                                    stream)
    torch.cuda.synchronize()
    return got, ref


@pytest.mark.timeout(300)
def test_noalloc_maps_match_scratch_entry_point_two_calls():
    from paper_2608_29809_amd import abi
    cases = [
        # the 1024 px localisation workload: 28 layers, 16 heads, 4096 tokens, 6 delta columns
        dict(L=28, H=16, g=64, nd=6, seed=3, frac=0.12),
        # then a smaller one: fewer layers, tokens and delta columns
        dict(L=3, H=4, g=16, nd=2, seed=5, frac=0.2),
    ]
    for k, c in enumerate(cases):
        N = c["g"] * c["g"]
        _say(f"call {k}: logits [{c['L']},{c['H']},{N},120], {c['nd']} delta columns")
        Z, delta, _ = synth.make_logits(c["L"], c["H"], N, 120, c["g"], c["g"], n_delta=c["nd"], seed=c["seed"],
                                        frac=c["frac"])
        Zt = torch.from_numpy(Z).to(torch.bfloat16).cuda()
        got, ref = _both(Zt, delta)
        assert torch.isfinite(ref).all()
        assert torch.equal(got, ref), k
        if k == 1:
            e = relerr(to_np(got), O.maps_from_logits(Z, delta))
            _say(f"small call vs oracle: {e:.2e}")
            assert e < 1e-4
    # a problem beyond the static scratch is refused before any launch
    d = (C.c_int32 * 8)(*range(8))
    out = torch.empty(16, dtype=torch.float32, device="cuda")
    with pytest.raises(abi.RcError) as ei:
        abi.rc_maps_from_logits_noalloc(C.c_void_p(Zt.data_ptr()), 33, 16, 16384, 120, C.cast(d, C.POINTER(C.c_int32)),
                                        8, C.c_void_p(out.data_ptr()), None)
    assert ei.value.status == -5
