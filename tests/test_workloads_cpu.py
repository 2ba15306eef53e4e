"""The seeded synthetic workloads the benchmark times (host side only): the
edit region of the 1024 px reuse step, the batch active-fraction masks and
the resolution masks have the sizes the benchmark reports, are valid token
lists, and do not change with the seed stream of other generators."""
import numpy as np

import synth


def _valid(idx, n):
    idx = np.asarray(idx)
    return idx.ndim == 1 and idx.size > 0 and idx.min() >= 0 and idx.max() < n and np.all(np.diff(idx) > 0)


def test_bench_edit_region():
    mask, frac, n_blobs = synth.c3_edit_region(0)
    idx = np.flatnonzero(mask)
    assert idx.size == 723 and 1 <= n_blobs <= 3 and 0.10 <= frac <= 0.20
    assert idx.size == round(frac * 4096)
    assert _valid(idx, 4096)


def test_sweep_regions_sizes():
    for f, n in ((0.05, 205), (0.10, 410), (0.25, 1024), (0.50, 2048), (1.00, 4096)):
        per = synth.sweep_regions(0, f)
        assert len(per) == 4
        assert [p.size for p in per] == [n] * 4
        assert all(_valid(p, 4096) for p in per)
    # chains draw their own blobs
    per = synth.sweep_regions(0, 0.10)
    assert not all(np.array_equal(per[0], p) for p in per[1:])


def test_resolution_regions_sizes():
    for g, n in ((32, 154), (64, 614), (128, 2458)):
        idx = synth.resolution_region(0, g)
        assert idx.size == n and _valid(idx, g * g)


def test_regions_are_seeded():
    a = synth.sweep_regions(3, 0.25)
    b = synth.sweep_regions(3, 0.25)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    assert not np.array_equal(synth.resolution_region(0, 64), synth.resolution_region(1, 64))
