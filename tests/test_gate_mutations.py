"""The parity gate of the full-size region-step tests can fail.

Four plausible self-attention mistakes are planted in the oracle (on the
CPU) at the benchmark's own region (1024 px, 4096 tokens, 723 active rows)
with the stress weights the GPU tests use; the broken step's slot is then
judged by the same teacher-forced per-block gate (tests/_cases.py) that
judges the GPU's slot, and must be rejected at the 2e-2 tolerance:

* attention output zero,
* uniform attention (softmax replaced by the mean over keys),
* stale cached keys/values for the active rows (attention reads the slot
  before the fresh keys/values are written: the ordering Sec. 3.4's fused
  scatter must respect),
* softmax scale sqrt(2) too large.

The unbroken oracle, rounded to bf16 like the GPU's slot, passes the same
gate (errors at storage-rounding level), so the
gate tests the attention, not the harness.  The storage-rounding floor the
gate adds to the per-block change (tests/_cases.py) is computed here from
the same bf16-rounded quantities it is computed from on the GPU.  Two blocks keep the CPU time
small; the gate is per block, so more blocks only add chances to fail."""
import contextlib
import dataclasses

import numpy as np
import pytest

import oracle as O
import oracle.rc_oracle as OM
import synth
from _cases import gate_failures, summarize, teacher_forced_reuse

TOL = 2e-2
_real_attention = OM.attention
_real_block_reuse = OM.block_reuse


@contextlib.contextmanager
def _patched(name, fn):
    old = getattr(OM, name)
    setattr(OM, name, fn)  # the module whose globals the oracle's functions resolve
    try:
        yield
    finally:
        setattr(OM, name, old)


def _self_attention_only(mut):
    """Wrap a mutated attention so that only the self-attention (the call
    over the N slot keys, without probabilities) is affected."""
    def att(q, k, v, return_probs=False):
        if return_probs:
            return _real_attention(q, k, v, return_probs)
        return mut(q, k, v)
    return att


def _zero(q, k, v):
    return np.zeros_like(q)


def _uniform(q, k, v):
    return np.broadcast_to(v.mean(axis=0, keepdims=True), q.shape).copy()


def _scaled(q, k, v):
    return _real_attention(q * np.sqrt(2.0), k, v)


def _stale_block_reuse(lw, X_act, idx, mod, textK, textV, cacheK, cacheV, cacheH, heads, delta=None,
                       dt=np.float64):
    stale_k = np.asarray(cacheK, dt).transpose(1, 0, 2)
    stale_v = np.asarray(cacheV, dt).transpose(1, 0, 2)

    def att(q, k, v, return_probs=False):
        if return_probs:
            return _real_attention(q, k, v, return_probs)
        return _real_attention(q, stale_k, stale_v)

    with _patched("attention", att):
        return _real_block_reuse(lw, X_act, idx, mod, textK, textV, cacheK, cacheV, cacheH, heads, delta, dt)


@pytest.fixture(scope="module")
def bench_case():
    s = dataclasses.replace(synth.shape_c3(), layers=2)
    W = synth.make_weights(s, seed=0, stress=True)
    idx = np.flatnonzero(synth.c3_edit_region(0)[0])
    assert idx.size == 723
    txt = synth.make_text(s, 1, 0)
    lat = synth.make_latent(s, 1, 0)[0]
    lat_next = synth.make_latent(s, 1, 0, stream=77)[0]
    slot = synth.make_cache_slot(s, 1, 0)
    cache = dict(K=slot["K"][:, 0], V=slot["V"][:, 0], H=slot["H"][:, 0])
    y = O.caption_projection(W, txt[0])
    tkv = [O.text_kv(lw, y, s.heads) for lw in W["layers"]]
    return s, W, idx, lat, lat_next, cache, tkv


def _run(case, ctx):
    s, W, idx, lat, lat_next, cache, tkv = case
    with ctx:
        r = O.reuse_step(s, W, lat, 842, 789, tkv, idx, cache, lat_next)
    # stored as the GPU stores its slot: rounded to bf16
    got = {k: synth.bf16_round(r[k].astype(np.float32)) for k in ("K", "V", "H")}
    return teacher_forced_reuse(s, W, lat, 842, tkv, idx, cache, got)


def test_unbroken_oracle_passes_the_gate(bench_case):
    per = _run(bench_case, contextlib.nullcontext())
    w = summarize(per)
    assert max(w["H"], w["dH"], w["K"], w["V"]) < 1e-2, w  # storage rounding only
    assert not gate_failures(per, TOL)


@pytest.mark.parametrize("mutation", ["zero_output", "uniform_softmax", "stale_kv", "scale_sqrt2"])
def test_gate_rejects_broken_self_attention(bench_case, mutation):
    ctx = {
        "zero_output": _patched("attention", _self_attention_only(_zero)),
        "uniform_softmax": _patched("attention", _self_attention_only(_uniform)),
        "stale_kv": _patched("block_reuse", _stale_block_reuse),
        "scale_sqrt2": _patched("attention", _self_attention_only(_scaled)),
    }[mutation]
    per = _run(bench_case, ctx)
    w = summarize(per)
    print(mutation, {k: f"{v:.3g}" for k, v in w.items()})
    # every block is rejected, by a wide margin: the per-block change of the
    # active rows carries the attention branch
    assert len(gate_failures(per, TOL)) == len(per), (mutation, per)
    assert all(e["dH"] > 5 * (TOL + e["dH_floor"]) for e in per), (mutation, per)
