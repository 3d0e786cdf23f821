"""Host checks of the workload set-up in ``synth``: every workload, shrunk to
a few chunks and layers, is laid out on the CPU under each layout option,
its tensors fit the one allocation reserved for them, and the views the call
receives cover distinct memory."""

import dataclasses

import pytest
import torch

import synth
from synth import harness


def _small(w):
    over = dict(n_chunks=min(w.n_chunks, 3), n_layers=min(w.n_layers, 2))
    if w.window_slots:
        over["window_slots"] = 4
    if w.paged:
        over["n_pool_pages"] = 3 * ((w.n_tokens + w.page_size - 1) // w.page_size) + 5
    return dataclasses.replace(w, **over)


def _span(t):
    lo = t.data_ptr()
    return lo, lo + t.element_size() * (1 + sum((s - 1) * st for s, st in zip(t.shape, t.stride())))


@pytest.mark.parametrize("name", sorted(synth.WORKLOADS))
@pytest.mark.parametrize("layout", [{}, {"separate_pools": True}, {"unit_major": False},
                                    {"pool_head_major": True}, {"u_token_major": True}])
def test_workload_fits_its_allocation(monkeypatch, name, layout):
    monkeypatch.setitem(synth.WORKLOADS, name, _small(synth.WORKLOADS[name]))
    p = harness.prepare(name, "cpu", **layout)
    arena = p.extra["arena"]
    assert arena is not None
    a_lo = arena.data_ptr()
    a_hi = a_lo + arena.numel()
    big = {k: t for k, t in p.tensors.items() if isinstance(t, torch.Tensor) and t.dtype == torch.bfloat16}
    assert big
    for k, t in big.items():
        lo, hi = _span(t)
        assert a_lo <= lo and hi <= a_hi, f"{k} lies outside the workload's allocation"
    # the inputs the call reads and the buffers it writes are distinct tensors of the arena
    # (views of one interleaved tensor aside, whose rows the library checks itself)
    owners = {k: t for k, t in big.items() if k in ("k_in", "v_in", "u_k", "u_v", "w_k", "w_v", "u_pe", "w_pe")}
    for k1, t1 in owners.items():
        for k2, t2 in owners.items():
            if k1 < k2 and not ({k1, k2} <= {"k_in", "v_in"} and "kv_window" in big):
                (l1, h1), (l2, h2) = _span(t1), _span(t2)
                assert h1 <= l2 or h2 <= l1, f"{k1} and {k2} overlap"


def test_arena_off_allocates_each_tensor():
    name = "gqa28l_8x1024_m16_reorder"
    w = synth.WORKLOADS[name]
    try:
        synth.WORKLOADS[name] = _small(w)
        p = harness.prepare(name, "cpu", arena=False)
    finally:
        synth.WORKLOADS[name] = w
    assert p.extra["arena"] is None
