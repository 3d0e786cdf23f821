"""The operator workloads at full size, every element checked against the fp64
reference: every (chunk, layer, head) unit of the one-layer chunk, the
28-layer reorder, the MLA chunks, the 80-layer paged recall and the other
workloads (relocation with removal patches, the MLA band patch, the deep-half
recall, the mid-size recall), keys and values, and every survivor unit of a
window slide.  Outputs are filled with a
NaN sentinel first: a written element that kept it fails the tolerance, and
the sentinels left in each output layer must be exactly its unwritten
extent (rows or pool slots no chunk maps to)."""

from __future__ import annotations

import numpy as np
import pytest

import synth
from synth import harness
from tests import full_check as fc
from tests.gpu_util import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def device():
    return require_gpu()


def _free():
    import gc

    import torch

    gc.collect()
    torch.cuda.empty_cache()


def _rope_kw(w):
    return dict(theta=w.theta, rope_dim=w.rope_dim, pairing=w.pairing, rope_offset=w.rope_offset,
                sections=w.sections, section_order=w.section_order)


def _sentinels(t) -> int:
    import torch

    return int((t.view(torch.int16) == fc.SENTINEL).sum().item())


@pytest.mark.parametrize("name", ["gqa1l_256tok_m8", "gqa28l_8x1024_m16_reorder", "mla27l_4x2048_m32",
                                  "gqa80l_64x1024_m64_mrope_paged"] + synth.EXTRA_WORKLOADS)
def test_every_element_of_the_workload(device, name):
    import torch

    print(f"[case] full {name}", flush=True)
    p = harness.prepare(name, device)
    w, T, meta = p.workload, p.tensors, p.meta
    C, L, H, n, D = w.n_chunks, w.n_layers, w.n_heads, w.n_tokens, w.head_dim
    if w.reloc:
        # in place: the survivors' keys and values as they were before the move
        outs = ["k_in", "v_in"] if w.has_v else ["k_in"]
        inputs = {(nm, l): fc.bits(T[nm][:, l]) for nm in outs for l in range(L)}
    else:
        outs = ["k_pool", "v_pool"] if w.paged else ["k_out_rows", "v_out_rows"]
        outs = [o for o in outs if o in T]
        for o in outs:
            T[o].view(torch.int16).fill_(fc.SENTINEL)
    p.step()
    torch.cuda.synchronize()

    if not w.reloc:
        # unwritten extent of each output layer: pool slots or rows no token maps to
        rows_total = w.n_pool_pages * w.page_size if w.paged else T[outs[0]].shape[1]
        for o in outs:
            for l in (0, L - 1):
                assert _sentinels(T[o][l]) == (rows_total - C * n) * H * D, (o, l)

    pos = [tuple(int(x) for x in meta.pos[c]) for c in range(C)]

    def fetch(l):
        if w.reloc:
            a = {"k_in": inputs[("k_in", l)], "k_out": fc.bits(T["k_in"][:, l])}
            if w.has_v:
                a["v_in"] = inputs[("v_in", l)]
                a["v_out"] = fc.bits(T["v_in"][:, l])
        else:
            a = {"k_in": fc.bits(T["k_in"][:, l]), "k_out": fc.bits(T[outs[0]][l])}
            if w.has_v:
                a["v_in"] = fc.bits(T["v_in"][:, l])
                a["v_out"] = fc.bits(T[outs[1]][l])
        if l >= w.patch_from_layer:
            for nm in ("u_k", "w_k", "u_v", "w_v", "u_pe", "w_pe"):
                if nm in T:
                    a[nm] = fc.bits(T[nm][:, l])
        return a

    def jobs(l, paths, gen):
        base = dict(paths=paths, gen=gen, layer=l, n=n, H=H, D=D, rope=_rope_kw(w), pos=pos,
                    pos_mode=w.pos_mode, grid_w=w.grid_w, paged=w.paged, page_size=w.page_size,
                    page_table=meta.page_table if w.paged else None,
                    row_base=None if w.paged else meta.row_base, patch_offset=w.patch_offset,
                    patch_from_layer=w.patch_from_layer, m_k=w.m_k, m_v=w.m_v if w.has_v else 0,
                    m_pe=w.m_pe, has_v=w.has_v, reloc=w.reloc,
                    delta=[tuple(int(x) for x in meta.delta[c]) for c in range(C)] if w.reloc else None)
        return [dict(base, c0=c, c1=c + 1) for c in range(C)]

    layer_bytes = sum(a.nbytes for a in fetch(L - 1).values())
    res = fc.run_layers(L, layer_bytes, fetch, jobs, fc.check_rehydrate_layer, name)
    planes = 2 if w.has_v else 1
    print(f"[full] {name}: {res.units} units ({C}x{L}x{H} x {planes} planes), {res.bad} elements out of "
          f"tolerance, worst err/bound {res.worst:.3f}, {res.seconds:.1f} s on {res.workers} workers", flush=True)
    assert res.units == C * L * H * planes
    assert res.bad == 0, f"first bad unit {res.first}"
    del p
    _free()


def test_every_survivor_of_a_window_slide(device):
    """The 32-layer window: all 15 survivor chunks x 32 layers x 32 heads of
    the first slide against one shift of the window as it was, and the
    evicted slot bit for bit untouched."""
    import torch

    print("[case] full window slide", flush=True)
    p = harness.prepare("mha32l_window16x512_shift", device)
    w, T = p.workload, p.tensors
    L, H, n = w.n_layers, w.n_heads, w.n_tokens
    p.extra["set_slide"](0)
    slots = [int(s) for s in synth.window_survivor_slots(w, 0)]
    evict = 0 % w.window_slots
    before = fc.bits(T["window"])                  # [L, S*n, H, D], the window before the slide
    p.step()
    torch.cuda.synchronize()
    after_ev = fc.bits(T["window"][:, evict * n:(evict + 1) * n])
    assert np.array_equal(after_ev, before[:, evict * n:(evict + 1) * n])

    def fetch(l):
        return {"before": before[l], "after": fc.bits(T["window"][l])}

    def jobs(l, paths, gen):
        return [dict(paths=paths, gen=gen, layer=l, n=n, H=H, rope=_rope_kw(w), delta=(w.delta,) * 3,
                     slots=slots[k:k + 4]) for k in range(0, len(slots), 4)]

    res = fc.run_layers(L, 2 * before[0].nbytes, fetch, jobs, fc.check_shift_layer, "window slide")
    print(f"[full] window slide: {res.units} survivor units, {res.bad} elements out of tolerance, "
          f"worst err/bound {res.worst:.3f}, {res.seconds:.1f} s on {res.workers} workers", flush=True)
    assert res.units == len(slots) * L * H
    assert res.bad == 0, f"first bad unit {res.first}"
    del p, before
    _free()
