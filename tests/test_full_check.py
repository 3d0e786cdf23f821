"""The element-complete checker itself (CPU): on a small paged workload whose
outputs are the reference's own bf16 results it finds nothing, and it finds
a single planted wrong element and a single unwritten (sentinel) element."""

from __future__ import annotations

import numpy as np

import oracle as ref
import synth
from tests import full_check as fc


def _case(seed=0):
    rng = np.random.default_rng(seed)
    C, L, H, n, D, m, P = 3, 2, 2, 48, 128, 16, 16
    rope = dict(theta=1e6, rope_dim=128, pairing="neox", rope_offset=0, sections=(16, 24, 24),
                section_order="blocked")
    orope = ref.Rope(**rope)
    pos = [tuple(int(x) for x in rng.integers(1, 4096, size=3)) for _ in range(C)]
    pages = C * n // P
    pt = rng.permutation(pages).reshape(C, n // P).astype(np.int32)
    K = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)
    V = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)
    U = synth.randn_bf16_numpy((C, L, H, n, m), 0.1, rng)
    W = synth.randn_bf16_numpy((C, L, H, m, D), 0.1, rng)
    Uv = synth.randn_bf16_numpy((C, L, H, n, m), 0.1, rng)
    Wv = synth.randn_bf16_numpy((C, L, H, m, D), 0.1, rng)
    kp = np.full((L, pages * P, H, D), fc.SENTINEL, np.uint16)
    vp = np.full_like(kp, fc.SENTINEL)
    for c in range(C):
        p3 = ref.positions_grid3(pos[c], 8, n)
        dst = [ref.paged_slot(pt[c], i, P) for i in range(n)]
        for l in range(L):
            for h in range(H):
                k = ref.rehydrate_k(ref.bf16_to_f64(K[c, l, :, h]), ref.bf16_to_f64(U[c, l, h]),
                                    ref.bf16_to_f64(W[c, l, h]), orope, p3)
                v = ref.rehydrate_v(ref.bf16_to_f64(V[c, l, :, h]), ref.bf16_to_f64(Uv[c, l, h]),
                                    ref.bf16_to_f64(Wv[c, l, h]))
                kp[l, dst, h] = ref.round_bf16(k)
                vp[l, dst, h] = ref.round_bf16(v)
    arrays = dict(K=K, V=V, U=U, W=W, Uv=Uv, Wv=Wv, kp=kp, vp=vp)
    meta = dict(C=C, L=L, H=H, n=n, D=D, m=m, P=P, rope=rope, pos=pos, pt=pt)
    return arrays, meta


def _run(arrays, meta):
    A, M = arrays, meta

    def fetch(l):
        return {"k_in": A["K"][:, l], "v_in": A["V"][:, l], "u_k": A["U"][:, l], "w_k": A["W"][:, l],
                "u_v": A["Uv"][:, l], "w_v": A["Wv"][:, l], "k_out": A["kp"][l], "v_out": A["vp"][l]}

    def jobs(l, paths, gen):
        base = dict(paths=paths, gen=gen, layer=l, n=M["n"], H=M["H"], D=M["D"], rope=M["rope"], pos=M["pos"],
                    pos_mode="grid3", grid_w=8, paged=True, page_size=M["P"], page_table=M["pt"], row_base=None,
                    patch_offset=0, patch_from_layer=0, m_k=M["m"], m_v=M["m"], m_pe=0, has_v=True, reloc=False,
                    delta=None)
        return [dict(base, c0=c, c1=c + 1) for c in range(M["C"])]

    return fc.run_layers(M["L"], 1 << 20, fetch, jobs, fc.check_rehydrate_layer, "checker self-test")


def test_full_checker_accepts_the_reference_and_catches_one_error():
    arrays, meta = _case()
    res = _run(arrays, meta)
    assert res.units == meta["C"] * meta["L"] * meta["H"] * 2
    assert res.bad == 0 and res.worst <= 1.0
    # one element off by 1/16 (8 x the tolerance) at the pool slot of chunk 1, token 5
    slot = ref.paged_slot(meta["pt"][1], 5, meta["P"])
    good = arrays["vp"][1, slot, 1, 77]
    arrays["vp"][1, slot, 1, 77] = ref.round_bf16(ref.bf16_to_f64(np.uint16(good)) + 0.0625)
    res = _run(arrays, meta)
    assert res.bad == 1 and res.first == ("V", 1, 1, 1)
    # and an element left unwritten (the NaN sentinel) fails as well
    arrays["vp"][1, slot, 1, 77] = good
    arrays["kp"][0, ref.paged_slot(meta["pt"][2], 40, meta["P"]), 0, 3] = fc.SENTINEL
    res = _run(arrays, meta)
    assert res.bad == 1 and res.first == ("K", 2, 0, 0)
