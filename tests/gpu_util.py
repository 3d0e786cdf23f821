"""Shared helpers of the GPU parity tests: bf16 transfers, the comparator and
small seeded cases run through the C ABI and through the fp64 reference."""

from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import numpy as np
import pytest

import oracle as ref
import synth

# |gpu - ref| <= 2^-7 * max(1, |ref|): a single bf16 rounding of an fp32
# result carries at most 2^-8 relative error, the rest is fp32 accumulation
# and angle error (~1e-6), so the bound leaves a 2x margin.
TOL = 2.0 ** -7
SENTINEL = 0x7FC1          # a NaN pattern no kernel output can produce from finite inputs


def require_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_23581_amd as km

    km.lib()  # a missing library where a GPU is present is a failure, not a skip
    return torch.device("cuda:0")


def bits(t) -> np.ndarray:
    import torch

    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16)


def dev(b: np.ndarray, device):
    import torch

    return torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(torch.bfloat16).to(device)


def dev_i32(a, device):
    import torch

    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).to(device)


def assert_close(gpu_bits: np.ndarray, want: np.ndarray, what: str):
    got = ref.bf16_to_f64(gpu_bits)
    err = np.abs(got - want)
    bound = TOL * np.maximum(1.0, np.abs(want))
    bad = ~(err <= bound)
    if bad.any():
        idx = np.argwhere(bad)[:5]
        worst = float(np.nanmax(err / bound))
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} elements out of tolerance "
                             f"(worst err/bound {worst:.3g}); first at {idx.tolist()}: "
                             f"got {got[tuple(idx[0])]} want {want[tuple(idx[0])]}")


def oracle_rope(rs) -> "ref.Rope":
    return ref.Rope(theta=rs.theta, rope_dim=rs.rope_dim, pairing=rs.pairing,
                    rope_offset=rs.rope_offset, sections=rs.sections, section_order=rs.section_order)


@dataclasses.dataclass
class RehydrateCase:
    C: int = 2
    L: int = 2
    H: int = 3
    n: int = 100
    D: int = 128
    m_k: int = 16
    m_v: int = 16
    theta: float = 1e6
    rope_dim: int = 128
    rope_offset: int = 0
    pairing: str = "neox"
    sections: Optional[Tuple[int, int, int]] = None
    section_order: str = "blocked"
    patch: Tuple[int, int] = (0, 128)
    has_v: bool = True
    pos_mode: str = "linear"           # linear | grid3 | explicit
    grid_w: int = 32
    p0_range: Tuple[int, int] = (0, 40000)
    paged: bool = False
    page_size: int = 16
    extra_pages: int = 5
    ragged: bool = False
    post_rope: bool = False
    shared_w: bool = False
    reloc: bool = False                # keys already rotated; move by a per-chunk delta
    m_pe: int = 0                      # separate patch on the rope band (MLA k_pe), keys only
    layer_rank: Optional[Tuple[int, ...]] = None   # rank used per layer (both planes)
    row_base: bool = True              # dense output: chunks at permuted row bases, else chunk c at rows c*n..
    in_place: bool = False             # dense output without row_base written over the input
    unit_major: bool = False           # input memory [C, L, H, n, D] (rows of one head contiguous)
    kv_interleaved: bool = False       # K and V outputs in one tensor [L, rows, K|V, H, D]
    kernel: int = 0                    # kamera_kernel_choice requested (0: AUTO)
    plan: Optional[int] = None         # kernel kamera_rehydrate_plan must report for the case
    max_workgroups: int = 0            # cap on the launch's workgroups (long segments per workgroup)
    schedule: int = 0                  # kamera_row_schedule requested (0: AUTO)
    sched: Optional[int] = None        # schedule kamera_rehydrate_schedule must report for the case
    seed: int = 0


def run_rehydrate(case: RehydrateCase, device):
    """Run one seeded case through the library and check every output element
    against the fp64 reference; untouched destination rows must keep the
    sentinel bits."""
    import paper_2606_23581_amd as km

    rng = np.random.default_rng(case.seed)
    C, L, H, n, D = case.C, case.L, case.H, case.n, case.D
    K = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)
    V = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng) if case.has_v else None
    pd = case.patch[1]

    def factors(m):
        if m == 0:
            return None, None
        U = synth.randn_bf16_numpy((C, L, H, n, m), 0.1, rng)
        Wc = 1 if case.shared_w else C
        W = synth.randn_bf16_numpy((Wc, L, H, m, pd), 0.1, rng)
        return U, W

    Uk, Wk = factors(case.m_k)
    Uv, Wv = factors(case.m_v) if case.has_v else (None, None)
    Upe = Wpe = None
    if case.m_pe:
        Upe = synth.randn_bf16_numpy((C, L, H, n, case.m_pe), 0.1, rng)
        Wpe = synth.randn_bf16_numpy((1 if case.shared_w else C, L, H, case.m_pe, case.rope_dim), 0.1, rng)
    delta = rng.integers(-3000, 3000, size=(C, 3)).astype(np.int32)
    if case.sections is None:
        delta[:, 1:] = delta[:, :1]
    n_c = (rng.integers(0, n + 1, size=C) if case.ragged else np.full(C, n)).astype(np.int32)
    if case.ragged:
        n_c[0] = n
    # positions
    pos = np.zeros((C, 3), dtype=np.int32)
    explicit = None
    if case.pos_mode == "linear":
        pos[:, :] = rng.integers(case.p0_range[0], case.p0_range[1], size=C)[:, None]
    elif case.pos_mode == "grid3":
        pos[:] = rng.integers(case.p0_range[0], case.p0_range[1], size=(C, 3))
    else:
        explicit = rng.integers(case.p0_range[0], case.p0_range[1], size=(C, n, 3)).astype(np.int32)
    # destination
    if case.paged:
        pages = (n + case.page_size - 1) // case.page_size
        n_pool_pages = C * pages + case.extra_pages
        pt = rng.permutation(n_pool_pages)[: C * pages].reshape(C, pages).astype(np.int32)
        slots = n_pool_pages * case.page_size
        out_shape = (L, slots, H, D)
    elif case.row_base:
        row_base = (rng.permutation(C) * (n + 3)).astype(np.int32)
        rows = int(row_base.max()) + n + 3
        out_shape = (L, rows, H, D)
    else:
        # chunk c at rows c*n .. c*n + n - 1 of a [L, C*n, H, D] buffer, seen as [C, L, n, H, D]
        row_base = (np.arange(C) * n).astype(np.int32)
        out_shape = (L, C * n, H, D)
    assert not case.in_place or (not case.paged and not case.row_base and not case.ragged)

    rs = km.RopeSpec(theta=case.theta, rope_dim=case.rope_dim, pairing=case.pairing,
                     rope_offset=case.rope_offset, sections=case.sections,
                     section_order=case.section_order)
    def chunk_rows(X):
        # [C, L, n, H, D] numpy -> its [L, C*n, H, D] memory
        return np.ascontiguousarray(X.transpose(1, 0, 2, 3, 4).reshape(L, C * n, H, D))

    def rows_view(t):
        # a [L, C*n, H, D] device buffer as the [C, L, n, H, D] tensor the call takes
        st = t.stride()
        return t.as_strided((C, L, n, H, D), (n * st[1], st[0], st[1], st[2], st[3]))

    def dev_in(X):
        if case.unit_major:
            return dev(np.ascontiguousarray(X.transpose(0, 1, 3, 2, 4)), device).permute(0, 1, 3, 2, 4)
        return dev(X, device)

    if case.in_place and case.kv_interleaved:
        kv_out = dev(np.stack([chunk_rows(K), chunk_rows(V)], axis=2), device)
        k_out, v_out = kv_out[:, :, 0], kv_out[:, :, 1]
    elif case.in_place:
        k_out = dev(chunk_rows(K), device)
        v_out = dev(chunk_rows(V), device) if case.has_v else None
    elif case.kv_interleaved:
        assert case.has_v
        kv_out = dev(np.full((*out_shape[:2], 2, *out_shape[2:]), SENTINEL, np.uint16), device)
        k_out, v_out = kv_out[:, :, 0], kv_out[:, :, 1]
    else:
        k_out = dev(np.full(out_shape, SENTINEL, np.uint16), device)
        v_out = dev(np.full(out_shape, SENTINEL, np.uint16), device) if case.has_v else None

    def wt(W):
        if W is None:
            return None
        t = dev(W, device)
        return t.expand(C, *t.shape[1:]) if case.shared_w else t

    kw = dict(rope=rs, u_k=dev(Uk, device) if Uk is not None else None, w_k=wt(Wk),
              k_patch=case.patch, patch_frame=km.PATCH_POST_ROPE if case.post_rope else km.PATCH_PRE_ROPE,
              pos_mode={"linear": km.POS_LINEAR, "grid3": km.POS_GRID3, "explicit": km.POS_EXPLICIT}[case.pos_mode],
              grid_w=case.grid_w, chunk_pos=dev_i32(pos, device),
              explicit_pos=dev_i32(explicit, device) if explicit is not None else None,
              chunk_tokens=dev_i32(n_c, device) if case.ragged else None, kernel=case.kernel,
              max_workgroups=case.max_workgroups, schedule=case.schedule)
    status = dev_i32(np.zeros(1), device)
    kw["status"] = status
    if case.reloc:
        kw["delta"] = dev_i32(delta, device)
    if case.m_pe:
        kw.update(u_pe=dev(Upe, device), w_pe=wt(Wpe))
    if case.layer_rank is not None:
        lr = dev_i32(np.array(case.layer_rank), device)
        kw.update(k_layer_rank=lr, v_layer_rank=lr, pe_layer_rank=lr)
    if case.has_v:
        kw.update(v_in=rows_view(v_out) if case.in_place else dev_in(V),
                  u_v=dev(Uv, device) if Uv is not None else None, w_v=wt(Wv), v_patch=case.patch)
    if case.paged:
        kw.update(page_table=dev_i32(pt, device), page_size=case.page_size, n_pool_pages=n_pool_pages)
        prep = km.prepare_rehydrate(dev_in(K), k_out, v_out=v_out, **kw)
    elif case.row_base:
        ko = k_out.unsqueeze(0).expand(C, *out_shape)
        vo = v_out.unsqueeze(0).expand(C, *out_shape) if case.has_v else None
        prep = km.prepare_rehydrate(dev_in(K), ko, v_out=vo, row_base=dev_i32(row_base, device), **kw)
    else:
        ko = rows_view(k_out)
        vo = rows_view(v_out) if case.has_v else None
        prep = km.prepare_rehydrate(ko if case.in_place else dev_in(K), ko, v_out=vo, **kw)
    if case.plan is not None:
        assert km.rehydrate_plan(prep) == case.plan
    if case.sched is not None:
        assert km.rehydrate_schedule(prep) == case.sched
    prep.launch()
    import torch

    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == 0
    kb = bits(k_out)
    vb = bits(v_out) if case.has_v else None

    orope = oracle_rope(rs)
    touched = np.zeros(out_shape[:2], dtype=bool)
    for c in range(C):
        nc = int(n_c[c])
        if case.pos_mode == "linear":
            p3 = ref.positions_linear(int(pos[c, 0]), nc)
        elif case.pos_mode == "grid3":
            p3 = ref.positions_grid3(pos[c], case.grid_w, nc)
        else:
            p3 = explicit[c, :nc].astype(np.int64)
        if case.paged:
            dst = np.array([ref.paged_slot(pt[c], i, case.page_size) for i in range(nc)], dtype=np.int64)
        else:
            dst = row_base[c] + np.arange(nc)
        for l in range(L):
            touched[l, dst] = True
            r_l = None if case.layer_rank is None else case.layer_rank[l]

            def fac(Ua, Wa, width_off):
                if Ua is None:
                    return None, None
                r = Ua.shape[-1] if r_l is None else min(r_l, Ua.shape[-1])
                u_ = ref.bf16_to_f64(Ua[c, l, h, :nc, :r])
                w_ = ref.bf16_to_f64(Wa[0 if case.shared_w else c, l, h, :r])
                return u_, w_

            for h in range(H):
                Kin = ref.bf16_to_f64(K[c, l, :nc, h])
                u, w = fac(Uk, Wk, 0)
                poff = case.patch[0]
                if case.m_pe:
                    # two patches on disjoint columns == one patch with a block basis
                    # (the latent's rank may be 0)
                    up, wp = fac(Upe, Wpe, 0)
                    ku = 0 if u is None else u.shape[1]
                    W_full = np.zeros((ku + up.shape[1], D))
                    if u is not None:
                        W_full[:ku, case.patch[0]:case.patch[0] + w.shape[1]] = w
                    W_full[ku:, case.rope_offset:case.rope_offset + case.rope_dim] = wp
                    u = up if u is None else np.concatenate([u, up], axis=1)
                    w, poff = W_full, 0
                if case.reloc:
                    want = ref.relocate_k(Kin, u, w, orope, p3, delta[c], poff, case.post_rope)
                else:
                    want = ref.rehydrate_k(Kin, u, w, orope, p3, poff, case.post_rope)
                assert_close(kb[l, dst, h], want, f"K c{c} l{l} h{h}")
                if case.has_v:
                    Vin = ref.bf16_to_f64(V[c, l, :nc, h])
                    u, w = fac(Uv, Wv, 0)
                    assert_close(vb[l, dst, h], ref.rehydrate_v(Vin, u, w, case.patch[0]),
                                 f"V c{c} l{l} h{h}")
    assert np.all(kb[~touched] == SENTINEL), "K rows outside the destination were written"
    if case.has_v:
        assert np.all(vb[~touched] == SENTINEL), "V rows outside the destination were written"
    return kb
