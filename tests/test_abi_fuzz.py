"""Randomised argument structs against the host-side validation (CPU only:
kamera_validate never launches and never touches device memory).  Each case
starts from a valid call and overwrites up to three fields with arbitrary
values.  Whatever the fields hold, validation returns one of the documented
codes, sets the error text exactly when it rejects, and accepts only structs
whose rows are 16-byte aligned and whose sizes lie in the documented ranges;
an untouched valid call is always accepted."""

from __future__ import annotations

import ctypes

import pytest

import paper_2606_23581_amd as km

pytest.importorskip("hypothesis")
from hypothesis import given, settings  # noqa: E402
from hypothesis import strategies as st  # noqa: E402

CODES = {km.OK, km.ERR_NULL, km.ERR_SHAPE, km.ERR_ALIGN, km.ERR_RANGE, km.ERR_ALIAS, km.ERR_UNSUPPORTED}
BASE = 0x7E0000000000        # 16-byte aligned, never dereferenced
GB = 1 << 36


def _library():
    try:
        return km.lib()
    except km.KameraUnavailable:
        pytest.skip("libkamera.so not built and cannot be built")


def valid_rehydrate():
    a = km.CRehydrateArgs()
    a.n_chunks, a.n_layers, a.n_heads, a.head_dim, a.n_tokens = 2, 3, 4, 128, 64
    a.rope = km.RopeSpec(theta=1e6, rope_dim=128).to_c()
    a.pos_mode = km.POS_LINEAR
    a.chunk_pos = BASE
    a.n_planes = 2
    st_ = [3 * 64 * 4 * 128, 64 * 4 * 128, 4 * 128, 128]
    for p in range(2):
        pl = a.plane[p]
        pl.in_, pl.out, pl.U, pl.W = BASE + (1 + p) * GB, BASE + (3 + p) * GB, BASE + (5 + p) * GB, BASE + (7 + p) * GB
        for k in range(4):
            pl.in_stride[k] = st_[k]
            pl.out_stride[k] = st_[k]
        for k, v in enumerate([3 * 4 * 64 * 16, 4 * 64 * 16, 64 * 16, 16]):
            pl.u_stride[k] = v
        for k, v in enumerate([3 * 4 * 16 * 128, 4 * 16 * 128, 16 * 128, 128]):
            pl.w_stride[k] = v
        pl.m, pl.rotate, pl.patch_offset, pl.patch_dim = 16, 1 - p, 0, 128
    return a


anyint = st.one_of(st.integers(-3, 3), st.sampled_from([8, 16, 30, 32, 64, 100, 127, 128, 129, 512, 576, 4096, 5000,
                                                       1 << 20, -(1 << 20), 2 ** 31 - 1, -2 ** 31]))
anyaddr = st.one_of(st.just(0), st.integers(0, 4096).map(lambda k: BASE + k * GB // 8),
                    st.integers(0, 64).map(lambda k: BASE + GB + 2 * k))
REH_FIELDS = ["n_chunks", "n_layers", "n_heads", "head_dim", "n_tokens", "patch_frame", "pos_mode", "grid_w",
              "explicit_chunk_stride", "n_planes", "paged", "pt_stride", "page_size", "n_pool_pages",
              "rope.rope_dim", "rope.rope_offset", "rope.pairing", "rope.n_sections", "rope.section_order",
              "p0.m", "p0.rotate", "p0.patch_offset", "p0.patch_dim", "p0.col_begin", "p0.col_end",
              "p1.m", "p1.rotate", "p1.col_begin", "p1.col_end", "p0.in_stride.2", "p1.out_stride.1",
              "p0.in_", "p0.out", "p1.in_", "p1.out", "p0.U", "p1.W", "chunk_pos", "page_table", "kernel"]


def _set(a, field, value):
    parts = field.split(".")
    obj = a
    if parts[0] in ("p0", "p1"):
        obj = a.plane[int(parts[0][1])]
        parts = parts[1:]
    elif parts[0] == "rope":
        obj = a.rope
        parts = parts[1:]
    if len(parts) == 2:
        getattr(obj, parts[0])[int(parts[1])] = value
        return
    name = parts[0]
    if name in ("in_", "out", "U", "W", "chunk_pos", "page_table"):
        setattr(obj, name, value or None)
    else:
        setattr(obj, name, int(value))


@settings(max_examples=500, deadline=None)
@given(edits=st.lists(st.tuples(st.sampled_from(REH_FIELDS), anyint, anyaddr), max_size=3))
def test_rehydrate_validation_never_misbehaves(edits):
    L = _library()
    a = valid_rehydrate()
    for field, v, p in edits:
        is_ptr = field.split(".")[-1] in ("in_", "out", "U", "W", "chunk_pos", "page_table")
        _set(a, field, p if is_ptr else v)
    rc = L.kamera_validate(0, ctypes.byref(a))
    assert rc in CODES
    assert (km.last_error() == "") == (rc == km.OK), (rc, km.last_error())
    # the plan agrees with validation: an error code, or a kernel (none for an empty call)
    plan = L.kamera_rehydrate_plan(ctypes.byref(a))
    assert plan == rc if rc != km.OK else plan in (km.PLAN_NONE, km.PLAN_PER_HEAD, km.PLAN_ROW_GROUP, km.PLAN_ROW_GROUP4)
    if rc == km.OK:
        assert a.kernel in (km.KERNEL_AUTO, km.KERNEL_PER_HEAD, km.KERNEL_ROW_GROUP, km.KERNEL_ROW_GROUP4)
    if not edits:
        assert rc == km.OK
    if rc == km.OK and min(a.n_chunks, a.n_layers, a.n_heads, a.n_tokens) > 0:
        assert 0 < a.head_dim <= 4096 and a.head_dim % 32 == 0
        assert a.n_planes in (1, 2)
        for p in range(a.n_planes):
            pl = a.plane[p]
            assert pl.in_ % 16 == 0 and pl.out % 16 == 0
            assert all(pl.in_stride[k] % 8 == 0 and pl.out_stride[k] % 8 == 0 for k in range(4))
            assert 0 <= pl.m <= 128
            if pl.m > 0:
                assert pl.U is not None and pl.W is not None


FORM_FIELDS = ["n_chunks", "n_layers", "n_heads", "n_tokens", "dim", "m", "sweeps", "n_orbit", "delta_stride.3",
               "orbit_stride", "delta", "U", "W", "sigma"]


def valid_form():
    a = km.CFormArgs()
    a.n_chunks, a.n_layers, a.n_heads, a.n_tokens, a.dim, a.m = 2, 3, 4, 100, 128, 16
    a.delta = BASE
    for k, v in enumerate([3 * 4 * 100 * 128, 4 * 100 * 128, 100 * 128, 128]):
        a.delta_stride[k] = v
    a.U, a.W = BASE + GB, BASE + 2 * GB
    return a


@settings(max_examples=300, deadline=None)
@given(edits=st.lists(st.tuples(st.sampled_from(FORM_FIELDS), anyint, anyaddr), max_size=3))
def test_form_validation_never_misbehaves(edits):
    L = _library()
    a = valid_form()
    for field, v, p in edits:
        if field in ("delta", "U", "W", "sigma"):
            setattr(a, field, p or None)
        elif field == "delta_stride.3":
            a.delta_stride[3] = v
        else:
            setattr(a, field, int(v))
    rc = L.kamera_validate(4, ctypes.byref(a))
    assert rc in CODES
    assert (km.last_error() == "") == (rc == km.OK)
    if not edits:
        assert rc == km.OK
    if rc == km.OK and min(a.n_chunks, a.n_layers, a.n_heads, a.n_tokens) > 0:
        assert 0 < a.dim <= 128 and a.dim % 4 == 0 and 1 <= a.m <= a.dim
        assert a.delta % 16 == 0 and a.delta_stride[3] % 4 == 0
