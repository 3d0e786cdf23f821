"""The C-ABI library on the host: it loads, exports every declared symbol, and
rejects bad arguments before any HIP call (no GPU needed for any of this)."""

from __future__ import annotations

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2606_23581_amd as km

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kamera.h")

def _library_available() -> bool:
    try:
        km.lib()            # builds the in-tree library once if it is missing
        return True
    except km.KameraUnavailable:
        return False


pytestmark = pytest.mark.skipif(not _library_available(), reason="libkamera.so not built and cannot be built")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(kamera_[a-z_0-9]+)\s*\(", text, re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ("kamera_rehydrate", "kamera_shift", "kamera_scatter_paged", "kamera_last_error",
                 "kamera_abi_version", "kamera_check_page_table", "kamera_struct_size", "kamera_validate",
                 "kamera_gather_paged", "kamera_form_patch"):
        assert want in names


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", km.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT\s+(kamera_[a-z_0-9]+)$", out, re.M))
    for name in declared_functions():
        assert name in exported, name
    L = km.lib()
    for name in declared_functions():
        assert hasattr(L, name)


def test_plain_c_consumer(tmp_path):
    """tests/c/abi_check.c: a C program built against include/kamera.h and
    linked to libkamera.so checks layouts, validation and the page-table check
    with no GPU (nothing is launched)."""
    exe = tmp_path / "abi_check"
    lib_dir = os.path.dirname(km.LIB_PATH)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "abi_check.c"), "-o", str(exe), "-L", lib_dir, "-lkamera",
                    f"-Wl,-rpath,{lib_dir}"], check=True, capture_output=True, text=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "ok"


def test_version_and_struct_layout():
    L = km.lib()
    assert L.kamera_abi_version() == 4
    assert L.kamera_struct_size(0) == ctypes.sizeof(km.CRehydrateArgs)
    assert L.kamera_struct_size(1) == ctypes.sizeof(km.CShiftArgs)
    assert L.kamera_struct_size(2) == ctypes.sizeof(km.CScatterArgs)
    assert L.kamera_struct_size(3) == ctypes.sizeof(km.CPlane)
    assert L.kamera_struct_size(4) == ctypes.sizeof(km.CRope)
    assert L.kamera_struct_size(5) == ctypes.sizeof(km.CFormArgs)
    assert L.kamera_struct_size(99) == -1


# ---------------------------------------------------------------------------
# validation: fake, never dereferenced device addresses
# ---------------------------------------------------------------------------

FAKE = 0x7F0000000000      # 16-byte aligned, never touched: every case fails before a launch


def rehydrate_args(**over):
    a = km.CRehydrateArgs()
    a.n_chunks, a.n_layers, a.n_heads, a.head_dim, a.n_tokens = 2, 3, 4, 128, 64
    a.rope = km.RopeSpec(theta=1e6, rope_dim=128).to_c()
    a.pos_mode = km.POS_LINEAR
    a.chunk_pos = FAKE + 0x100000000
    a.n_planes = 2
    big = 1 << 32
    for p in range(2):
        pl = a.plane[p]
        pl.in_ = FAKE + (p + 1) * big * 4
        pl.out = FAKE + (p + 3) * big * 4
        strides = [3 * 64 * 4 * 128, 64 * 4 * 128, 4 * 128, 128]
        for k in range(4):
            pl.in_stride[k] = strides[k]
            pl.out_stride[k] = strides[k]
        pl.U = FAKE + (p + 5) * big * 4
        pl.W = FAKE + (p + 7) * big * 4
        us = [3 * 4 * 64 * 16, 4 * 64 * 16, 64 * 16, 16]
        ws = [3 * 4 * 16 * 128, 4 * 16 * 128, 16 * 128, 128]
        for k in range(4):
            pl.u_stride[k] = us[k]
            pl.w_stride[k] = ws[k]
        pl.m = 16
        pl.rotate = 1 if p == 0 else 0
        pl.patch_offset, pl.patch_dim = 0, 128
    for k, v in over.items():
        setattr(a, k, v)
    return a


def call_rehydrate(a):
    return km.lib().kamera_rehydrate(ctypes.byref(a), None)


def test_empty_call_is_a_noop():
    a = rehydrate_args()
    a.n_tokens = 0
    assert call_rehydrate(a) == km.OK
    assert km.last_error() == ""


def _plan_case(case):
    a = rehydrate_args()
    a.kernel = km.KERNEL_ROW_GROUP
    if case == "auto_small":
        a.kernel = km.KERNEL_AUTO
    elif case == "per_head_requested":
        a.kernel = km.KERNEL_PER_HEAD
    elif case == "kernel_choice_unknown":
        a.kernel = 7
    elif case == "row_group4_requested":
        a.kernel = km.KERNEL_ROW_GROUP4
    elif case.startswith("auto_") or case == "row_group_8_heads":
        # chunks x layers of H heads x n tokens, token-major rows
        if case != "row_group_8_heads":
            a.kernel = km.KERNEL_AUTO
        if case == "auto_recall_relocation":
            a.delta = FAKE + 0x300000000
        C, Ln, H, n = {"auto_recall": (64, 80, 8, 1024), "auto_recall_relocation": (64, 80, 8, 1024),
                       "auto_recall_128_token_chunks": (64, 80, 8, 128), "auto_dense_window": (16, 32, 4, 1024),
                       "auto_dense_window_rank_64": (16, 32, 4, 1024),
                       "auto_dense_window_low_end": (8, 32, 4, 1024), "auto_below_dense_window": (8, 32, 4, 1023),
                       "row_group_8_heads": (2, 3, 8, 64), "auto_recall_4_heads": (64, 80, 4, 1024),
                       "auto_recall_short_chunks": (64, 80, 8, 256), "auto_mid_8_heads": (16, 32, 8, 1024),
                       "auto_reorder_shape": (8, 28, 4, 1024), "auto_small_8_heads": (8, 28, 8, 1024),
                       "auto_2_19_rows": (4, 16, 4, 1024), "auto_below_2_19_rows": (4, 16, 4, 1023),
                       "auto_6_heads": (64, 80, 6, 1024)}[case]
        a.n_chunks, a.n_layers, a.n_heads, a.n_tokens = C, Ln, H, n
        for p in range(2):
            strides = [Ln * n * H * 128, n * H * 128, H * 128, 128]
            us = [Ln * H * n * 16, H * n * 16, n * 16, 16]
            ws = [Ln * H * 16 * 128, H * 16 * 128, 16 * 128, 128]
            for k in range(4):
                a.plane[p].in_stride[k] = a.plane[p].out_stride[k] = strides[k]
                a.plane[p].u_stride[k], a.plane[p].w_stride[k] = us[k], ws[k]
        if case == "auto_dense_window_rank_64":
            for p in range(2):
                a.plane[p].m = 64
                a.plane[p].u_stride[0], a.plane[p].u_stride[1] = Ln * H * n * 64, H * n * 64
                a.plane[p].u_stride[2], a.plane[p].u_stride[3] = n * 64, 64
                a.plane[p].w_stride[0], a.plane[p].w_stride[1] = Ln * H * 64 * 128, H * 64 * 128
                a.plane[p].w_stride[2] = 64 * 128
    elif case == "heads_9":
        a.n_heads = 9
    elif case == "rank_72":
        for p in range(2):
            a.plane[p].m = 72
            a.plane[p].u_stride[2], a.plane[p].u_stride[3] = 64 * 72, 72
    elif case == "rank_12":
        a.plane[0].m = 12
    elif case == "explicit":
        a.pos_mode = km.POS_EXPLICIT
        a.explicit_pos = FAKE + 0x200000000
    elif case == "relocation":
        a.delta = FAKE + 0x300000000
    elif case == "head_dim_256":
        a.head_dim = 256
        a.rope = km.RopeSpec(theta=1e6, rope_dim=128, rope_offset=128).to_c()
    elif case == "partial_band":
        a.rope = km.RopeSpec(theta=1e6, rope_dim=64, rope_offset=64).to_c()
    elif case == "patch_64":
        a.plane[0].patch_offset, a.plane[0].patch_dim = 32, 64
    elif case == "offsets_past_2g":
        for p in range(2):
            a.plane[p].in_stride[2] = 1 << 26
    elif case == "empty":
        a.n_tokens = 0
    elif case == "invalid":
        a.plane[0].m = -1
    return a


@pytest.mark.parametrize("case,plan", [
    ("default", km.PLAN_ROW_GROUP4),
    ("row_group_8_heads", km.PLAN_ROW_GROUP),
    ("auto_small", km.PLAN_PER_HEAD),
    ("per_head_requested", km.PLAN_PER_HEAD),
    ("kernel_choice_unknown", km.ERR_SHAPE),
    ("row_group4_requested", km.PLAN_ROW_GROUP4),
    ("auto_recall", km.PLAN_ROW_GROUP4),
    ("auto_recall_4_heads", km.PLAN_ROW_GROUP4),
    ("auto_recall_short_chunks", km.PLAN_ROW_GROUP4),
    ("auto_recall_128_token_chunks", km.PLAN_PER_HEAD),
    ("auto_dense_window", km.PLAN_PER_HEAD),
    ("auto_dense_window_rank_64", km.PLAN_ROW_GROUP4),
    ("auto_dense_window_low_end", km.PLAN_PER_HEAD),
    ("auto_below_dense_window", km.PLAN_ROW_GROUP4),
    ("auto_recall_relocation", km.PLAN_ROW_GROUP4),
    ("auto_mid_8_heads", km.PLAN_ROW_GROUP4),
    ("auto_reorder_shape", km.PLAN_ROW_GROUP4),
    ("auto_small_8_heads", km.PLAN_PER_HEAD),
    ("auto_2_19_rows", km.PLAN_ROW_GROUP4),
    ("auto_below_2_19_rows", km.PLAN_PER_HEAD),
    ("auto_6_heads", km.PLAN_PER_HEAD),
    ("heads_9", km.PLAN_PER_HEAD),
    ("rank_72", km.PLAN_PER_HEAD),
    ("rank_12", km.PLAN_PER_HEAD),
    ("explicit", km.PLAN_PER_HEAD),
    ("relocation", km.PLAN_ROW_GROUP4),
    ("head_dim_256", km.PLAN_PER_HEAD),
    ("partial_band", km.PLAN_PER_HEAD),
    ("patch_64", km.PLAN_PER_HEAD),
    ("offsets_past_2g", km.PLAN_PER_HEAD),
    ("empty", km.PLAN_NONE),
    ("invalid", km.ERR_RANGE),
])
def test_rehydrate_plan_picks_the_kernel(case, plan):
    """kamera_rehydrate_plan runs the call's host checks and names the kernel:
    the row-group kernel, when requested, only for rows of <= 8 heads x 128
    columns with one block per head, rank <= 64 in whole 16-byte U chunks, no
    explicit positions, and every byte offset below 2^31, with 8 heads per
    workgroup for wider rows and 4 for rows of <= 4 heads; AUTO takes it, with
    4 heads per workgroup, for rows of 4 or 8 heads, chunks of >= 256 tokens
    and >= 2^19 rows (planes x chunks x layers x tokens x heads), except dense
    outputs at rank <= 32 with 2^21 to 2^23 rows."""
    a = _plan_case(case)
    assert km.lib().kamera_rehydrate_plan(ctypes.byref(a)) == plan
    assert km.lib().kamera_validate(0, ctypes.byref(a)) == min(plan, 0)


@pytest.mark.parametrize("case,schedule,cap,want", [
    # 64 x 80 units x 2 planes x 2 head groups: 20480 blocks of 1024 tokens
    ("auto_recall", km.SCHEDULE_AUTO, 0, km.SCHEDULE_BLOCKS),
    ("auto_recall_relocation", km.SCHEDULE_AUTO, 0, km.SCHEDULE_BLOCKS),
    ("auto_recall_short_chunks", km.SCHEDULE_AUTO, 0, km.SCHEDULE_BLOCKS),
    # 2048 unit lanes: blocks of 512 tokens reach 4096
    ("auto_mid_8_heads", km.SCHEDULE_AUTO, 0, km.SCHEDULE_BLOCKS),
    # 448 unit lanes: blocks would shrink to 64 tokens
    ("auto_reorder_shape", km.SCHEDULE_AUTO, 0, km.SCHEDULE_PERSISTENT),
    ("auto_2_19_rows", km.SCHEDULE_AUTO, 0, km.SCHEDULE_PERSISTENT),
    ("default", km.SCHEDULE_AUTO, 0, km.SCHEDULE_PERSISTENT),
    # a cap on the workgroups asks for the persistent schedule
    ("auto_recall", km.SCHEDULE_AUTO, 64, km.SCHEDULE_PERSISTENT),
    ("auto_recall", km.SCHEDULE_PERSISTENT, 0, km.SCHEDULE_PERSISTENT),
    ("auto_reorder_shape", km.SCHEDULE_BLOCKS, 0, km.SCHEDULE_BLOCKS),
    ("default", km.SCHEDULE_BLOCKS, 0, km.SCHEDULE_BLOCKS),
    ("auto_recall", km.SCHEDULE_BLOCKS, 8, km.ERR_SHAPE),
    ("auto_recall", 3, 0, km.ERR_SHAPE),
    ("auto_recall", -1, 0, km.ERR_SHAPE),
    # the per-head kernel, or nothing to do: no schedule
    ("auto_small_8_heads", km.SCHEDULE_AUTO, 0, 0),
    ("per_head_requested", km.SCHEDULE_BLOCKS, 0, 0),
    ("empty", km.SCHEDULE_AUTO, 0, 0),
])
def test_rehydrate_schedule_of_the_row_group_kernel(case, schedule, cap, want):
    """kamera_rehydrate_schedule names how the row-group kernel spreads a
    call: AUTO takes one workgroup per token block where the blocks (up to
    1024 tokens, shrunk to >= 64 until the launch has 4096 of them) stay
    >= 512 tokens, else the persistent schedule, which a cap on the
    workgroups also selects; a request for blocks with a cap, or an unknown
    schedule, is rejected by the call's own checks."""
    a = _plan_case(case)
    a.schedule = schedule
    a.max_workgroups = cap
    assert km.lib().kamera_rehydrate_schedule(ctypes.byref(a)) == want
    assert km.lib().kamera_validate(0, ctypes.byref(a)) == min(want, 0)


@pytest.mark.parametrize("layers,code", [(3, km.OK), (4, km.ERR_RANGE)])
def test_row_group_blocks_fit_one_dispatch(layers, code):
    """The block schedule launches one workgroup of 256 threads per token
    block; a dispatch counts its work-items in 32 bits, so 2^21 chunks x 4
    layers x 2 planes of 256-token blocks (2^32 work-items, blocks far below
    2^31) are rejected while 3 layers (3 x 2^30) still launch."""
    a = _plan_case("auto_reorder_shape")
    a.kernel, a.schedule = km.KERNEL_ROW_GROUP4, km.SCHEDULE_BLOCKS
    C, Ln, H, n = 1 << 21, layers, 4, 256
    a.n_chunks, a.n_layers, a.n_heads, a.n_tokens = C, Ln, H, n
    a.chunk_pos = FAKE + (1 << 41)
    for p in range(2):
        strides = [Ln * n * H * 128, n * H * 128, H * 128, 128]
        us = [Ln * H * n * 16, H * n * 16, n * 16, 16]
        ws = [Ln * H * 16 * 128, H * 16 * 128, 16 * 128, 128]
        for k in range(4):
            a.plane[p].in_stride[k] = a.plane[p].out_stride[k] = strides[k]
            a.plane[p].u_stride[k], a.plane[p].w_stride[k] = us[k], ws[k]
        for i, f in enumerate(("in_", "out", "U", "W")):
            setattr(a.plane[p], f, FAKE + (1 + 4 * p + i) * (1 << 42))
    assert km.lib().kamera_validate(0, ctypes.byref(a)) == code, km.last_error()
    if code == km.ERR_RANGE:
        assert "exceed one launch" in km.last_error()
    else:
        assert km.lib().kamera_rehydrate_schedule(ctypes.byref(a)) == km.SCHEDULE_BLOCKS


def _interleaved_case(case):
    """Both planes write one tensor [C][L][n][K|V][H][D] (dense) or a pool
    [L][slot][K|V][H][D] (paged): H = 4, D = 128, so a row of one plane spans
    512 elements and the row stride is 1024."""
    a = rehydrate_args()
    C, Ln, n, H, D = 2, 3, 64, 4, 128
    base = FAKE + 20 * (1 << 34)
    r, d = 2 * H * D, H * D
    if case.startswith("paged"):
        a.paged, a.page_size, a.n_pool_pages, a.pt_stride = 1, 16, 8, 4
        a.page_table = FAKE + 0x400000000
        st = [0, 8 * 16 * r, r, D]
    else:
        st = [Ln * n * r, n * r, r, D]
    outs = [base, base + 2 * d]
    if case == "dense_v_first":
        outs = outs[::-1]
    elif case == "dense_gap_short":
        outs[1] = base + 2 * (d // 2)
    elif case == "dense_gap_long":
        outs[1] = base + 2 * (d + d // 2)
    elif case == "dense_gap_odd_bytes":
        outs[1] = base + 2 * d + 1
    for p in range(2):
        a.plane[p].out = outs[p]
        for k in range(4):
            a.plane[p].out_stride[k] = st[k]
    if case.startswith("dense_in_place"):
        # each plane exactly in place on one tensor [C][L][n][K|V][H][D]
        if case == "dense_in_place_gap_short":
            outs[1] = base + 2 * (d // 2)
        for p in range(2):
            a.plane[p].out = a.plane[p].in_ = outs[p]
            for k in range(4):
                a.plane[p].in_stride[k] = st[k]
    if case == "dense_strides_differ":
        a.plane[1].out_stride[2] = r + D
    elif case == "dense_layer_stride_not_rows":
        for p in range(2):
            a.plane[p].out_stride[1] = n * r + d
            a.plane[p].out_stride[0] = Ln * (n * r + d)
    return a


@pytest.mark.parametrize("case,code", [
    ("dense", km.OK),
    ("dense_v_first", km.OK),
    ("paged", km.OK),
    ("dense_gap_short", km.ERR_ALIAS),
    ("dense_gap_long", km.ERR_ALIAS),
    ("dense_gap_odd_bytes", km.ERR_ALIGN),
    ("dense_strides_differ", km.ERR_ALIAS),
    ("dense_layer_stride_not_rows", km.ERR_ALIAS),
    ("dense_in_place", km.OK),
    ("dense_in_place_gap_short", km.ERR_ALIAS),
])
def test_interleaved_plane_outputs(case, code):
    """The K and V planes may write one tensor with their rows interleaved (the
    rows of one plane in the gaps between the rows of the other), also each
    plane in place on such a tensor; any other overlap is rejected."""
    a = _interleaved_case(case)
    assert km.lib().kamera_validate(0, ctypes.byref(a)) == code, km.last_error()
    if code == km.ERR_ALIAS:
        assert "overlap" in km.last_error()


@pytest.mark.parametrize("case,code", [
    ("null_args", km.ERR_NULL),
    ("negative", km.ERR_SHAPE),
    ("head_dim_not_32", km.ERR_UNSUPPORTED),
    ("head_dim_huge", km.ERR_RANGE),
    ("n_planes_3", km.ERR_SHAPE),
    ("rope_odd", km.ERR_SHAPE),
    ("rope_outside_row", km.ERR_SHAPE),
    ("rope_too_wide", km.ERR_RANGE),
    ("sections_sum", km.ERR_SHAPE),
    ("theta_negative", km.ERR_SHAPE),
    ("neox_32", km.ERR_UNSUPPORTED),
    ("band_unaligned", km.ERR_UNSUPPORTED),
    ("rank_too_big", km.ERR_RANGE),
    ("rank_negative", km.ERR_RANGE),
    ("patch_outside", km.ERR_SHAPE),
    ("patch_unaligned", km.ERR_UNSUPPORTED),
    ("u_null", km.ERR_NULL),
    ("in_null", km.ERR_NULL),
    ("pos_null", km.ERR_NULL),
    ("misaligned_base", km.ERR_ALIGN),
    ("misaligned_stride", km.ERR_ALIGN),
    ("alias", km.ERR_ALIAS),
    ("paged_no_table", km.ERR_NULL),
    ("paged_short_table", km.ERR_SHAPE),
    ("paged_page_size", km.ERR_SHAPE),
    ("grid_w_zero", km.ERR_SHAPE),
    ("bad_pos_mode", km.ERR_SHAPE),
    ("bad_frame", km.ERR_SHAPE),
    ("cols_unaligned", km.ERR_UNSUPPORTED),
    ("cols_empty", km.ERR_SHAPE),
    ("cols_outside_row", km.ERR_SHAPE),
    ("cols_miss_band", km.ERR_SHAPE),
    ("patch_outside_cols", km.ERR_SHAPE),
])
def test_rehydrate_rejects(case, code):
    L = km.lib()
    if case == "null_args":
        assert L.kamera_rehydrate(None, None) == code
        assert "NULL" in km.last_error()
        return
    a = rehydrate_args()
    if case == "negative":
        a.n_layers = -1
    elif case == "head_dim_not_32":
        a.head_dim = 120
    elif case == "head_dim_huge":
        a.head_dim = 8192
    elif case == "n_planes_3":
        a.n_planes = 3
    elif case == "rope_odd":
        a.rope.rope_dim = 127
    elif case == "rope_outside_row":
        a.rope.rope_offset = 64
    elif case == "rope_too_wide":
        a.head_dim = 256
        a.rope.rope_dim = 256
    elif case == "sections_sum":
        a.rope.n_sections = 3
        a.rope.sections[0], a.rope.sections[1], a.rope.sections[2] = 16, 24, 23
    elif case == "theta_negative":
        a.rope.theta = -1.0
    elif case == "neox_32":
        a.rope.rope_dim = 32
    elif case == "band_unaligned":
        a.rope.rope_offset = 16
        a.rope.rope_dim = 64
        a.rope.pairing = km.PAIR_INTERLEAVED
    elif case == "rank_too_big":
        a.plane[0].m = 129
    elif case == "rank_negative":
        a.plane[1].m = -2
    elif case == "patch_outside":
        a.plane[0].patch_offset = 64
    elif case == "patch_unaligned":
        a.plane[0].patch_dim = 100
    elif case == "u_null":
        a.plane[1].U = None
    elif case == "in_null":
        a.plane[0].in_ = None
    elif case == "pos_null":
        a.chunk_pos = None
    elif case == "misaligned_base":
        a.plane[0].out = a.plane[0].out + 2
    elif case == "misaligned_stride":
        a.plane[1].in_stride[2] = 4 * 128 + 4
    elif case == "alias":
        a.plane[1].out = a.plane[0].in_ + 4096
    elif case == "paged_no_table":
        a.paged = 1
        a.page_size, a.n_pool_pages, a.pt_stride = 16, 64, 4
    elif case == "paged_short_table":
        a.paged = 1
        a.page_table = FAKE + (9 << 36)
        a.page_size, a.n_pool_pages, a.pt_stride = 16, 64, 3
    elif case == "paged_page_size":
        a.paged = 1
        a.page_table = FAKE + (9 << 36)
        a.page_size, a.n_pool_pages, a.pt_stride = 0, 64, 4
    elif case == "grid_w_zero":
        a.pos_mode = km.POS_GRID3
        a.grid_w = 0
    elif case == "bad_pos_mode":
        a.pos_mode = 7
    elif case == "bad_frame":
        a.patch_frame = 5
    elif case == "cols_unaligned":
        a.plane[1].col_begin, a.plane[1].col_end = 16, 128
    elif case == "cols_empty":
        a.plane[1].col_begin, a.plane[1].col_end = 64, 64
    elif case == "cols_outside_row":
        a.plane[1].col_begin, a.plane[1].col_end = 0, 160
    elif case == "cols_miss_band":
        a.plane[0].col_begin, a.plane[0].col_end = 0, 64
    elif case == "patch_outside_cols":
        a.plane[1].col_begin, a.plane[1].col_end = 64, 128
    assert call_rehydrate(a) == code, km.last_error()
    assert km.last_error().startswith("kamera_rehydrate")


def test_plane_outputs_may_share_a_tensor_only_on_disjoint_columns():
    """Two planes writing one output tensor: accepted through the same mapping on
    disjoint column ranges (the MLA latent and its rope band), rejected when the
    ranges intersect or the mappings differ."""
    L = km.lib()

    def two_planes(c0, c1, shift=0):
        a = rehydrate_args()
        a.head_dim = 256
        a.rope = km.RopeSpec(theta=1e6, rope_dim=64, rope_offset=192).to_c()
        for p in range(2):
            pl = a.plane[p]
            st = [3 * 64 * 4 * 256, 64 * 4 * 256, 4 * 256, 256]
            for k in range(4):
                pl.in_stride[k] = st[k]
                pl.out_stride[k] = st[k]
            pl.m = 16
            pl.rotate = 1 if p == 1 else 0
        a.plane[1].in_ = a.plane[0].in_
        a.plane[1].out = a.plane[0].out + shift
        (a.plane[0].col_begin, a.plane[0].col_end), (a.plane[1].col_begin, a.plane[1].col_end) = c0, c1
        a.plane[0].patch_offset, a.plane[0].patch_dim = c0[0], c0[1] - c0[0]
        a.plane[1].patch_offset, a.plane[1].patch_dim = c1[0], c1[1] - c1[0]
        return a

    assert L.kamera_validate(0, ctypes.byref(two_planes((0, 192), (192, 256)))) == km.OK, km.last_error()
    assert L.kamera_validate(0, ctypes.byref(two_planes((0, 224), (192, 256)))) == km.ERR_ALIAS
    assert L.kamera_validate(0, ctypes.byref(two_planes((0, 192), (192, 256), shift=512))) == km.ERR_ALIAS


def test_exact_in_place_is_accepted_but_shifted_overlap_is_not():
    """In place (same base and strides, dense, no row base) passes validation;
    any other overlap is rejected.  The in-place case is stopped right before
    the launch by an empty token count, so nothing runs."""
    L = km.lib()
    a = rehydrate_args()
    assert L.kamera_validate(0, ctypes.byref(a)) == km.OK
    for p in range(2):
        a.plane[p].out = a.plane[p].in_
    assert L.kamera_validate(0, ctypes.byref(a)) == km.OK, km.last_error()
    a = rehydrate_args()
    a.plane[0].out = a.plane[0].in_ + 256
    assert L.kamera_validate(0, ctypes.byref(a)) == km.ERR_ALIAS
    # two planes in place on one tensor: only with disjoint columns
    a = rehydrate_args()
    a.plane[1].in_ = a.plane[0].in_
    a.plane[0].out = a.plane[1].out = a.plane[0].in_
    assert L.kamera_validate(0, ctypes.byref(a)) == km.ERR_ALIAS
    a.head_dim = 256
    a.plane[0].col_begin, a.plane[0].col_end = 0, 128
    a.plane[1].col_begin, a.plane[1].col_end = 128, 256
    a.plane[1].patch_offset = 128
    for p in range(2):
        a.plane[p].in_stride[3] = a.plane[p].out_stride[3] = 256
        a.plane[p].in_stride[2] = a.plane[p].out_stride[2] = 4 * 256
    assert L.kamera_validate(0, ctypes.byref(a)) == km.OK, km.last_error()
    assert L.kamera_validate(7, ctypes.byref(a)) == km.ERR_SHAPE


def test_error_text_is_per_thread():
    import threading

    a = rehydrate_args()
    a.head_dim = 120
    assert call_rehydrate(a) == km.ERR_UNSUPPORTED
    seen = {}

    def other():
        seen["text"] = km.last_error()

    th = threading.Thread(target=other)
    th.start()
    th.join()
    assert seen["text"] == ""
    assert "head_dim" in km.last_error()


def shift_args():
    a = km.CShiftArgs()
    a.n_chunks, a.n_layers, a.n_heads, a.head_dim, a.n_tokens = 3, 2, 4, 128, 32
    a.rope = km.RopeSpec(theta=1e4, rope_dim=128, pairing="interleaved").to_c()
    a.delta = FAKE
    a.k = FAKE + (1 << 36)
    for k, s in enumerate([2 * 32 * 4 * 128, 32 * 4 * 128, 4 * 128, 128]):
        a.k_stride[k] = s
    return a


@pytest.mark.parametrize("case,code", [
    ("k_null", km.ERR_NULL), ("delta_null", km.ERR_NULL), ("rope_dim_12_neox", km.ERR_UNSUPPORTED),
    ("offset_4", km.ERR_UNSUPPORTED), ("misaligned", km.ERR_ALIGN), ("band_outside", km.ERR_SHAPE),
    ("paged_no_table", km.ERR_NULL),
])
def test_shift_rejects(case, code):
    a = shift_args()
    if case == "k_null":
        a.k = None
    elif case == "delta_null":
        a.delta = None
    elif case == "rope_dim_12_neox":
        a.rope.pairing = km.PAIR_NEOX
        a.rope.rope_dim = 24
    elif case == "offset_4":
        a.rope.rope_offset = 4
        a.rope.rope_dim = 64
    elif case == "misaligned":
        a.k_stride[3] = 132
    elif case == "band_outside":
        a.rope.rope_offset = 8
    elif case == "paged_no_table":
        a.paged = 1
        a.page_size, a.pt_stride, a.n_pool_pages = 16, 2, 8
    assert km.lib().kamera_shift(ctypes.byref(a), None) == code, km.last_error()


def test_shift_empty_ok():
    a = shift_args()
    a.n_chunks = 0
    a.k = None
    assert km.lib().kamera_shift(ctypes.byref(a), None) == km.OK


def scatter_args():
    a = km.CScatterArgs()
    a.n_chunks, a.n_layers, a.n_tokens = 2, 3, 40
    a.row_bytes = 2048
    a.rows = FAKE
    a.rows_stride_bytes[0], a.rows_stride_bytes[1], a.rows_stride_bytes[2] = 3 * 40 * 2048, 40 * 2048, 2048
    a.pool = FAKE + (1 << 36)
    a.pool_stride_bytes[0], a.pool_stride_bytes[1] = 64 * 16 * 2048, 2048
    a.page_table = FAKE + (2 << 36)
    a.pt_stride, a.page_size, a.n_pool_pages = 3, 16, 64
    return a


@pytest.mark.parametrize("case,code", [
    ("row_bytes", km.ERR_ALIGN), ("rows_null", km.ERR_NULL), ("table_null", km.ERR_NULL),
    ("short_table", km.ERR_SHAPE), ("stride", km.ERR_ALIGN), ("alias", km.ERR_ALIAS),
])
def test_scatter_rejects(case, code):
    a = scatter_args()
    if case == "row_bytes":
        a.row_bytes = 2040
    elif case == "rows_null":
        a.rows = None
    elif case == "table_null":
        a.page_table = None
    elif case == "short_table":
        a.pt_stride = 2
    elif case == "stride":
        a.rows_stride_bytes[2] = 2056
    elif case == "alias":
        a.pool = a.rows + 4096
    assert km.lib().kamera_scatter_paged(ctypes.byref(a), None) == code, km.last_error()
    assert km.lib().kamera_gather_paged(ctypes.byref(a), None) == code, km.last_error()
    assert km.last_error().startswith("kamera_gather_paged")
    assert km.lib().kamera_validate(3, ctypes.byref(a)) == code


def test_check_page_table():
    pt = np.arange(12, dtype=np.int32).reshape(3, 4)
    km.check_page_table(pt, n_tokens=64, page_size=16, n_pool_pages=12)
    bad = pt.copy()
    bad[2, 1] = 3
    with pytest.raises(km.KameraError) as e:
        km.check_page_table(bad, n_tokens=64, page_size=16, n_pool_pages=12)
    assert e.value.code == km.ERR_ALIAS
    bad = pt.copy()
    bad[1, 0] = 12
    with pytest.raises(km.KameraError) as e:
        km.check_page_table(bad, n_tokens=64, page_size=16, n_pool_pages=12)
    assert e.value.code == km.ERR_RANGE
    # only the pages the tokens use are checked: 40 tokens need 3 of the 4
    tail = pt.copy()
    tail[:, 3] = -1
    km.check_page_table(tail, n_tokens=40, page_size=16, n_pool_pages=12)


def test_product_path_has_no_fallback(monkeypatch):
    """Without the library every entry point raises; nothing runs on the CPU."""
    monkeypatch.setattr(km, "_LIB", None)
    monkeypatch.setattr(km, "LIB_PATH", km.LIB_PATH + ".missing")
    with pytest.raises(km.KameraUnavailable):
        km.lib()
    with pytest.raises(km.KameraUnavailable):
        km.check_page_table(np.zeros((1, 1), np.int32), 16, 16, 1)


def test_product_package_does_not_import_the_oracle():
    pkg = os.path.join(ROOT, "paper_2606_23581_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text.replace("oracles", ""), f


def form_args():
    a = km.CFormArgs()
    a.n_chunks, a.n_layers, a.n_heads, a.n_tokens, a.dim, a.m = 2, 3, 4, 100, 128, 16
    a.delta = FAKE
    for k, st in enumerate([3 * 4 * 100 * 128, 4 * 100 * 128, 100 * 128, 128]):
        a.delta_stride[k] = st
    a.U = FAKE + (1 << 36)
    a.W = FAKE + (2 << 36)
    return a


@pytest.mark.parametrize("case,code", [
    ("ok", km.OK), ("dim_not_4", km.ERR_UNSUPPORTED), ("dim_big", km.ERR_RANGE), ("m_zero", km.ERR_RANGE),
    ("m_big", km.ERR_RANGE), ("null", km.ERR_NULL), ("unaligned", km.ERR_ALIGN), ("stride", km.ERR_ALIGN),
    ("sweeps", km.ERR_SHAPE), ("negative", km.ERR_SHAPE), ("orbit_negative", km.ERR_SHAPE),
    ("orbit_stride", km.ERR_ALIGN), ("orbit_ok", km.OK), ("u_over_delta", km.ERR_ALIAS),
    ("w_over_orbit", km.ERR_ALIAS), ("sigma_over_delta", km.ERR_ALIAS), ("sigma_apart", km.OK),
    ("done_over_delta", km.ERR_ALIAS), ("u_over_w", km.ERR_ALIAS), ("too_many_units", km.ERR_RANGE),
    ("too_many_rows", km.ERR_RANGE),
])
def test_form_patch_validation(case, code):
    a = form_args()
    if case == "dim_not_4":
        a.dim = 126
    elif case == "dim_big":
        a.dim = 256
    elif case == "m_zero":
        a.m = 0
    elif case == "m_big":
        a.m = 129
    elif case == "null":
        a.W = None
    elif case == "unaligned":
        a.delta = FAKE + 4
    elif case == "stride":
        a.delta_stride[3] = 130
    elif case == "sweeps":
        a.sweeps = -1
    elif case == "negative":
        a.n_tokens = -5
    elif case == "orbit_negative":
        a.n_orbit = -1
    elif case == "orbit_stride":
        a.n_orbit, a.orbit_stride = 3, 2 * 3 * 4 * 100 * 128 + 2
    elif case == "orbit_ok":
        a.n_orbit, a.orbit_stride = 3, 2 * 3 * 4 * 100 * 128
    elif case == "u_over_delta":
        a.U = FAKE + 4 * 1000
    elif case == "w_over_orbit":
        # W sits in the second orbit member's deficit
        a.n_orbit, a.orbit_stride = 2, 2 * 3 * 4 * 100 * 128
        a.W = FAKE + 4 * (2 * 3 * 4 * 100 * 128 + 64)
    elif case == "sigma_over_delta":
        a.sigma = FAKE + 4 * 128
    elif case == "sigma_apart":
        a.sigma = FAKE + (3 << 36)
    elif case == "done_over_delta":
        a.sweeps_done = FAKE + 4 * 256
    elif case == "u_over_w":
        # U is formed from the stored W, so the two may not share memory
        a.U = a.W + 8
    elif case == "too_many_units":
        # 2^22 + 1 units of 1024 work-items: more than a dispatch counts
        a.n_chunks, a.n_layers, a.n_heads = 4097, 32, 32
    elif case == "too_many_rows":
        # 2^16 units of 2^16 tokens: 2^32 work-items of the U kernel
        a.n_chunks, a.n_layers, a.n_heads, a.n_tokens = 64, 32, 32, 1 << 16
    assert km.lib().kamera_validate(4, ctypes.byref(a)) == code, km.last_error()
    if code != km.OK:
        assert km.lib().kamera_form_patch(ctypes.byref(a), None) == code
