"""Kamera chunk-reuse operator on AMD Instinct MI355X (gfx950).

Thin ctypes binding over ``libkamera.so`` (declared in ``include/kamera.h``).
Every step of the operator runs in the library's HIP kernels; this module only
turns torch tensors (device memory, strides) and the current HIP stream into
the C argument structs.  There is no fallback: if the library is not built,
importing works but every call raises ``KameraUnavailable``.

Entry points (same names as the C ABI):

* ``rehydrate``     K' = R(pos)(K + U_k W_k), V' = V + U_v W_v
                    (Eq. ``eq:operator``, Sec. 3; App. A serve step)
* ``shift``         K' = R(delta) K in place (Sec. 1, Sec. 5 survivors)
* ``scatter_paged`` bit copy of dense token rows into page-table slots
                    (App. E clean-view overwrite, Sec. 6 paged pool)
* ``gather_paged``  the inverse copy, pool slots back into dense rows
* ``form_patch``    the compile step's truncated SVD of given deficits
                    (App. A): U = U_svd S [:, :m], W = Vt[:m]
"""

from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional, Sequence, Tuple

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libkamera.so")
_DEFAULT_LIB_PATH = LIB_PATH

OK = 0
ERR_NULL = -1
ERR_SHAPE = -2
ERR_ALIGN = -3
ERR_RANGE = -4
ERR_ALIAS = -5
ERR_UNSUPPORTED = -6
ERR_HIP = -7
STATUS_BAD_PAGE = 1
MAX_RANK = 128

PAIR_NEOX = 0
PAIR_INTERLEAVED = 1
SECTIONS_BLOCKED = 0
SECTIONS_INTERLEAVED = 1
POS_LINEAR = 0
POS_GRID3 = 1
POS_EXPLICIT = 2
PATCH_PRE_ROPE = 0
PATCH_POST_ROPE = 1
KERNEL_AUTO = 0
KERNEL_PER_HEAD = 1
KERNEL_ROW_GROUP = 2
KERNEL_ROW_GROUP4 = 3
PLAN_NONE = 0
PLAN_PER_HEAD = 1
PLAN_ROW_GROUP = 2
PLAN_ROW_GROUP4 = 3
SCHEDULE_AUTO = 0
SCHEDULE_PERSISTENT = 1
SCHEDULE_BLOCKS = 2


class KameraUnavailable(RuntimeError):
    """libkamera.so is missing or cannot be loaded."""


class KameraError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"[{code}] {message}")
        self.code = code
        self.message = message


# ---------------------------------------------------------------------------
# C structs (must match include/kamera.h; checked against kamera_struct_size)
# ---------------------------------------------------------------------------

_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_vp = ctypes.c_void_p


class CRope(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_double), ("rope_offset", _i32), ("rope_dim", _i32),
                ("pairing", _i32), ("n_sections", _i32), ("sections", _i32 * 3),
                ("section_order", _i32)]


class CPlane(ctypes.Structure):
    _fields_ = [("in_", _vp), ("in_stride", _i64 * 4), ("out", _vp), ("out_stride", _i64 * 4),
                ("U", _vp), ("u_stride", _i64 * 4), ("W", _vp), ("w_stride", _i64 * 4),
                ("m", _i32), ("rotate", _i32), ("patch_offset", _i32), ("patch_dim", _i32),
                ("col_begin", _i32), ("col_end", _i32), ("layer_rank", _vp)]


class CRehydrateArgs(ctypes.Structure):
    _fields_ = [("n_chunks", _i32), ("n_layers", _i32), ("n_heads", _i32), ("head_dim", _i32),
                ("n_tokens", _i32), ("chunk_tokens", _vp), ("patch_frame", _i32), ("rope", CRope),
                ("pos_mode", _i32), ("chunk_pos", _vp), ("grid_w", _i32), ("explicit_pos", _vp),
                ("explicit_chunk_stride", _i64), ("n_planes", _i32), ("plane", CPlane * 2),
                ("paged", _i32), ("row_base", _vp), ("page_table", _vp), ("pt_stride", _i32),
                ("page_size", _i32), ("n_pool_pages", _i32), ("status", _vp), ("delta", _vp),
                ("kernel", _i32), ("max_workgroups", _i32), ("schedule", _i32)]


class CShiftArgs(ctypes.Structure):
    _fields_ = [("n_chunks", _i32), ("n_layers", _i32), ("n_heads", _i32), ("head_dim", _i32),
                ("n_tokens", _i32), ("chunk_tokens", _vp), ("rope", CRope), ("delta", _vp),
                ("k", _vp), ("k_stride", _i64 * 4), ("paged", _i32), ("row_base", _vp),
                ("page_table", _vp), ("pt_stride", _i32), ("page_size", _i32),
                ("n_pool_pages", _i32), ("status", _vp)]


class CScatterArgs(ctypes.Structure):
    _fields_ = [("n_chunks", _i32), ("n_layers", _i32), ("n_tokens", _i32), ("chunk_tokens", _vp),
                ("row_bytes", _i64), ("rows", _vp), ("rows_stride_bytes", _i64 * 3), ("pool", _vp),
                ("pool_stride_bytes", _i64 * 2), ("page_table", _vp), ("pt_stride", _i32),
                ("page_size", _i32), ("n_pool_pages", _i32), ("status", _vp)]


class CFormArgs(ctypes.Structure):
    _fields_ = [("n_chunks", _i32), ("n_layers", _i32), ("n_heads", _i32), ("n_tokens", _i32),
                ("dim", _i32), ("m", _i32), ("sweeps", _i32), ("n_orbit", _i32),
                ("delta", _vp), ("delta_stride", _i64 * 4), ("U", _vp), ("u_stride", _i64 * 4),
                ("W", _vp), ("w_stride", _i64 * 4), ("sigma", _vp), ("sigma_stride", _i64 * 3),
                ("orbit_stride", _i64), ("sweeps_done", _vp)]


EXPORTS = ("kamera_rehydrate", "kamera_shift", "kamera_scatter_paged", "kamera_gather_paged",
           "kamera_form_patch",
           "kamera_check_page_table",
           "kamera_validate", "kamera_rehydrate_plan", "kamera_rehydrate_schedule", "kamera_last_error",
           "kamera_abi_version",
           "kamera_struct_size")

_LIB = None


def lib() -> ctypes.CDLL:
    """The loaded library.  When the in-tree library has not been built yet it
    is compiled once (hipcc, gfx950); if that is impossible, or another path
    was configured and is missing, KameraUnavailable is raised -- there is no
    other implementation to fall back to."""
    global _LIB
    if _LIB is not None:
        return _LIB
    # torch ships its own HIP runtime: load it first so that the library binds
    # to the same runtime instance torch's tensors and streams live in
    import torch  # noqa: F401

    if not os.path.exists(LIB_PATH) and LIB_PATH == _DEFAULT_LIB_PATH:
        try:
            from . import build as _build

            _build.build()
        except Exception as e:  # no hipcc, or the compile failed
            raise KameraUnavailable(f"{LIB_PATH} is not built and building it failed: {e}") from e
    if not os.path.exists(LIB_PATH):
        raise KameraUnavailable(f"{LIB_PATH} is not built (run __graft_entry__.build())")
    try:
        L = ctypes.CDLL(LIB_PATH)
    except OSError as e:  # pragma: no cover - depends on the ROCm install
        raise KameraUnavailable(f"cannot load {LIB_PATH}: {e}") from e
    L.kamera_rehydrate.argtypes = [ctypes.POINTER(CRehydrateArgs), _vp]
    L.kamera_rehydrate.restype = _i32
    L.kamera_shift.argtypes = [ctypes.POINTER(CShiftArgs), _vp]
    L.kamera_shift.restype = _i32
    L.kamera_scatter_paged.argtypes = [ctypes.POINTER(CScatterArgs), _vp]
    L.kamera_scatter_paged.restype = _i32
    L.kamera_gather_paged.argtypes = [ctypes.POINTER(CScatterArgs), _vp]
    L.kamera_gather_paged.restype = _i32
    L.kamera_check_page_table.argtypes = [_vp, _i32, _i32, _i32, _i32, _i32]
    L.kamera_check_page_table.restype = _i32
    L.kamera_last_error.argtypes = []
    L.kamera_last_error.restype = ctypes.c_char_p
    L.kamera_abi_version.argtypes = []
    L.kamera_abi_version.restype = _i32
    L.kamera_form_patch.argtypes = [ctypes.POINTER(CFormArgs), _vp]
    L.kamera_form_patch.restype = _i32
    L.kamera_validate.argtypes = [_i32, _vp]
    L.kamera_validate.restype = _i32
    L.kamera_rehydrate_plan.argtypes = [ctypes.POINTER(CRehydrateArgs)]
    L.kamera_rehydrate_plan.restype = _i32
    L.kamera_rehydrate_schedule.argtypes = [ctypes.POINTER(CRehydrateArgs)]
    L.kamera_rehydrate_schedule.restype = _i32
    L.kamera_struct_size.argtypes = [_i32]
    L.kamera_struct_size.restype = _i64
    sizes = {0: CRehydrateArgs, 1: CShiftArgs, 2: CScatterArgs, 3: CPlane, 4: CRope, 5: CFormArgs}
    for k, cls in sizes.items():
        if L.kamera_struct_size(k) != ctypes.sizeof(cls):
            raise KameraUnavailable(f"struct layout mismatch for {cls.__name__}: "
                                    f"C {L.kamera_struct_size(k)} vs ctypes {ctypes.sizeof(cls)}")
    _LIB = L
    return L


def last_error() -> str:
    return lib().kamera_last_error().decode()


def _check(rc: int):
    if rc != OK:
        raise KameraError(rc, last_error())


# ---------------------------------------------------------------------------
# descriptors
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class RopeSpec:
    """RoPE variant: band [rope_offset, rope_offset + rope_dim), pairing
    "neox" | "interleaved", optional (t, h, w) pair sections."""

    theta: float
    rope_dim: int
    pairing: str = "neox"
    rope_offset: int = 0
    sections: Optional[Tuple[int, int, int]] = None
    section_order: str = "blocked"

    def to_c(self) -> CRope:
        r = CRope()
        r.theta = float(self.theta)
        r.rope_offset = int(self.rope_offset)
        r.rope_dim = int(self.rope_dim)
        r.pairing = {"neox": PAIR_NEOX, "interleaved": PAIR_INTERLEAVED}[self.pairing]
        if self.sections is None:
            r.n_sections = 1
        else:
            r.n_sections = 3
            for k in range(3):
                r.sections[k] = int(self.sections[k])
        r.section_order = {"blocked": SECTIONS_BLOCKED, "interleaved": SECTIONS_INTERLEAVED}[self.section_order]
        return r


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch

    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _strides(t, n: int) -> Sequence[int]:
    """The first n strides (elements) of a tensor whose last stride must be 1."""
    if t.numel() > 0 and t.stride(-1) != 1 and t.shape[-1] > 1:
        raise ValueError("the innermost dimension must be contiguous")
    return [int(s) for s in t.stride()[:n]]


def _bf16(t, name):
    import torch

    if t is not None and t.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be bfloat16 (got {t.dtype})")
    return t


def _i32_dev(t, name):
    import torch

    if t is not None and t.dtype != torch.int32:
        raise TypeError(f"{name} must be int32 (got {t.dtype})")
    return t


def _fill_plane(pl: CPlane, x_in, x_out, U, W, rotate: bool, patch: Tuple[int, int], paged: bool,
                cols: Tuple[int, int] = (0, 0), layer_rank=None):
    pl.in_ = _ptr(x_in)
    for k, s in enumerate(_strides(x_in, 4)):
        pl.in_stride[k] = s
    pl.out = _ptr(x_out)
    if paged:       # pool [L, slots, H, D]: chunk stride unused
        st = _strides(x_out, 3)
        pl.out_stride[0], pl.out_stride[1], pl.out_stride[2], pl.out_stride[3] = 0, st[0], st[1], st[2]
    else:           # dense out [C, L, rows, H, D]
        for k, s in enumerate(_strides(x_out, 4)):
            pl.out_stride[k] = s
    pl.rotate = 1 if rotate else 0
    if U is not None and W is not None and U.shape[-1] > 0:
        pl.m = int(U.shape[-1])
        pl.U = _ptr(U)
        pl.W = _ptr(W)
        for k, s in enumerate(_strides(U, 4)):
            pl.u_stride[k] = s
        for k, s in enumerate(_strides(W, 4)):
            pl.w_stride[k] = s
        pl.patch_offset, pl.patch_dim = int(patch[0]), int(patch[1])
    else:
        pl.m = 0
    pl.col_begin, pl.col_end = int(cols[0]), int(cols[1])
    pl.layer_rank = _ptr(layer_rank)


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

class Prepared:
    """A fully marshalled call: ``launch()`` only crosses into the library.

    Holds references to every tensor the argument struct points at, so the
    memory stays alive as long as the prepared call does.
    """

    def __init__(self, fn, args, keep):
        self._fn = fn
        self.args = args
        self._keep = keep

    def launch(self, stream=None) -> None:
        _check(self._fn(ctypes.byref(self.args), _stream(stream)))


def rehydrate(*a, stream=None, **kw) -> None:
    """``kamera_rehydrate``; see ``prepare_rehydrate`` for the arguments."""
    prepare_rehydrate(*a, **kw).launch(stream)


def rehydrate_plan(prepared: "Prepared") -> int:
    """``kamera_rehydrate_plan`` of a prepared rehydrate call: PLAN_PER_HEAD,
    PLAN_ROW_GROUP or PLAN_ROW_GROUP4 (the kernel the call launches, with 8 or
    4 heads per row-group workgroup), PLAN_NONE, or an error."""
    rc = lib().kamera_rehydrate_plan(ctypes.byref(prepared.args))
    _check(min(rc, 0))
    return rc


def rehydrate_schedule(prepared: "Prepared") -> int:
    """``kamera_rehydrate_schedule`` of a prepared rehydrate call:
    SCHEDULE_PERSISTENT or SCHEDULE_BLOCKS for the row-group kernel, 0 for the
    per-head kernel or nothing to do, or an error."""
    rc = lib().kamera_rehydrate_schedule(ctypes.byref(prepared.args))
    _check(min(rc, 0))
    return rc


def prepare_rehydrate(k_in, k_out, *, rope: RopeSpec, chunk_pos=None, v_in=None, v_out=None,
                      u_k=None, w_k=None, u_v=None, w_v=None, k_patch: Tuple[int, int] = None,
                      v_patch: Tuple[int, int] = None, pos_mode: int = POS_LINEAR, grid_w: int = 0,
                      explicit_pos=None, chunk_tokens=None, row_base=None, page_table=None,
                      page_size: int = 16, n_pool_pages: int = 0,
                      patch_frame: int = PATCH_PRE_ROPE, status=None, delta=None,
                      u_pe=None, w_pe=None, k_layer_rank=None, v_layer_rank=None,
                      pe_layer_rank=None, kernel: int = KERNEL_AUTO, max_workgroups: int = 0,
                      schedule: int = SCHEDULE_AUTO) -> Prepared:
    """Rebuild cached chunks at their target positions (``kamera_rehydrate``).

    k_in, v_in: [C, L, n, H, D] bf16 (any strides, last dim contiguous).
    k_out, v_out: dense [C, L, rows, H, D], or with ``page_table`` the pools
    [L, slots, H, D].  u_*: [C, L, H, n, m]; w_*: [C, L, H, m, patch_dim]
    (expand() views with stride 0 share a factor).  chunk_pos: int32 [C, 3]
    device tensor (p0 or the grid origin).  Keys rotate; values do not.

    delta: int32 [C, 3] device tensor -> relocation: the keys are already
    rotated (at target - delta) and become R(delta) K + R(target) U W.
    u_pe, w_pe: a second, separate patch on the rope band (MLA k_pe band):
    the row splits into two planes, [0, rope_offset) patched by u_k/w_k and the
    band patched by u_pe/w_pe ([C, L, H, n, m_pe], [C, L, H, m_pe, rope_dim]).
    *_layer_rank: int32 [L] device tensors lowering the rank per layer.
    kernel: KERNEL_AUTO, KERNEL_PER_HEAD, KERNEL_ROW_GROUP or KERNEL_ROW_GROUP4 (same results).
    max_workgroups: 0 = one resident wave on the whole device, else a cap (same results).
    schedule: SCHEDULE_AUTO, SCHEDULE_PERSISTENT or SCHEDULE_BLOCKS for the row-group kernel
    (same results).
    """
    L = lib()
    _bf16(k_in, "k_in"), _bf16(k_out, "k_out"), _bf16(v_in, "v_in"), _bf16(v_out, "v_out")
    for t, nm in ((u_k, "u_k"), (w_k, "w_k"), (u_v, "u_v"), (w_v, "w_v")):
        _bf16(t, nm)
    for t, nm in ((chunk_pos, "chunk_pos"), (explicit_pos, "explicit_pos"), (chunk_tokens, "chunk_tokens"),
                  (row_base, "row_base"), (page_table, "page_table")):
        _i32_dev(t, nm)
    C, Ln, n, H, D = (int(s) for s in k_in.shape)
    a = CRehydrateArgs()
    a.n_chunks, a.n_layers, a.n_tokens, a.n_heads, a.head_dim = C, Ln, n, H, D
    a.chunk_tokens = _ptr(chunk_tokens)
    a.patch_frame = patch_frame
    a.rope = rope.to_c()
    a.pos_mode = pos_mode
    a.chunk_pos = _ptr(chunk_pos)
    a.grid_w = grid_w
    a.explicit_pos = _ptr(explicit_pos)
    a.explicit_chunk_stride = int(explicit_pos.stride(0)) if explicit_pos is not None else 0
    paged = page_table is not None
    if u_pe is not None:
        if v_in is not None:
            raise ValueError("a separate rope-band patch splits the key row into two planes; "
                             "values need a call of their own")
        _bf16(u_pe, "u_pe"), _bf16(w_pe, "w_pe")
        ro = int(rope.rope_offset)
        _fill_plane(a.plane[0], k_in, k_out, u_k, w_k, False, k_patch or (0, ro), paged, (0, ro),
                    k_layer_rank)
        _fill_plane(a.plane[1], k_in, k_out, u_pe, w_pe, True, (ro, int(rope.rope_dim)), paged, (ro, D),
                    pe_layer_rank)
        a.n_planes = 2
    else:
        _fill_plane(a.plane[0], k_in, k_out, u_k, w_k, True, k_patch or (0, D), paged, (0, 0), k_layer_rank)
        a.n_planes = 1
    if v_in is not None:
        _fill_plane(a.plane[1], v_in, v_out, u_v, w_v, False, v_patch or (0, D), paged, (0, 0), v_layer_rank)
        a.n_planes = 2
    a.paged = 1 if paged else 0
    a.row_base = _ptr(row_base)
    if paged:
        a.page_table = _ptr(page_table)
        a.pt_stride = int(page_table.stride(0))
        a.page_size = int(page_size)
        a.n_pool_pages = int(n_pool_pages)
    a.status = _ptr(status)
    _i32_dev(delta, "delta")
    a.delta = _ptr(delta)
    a.kernel = int(kernel)
    a.max_workgroups = int(max_workgroups)
    a.schedule = int(schedule)
    keep = (k_in, k_out, v_in, v_out, u_k, w_k, u_v, w_v, chunk_pos, explicit_pos, chunk_tokens,
            row_base, page_table, status, delta, u_pe, w_pe, k_layer_rank, v_layer_rank, pe_layer_rank)
    return Prepared(L.kamera_rehydrate, a, keep)


def shift(*a, stream=None, **kw) -> None:
    """``kamera_shift``; see ``prepare_shift`` for the arguments."""
    prepare_shift(*a, **kw).launch(stream)


def prepare_shift(k, delta, *, rope: RopeSpec, n_chunks: int = None, n_tokens: int = None,
                  chunk_tokens=None, row_base=None, page_table=None, page_size: int = 16,
                  n_pool_pages: int = 0, status=None) -> Prepared:
    """Rotate already-rotated keys by each chunk's delta, in place (``kamera_shift``).

    k: [C, L, n, H, D] (chunks along dim 0), or [L, rows, H, D] with
    ``row_base`` (chunk c starts at row row_base[c]) or with ``page_table``
    (a pool).  delta: int32 [C, 3] device tensor.
    """
    L = lib()
    _bf16(k, "k")
    for t, nm in ((delta, "delta"), (chunk_tokens, "chunk_tokens"), (row_base, "row_base"),
                  (page_table, "page_table")):
        _i32_dev(t, nm)
    a = CShiftArgs()
    if k.dim() == 5:
        C, Ln, n, H, D = (int(s) for s in k.shape)
        for i, s in enumerate(_strides(k, 4)):
            a.k_stride[i] = s
    else:
        Ln, _, H, D = (int(s) for s in k.shape)
        C, n = int(n_chunks), int(n_tokens)
        st = _strides(k, 3)
        a.k_stride[0], a.k_stride[1], a.k_stride[2], a.k_stride[3] = 0, st[0], st[1], st[2]
    a.n_chunks, a.n_layers, a.n_heads, a.head_dim, a.n_tokens = C, Ln, H, D, n
    a.chunk_tokens = _ptr(chunk_tokens)
    a.rope = rope.to_c()
    a.delta = _ptr(delta)
    a.k = _ptr(k)
    a.row_base = _ptr(row_base)
    if page_table is not None:
        a.paged = 1
        a.page_table = _ptr(page_table)
        a.pt_stride = int(page_table.stride(0))
        a.page_size = int(page_size)
        a.n_pool_pages = int(n_pool_pages)
    a.status = _ptr(status)
    return Prepared(L.kamera_shift, a, (k, delta, chunk_tokens, row_base, page_table, status))


def scatter_paged(*a, stream=None, **kw) -> None:
    """``kamera_scatter_paged``; see ``prepare_scatter_paged`` for the arguments."""
    prepare_scatter_paged(*a, **kw).launch(stream)


def gather_paged(*a, stream=None, **kw) -> None:
    """``kamera_gather_paged``: pool rows back into dense rows (the arguments of
    ``prepare_scatter_paged``, with ``rows`` the destination)."""
    prepare_scatter_paged(*a, gather=True, **kw).launch(stream)


def prepare_scatter_paged(rows, pool, page_table, *, page_size: int, n_pool_pages: int,
                          chunk_tokens=None, status=None, gather: bool = False) -> Prepared:
    """Bit copy between dense token rows and page-table slots.

    rows: [C, L, n, ...] (each token row contiguous); pool: [L, slots, ...]
    with the same row shape and dtype.  Scatter copies rows -> pool (the
    default), gather copies pool -> rows.
    """
    L = lib()
    _i32_dev(page_table, "page_table")
    C, Ln, n = (int(x) for x in rows.shape[:3])
    row_elems = 1
    for x in rows.shape[3:]:
        row_elems *= int(x)
    es = rows.element_size()
    if pool.dtype != rows.dtype or tuple(pool.shape[2:]) != tuple(rows.shape[3:]):
        raise ValueError("pool rows must match the dense rows in shape and dtype")
    a = CScatterArgs()
    a.n_chunks, a.n_layers, a.n_tokens = C, Ln, n
    a.chunk_tokens = _ptr(chunk_tokens)
    a.row_bytes = row_elems * es
    a.rows = _ptr(rows)
    for i in range(3):
        a.rows_stride_bytes[i] = int(rows.stride(i)) * es
    a.pool = _ptr(pool)
    for i in range(2):
        a.pool_stride_bytes[i] = int(pool.stride(i)) * es
    a.page_table = _ptr(page_table)
    a.pt_stride = int(page_table.stride(0))
    a.page_size = int(page_size)
    a.n_pool_pages = int(n_pool_pages)
    a.status = _ptr(status)
    fn = L.kamera_gather_paged if gather else L.kamera_scatter_paged
    return Prepared(fn, a, (rows, pool, page_table, chunk_tokens, status))


def form_patch(*a, stream=None, **kw) -> None:
    """``kamera_form_patch``; see ``prepare_form_patch``."""
    prepare_form_patch(*a, **kw).launch(stream)


def prepare_form_patch(delta, U, W, *, sigma=None, sweeps: int = 0, sweeps_done=None) -> Prepared:
    """Top-m truncated SVD of every deficit (App. A compile step).

    delta: fp32 [C, L, H, n, d], or [K, C, L, H, n, d] for an orbit patch
    (Sec. 5, reorder: the K orderings' deficits are averaged first);
    U: bf16 [C, L, H, n, m] (receives U S); W: bf16 [C, L, H, m, d]
    (receives Vt[:m]); sigma: optional fp32 [C, L, H, m] (receives S[:m]).
    m is U's last dimension.  sweeps: 0 (default) takes the tridiagonal
    eigensolver, > 0 block Jacobi with that sweep limit.  sweeps_done:
    optional int32 [C, L, H] (contiguous), receives the Jacobi sweeps each
    unit ran (0 with the tridiagonal solver).
    """
    import torch

    L = lib()
    if delta.dtype != torch.float32:
        raise TypeError(f"delta must be float32 (got {delta.dtype})")
    _bf16(U, "U"), _bf16(W, "W")
    n_orbit, orbit_stride = 0, 0
    if delta.dim() == 6:
        n_orbit, orbit_stride = int(delta.shape[0]), int(delta.stride(0))
        if n_orbit == 0:
            raise ValueError("an orbit patch needs at least one ordering's deficit")
        delta_m = delta[0]
    elif delta.dim() == 5:
        delta_m = delta
    else:
        raise ValueError("delta must be [C, L, H, n, d] or [K, C, L, H, n, d]")
    C, Ln, H, n, d = (int(x) for x in delta_m.shape)
    m = int(U.shape[-1])
    if tuple(U.shape) != (C, Ln, H, n, m) or tuple(W.shape) != (C, Ln, H, m, d):
        raise ValueError("U must be [C, L, H, n, m] and W [C, L, H, m, d]")
    a = CFormArgs()
    a.n_chunks, a.n_layers, a.n_heads, a.n_tokens, a.dim, a.m, a.sweeps = C, Ln, H, n, d, m, int(sweeps)
    a.n_orbit, a.orbit_stride = n_orbit, orbit_stride
    a.delta = _ptr(delta_m)
    for i, st in enumerate(_strides(delta_m, 4)):
        a.delta_stride[i] = st
    a.U = _ptr(U)
    for i, st in enumerate(_strides(U, 4)):
        a.u_stride[i] = st
    a.W = _ptr(W)
    for i, st in enumerate(_strides(W, 4)):
        a.w_stride[i] = st
    if sigma is not None:
        if sigma.dtype != torch.float32 or tuple(sigma.shape) != (C, Ln, H, m):
            raise ValueError("sigma must be float32 [C, L, H, m]")
        a.sigma = _ptr(sigma)
        for i, st in enumerate(_strides(sigma, 3)):
            a.sigma_stride[i] = st
    if sweeps_done is not None:
        if (sweeps_done.dtype != torch.int32 or tuple(sweeps_done.shape) != (C, Ln, H)
                or not sweeps_done.is_contiguous()):
            raise ValueError("sweeps_done must be a contiguous int32 [C, L, H] tensor")
        a.sweeps_done = _ptr(sweeps_done)
    return Prepared(L.kamera_form_patch, a, (delta, U, W, sigma, sweeps_done))


def check_page_table(page_table_host, n_tokens: int, page_size: int, n_pool_pages: int) -> None:
    """Host check of a page table copy (CPU int32 tensor or numpy [C, pages])."""
    import numpy as np

    arr = np.ascontiguousarray(np.asarray(page_table_host, dtype=np.int32))
    C = arr.shape[0]
    stride = arr.shape[1] if arr.ndim == 2 else 0
    _check(lib().kamera_check_page_table(arr.ctypes.data if arr.size else None, C, stride, n_tokens,
                                         page_size, n_pool_pages))
