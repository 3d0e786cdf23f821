"""Seeded synthetic inputs for Kamera's chunk-reuse operator.

This module only draws numbers and describes shapes: it holds none of the
operator's arithmetic (no rotation, no patch, no page-slot formula).  The tests
and the benchmark use it to give the HIP library and the fp64 reference the
same inputs.

The paper's workloads are cached video segments of a few hundred to a couple of
thousand tokens (Sec. 1: 1024-token segments; App. D/ deploy figure: segments
of 256 to 2048 tokens) on GQA, MHA and MLA backbones with 27 to 80 layers.  Its
datasets and model weights are not available, so every tensor here is a
seeded stand-in with those shapes: K, V (and the MLA latent and rope key)
~ N(0, 1), patch coefficients U and bases W ~ N(0, 0.1^2), all rounded to bf16.

``WORKLOADS`` lists the operator workloads the benchmark and the parity tests
use: five from a one-layer GQA chunk up to the 80-layer paged recall
(``WORKLOAD_ORDER``), and three for the operator's other modes -- relocation
with a removal patch, the MLA rope-band patch and deep-half factors
(``EXTRA_WORKLOADS``).
"""

from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

NEOX = "neox"
INTERLEAVED = "interleaved"


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and layout description of one operator call."""

    name: str
    kind: str                    # "rehydrate" or "shift"
    n_chunks: int
    n_layers: int
    n_heads: int                 # KV heads (1 for the MLA latent row)
    head_dim: int                # row width in elements (576 for MLA)
    n_tokens: int                # tokens per chunk
    theta: float
    rope_dim: int
    rope_offset: int = 0
    pairing: str = NEOX
    sections: Optional[Tuple[int, int, int]] = None
    section_order: str = "blocked"
    m_k: int = 0
    m_v: int = 0
    patch_offset: int = 0
    patch_dim: int = 0
    has_v: bool = True
    paged: bool = False
    page_size: int = 16
    n_pool_pages: int = 0
    pos_mode: str = "linear"     # "linear" | "grid3"
    grid_w: int = 0
    seed: int = 0
    u_std: float = 0.1
    w_std: float = 0.1
    # shift workloads: a ring window of chunk slots
    window_slots: int = 0
    delta: int = 0
    slides: int = 1
    # survivors moved by delta with a removal patch, in place (relocation)
    reloc: bool = False
    # separate rank on the rope band (MLA k_pe) and deep-half patches
    m_pe: int = 0
    patch_from_layer: int = 0       # layers below carry no factors (rank 0)

    def units(self) -> int:
        return self.n_chunks * self.n_layers * self.n_heads


WORKLOADS: Dict[str, Workload] = {
    # one-layer GQA chunk: 256 tokens, 8 KV heads, rank-8 patch, placed at 1000
    "gqa1l_256tok_m8": Workload(
        name="gqa1l_256tok_m8", kind="rehydrate", n_chunks=1, n_layers=1,
        n_heads=8, head_dim=128, n_tokens=256, theta=1e6, rope_dim=128,
        pairing=NEOX, m_k=8, m_v=8, patch_dim=128, seed=1001, delta=-256),
    # reorder: 8 video-segment chunks of 1024 tokens in a permuted order
    "gqa28l_8x1024_m16_reorder": Workload(
        name="gqa28l_8x1024_m16_reorder", kind="rehydrate", n_chunks=8,
        n_layers=28, n_heads=4, head_dim=128, n_tokens=1024, theta=1e6,
        rope_dim=128, pairing=NEOX, m_k=16, m_v=16, patch_dim=128, seed=1002),
    # sliding window: 16 slots x 512 tokens, survivors rotate by -512, 8 slides
    "mha32l_window16x512_shift": Workload(
        name="mha32l_window16x512_shift", kind="shift", n_chunks=15,
        n_layers=32, n_heads=32, head_dim=128, n_tokens=512, theta=1e4,
        rope_dim=128, pairing=INTERLEAVED, seed=1003, window_slots=16,
        delta=-512, slides=8),
    # MLA: latent 512 (patched, rank 32) + decoupled rope key 64 (rotated)
    "mla27l_4x2048_m32": Workload(
        name="mla27l_4x2048_m32", kind="rehydrate", n_chunks=4, n_layers=27,
        n_heads=1, head_dim=576, n_tokens=2048, theta=1e4, rope_dim=64,
        rope_offset=512, pairing=INTERLEAVED, m_k=32, m_v=0, patch_dim=512,
        has_v=False, seed=1004),
    # recall: 64 frame chunks (32x32 patch grid) into a paged pool, M-RoPE
    "gqa80l_64x1024_m64_mrope_paged": Workload(
        name="gqa80l_64x1024_m64_mrope_paged", kind="rehydrate", n_chunks=64,
        n_layers=80, n_heads=8, head_dim=128, n_tokens=1024, theta=1e6,
        rope_dim=128, pairing=NEOX, sections=(16, 24, 24),
        section_order="blocked", m_k=64, m_v=64, patch_dim=128, paged=True,
        page_size=16, n_pool_pages=4096, pos_mode="grid3", grid_w=32,
        seed=1005),
    # --- the operator's other modes ---
    # survivors of a slide on a 36-layer deepstack-style GQA model: 15 frame
    # chunks moved back by one chunk, in place, with rank-64 removal patches
    "gqa36l_15x1024_survivor_m64": Workload(
        name="gqa36l_15x1024_survivor_m64", kind="rehydrate", n_chunks=15,
        n_layers=36, n_heads=8, head_dim=128, n_tokens=1024, theta=5e6,
        rope_dim=128, pairing=NEOX, sections=(24, 20, 20),
        section_order="interleaved", m_k=64, m_v=64, patch_dim=128,
        pos_mode="grid3", grid_w=32, reloc=True, delta=-1024, window_slots=16,
        seed=1006),
    # MLA with the extra rank-16 patch on the 64-dim rope key band
    "mla27l_4x2048_m32_pe16": Workload(
        name="mla27l_4x2048_m32_pe16", kind="rehydrate", n_chunks=4, n_layers=27,
        n_heads=1, head_dim=576, n_tokens=2048, theta=1e4, rope_dim=64,
        rope_offset=512, pairing=INTERLEAVED, m_k=32, m_v=0, m_pe=16,
        patch_dim=512, has_v=False, seed=1007),
    # the 80-layer paged recall with factors on the deepest 40 layers only
    "gqa80l_64x1024_m64_mrope_paged_deephalf": Workload(
        name="gqa80l_64x1024_m64_mrope_paged_deephalf", kind="rehydrate",
        n_chunks=64, n_layers=80, n_heads=8, head_dim=128, n_tokens=1024,
        theta=1e6, rope_dim=128, pairing=NEOX, sections=(16, 24, 24),
        section_order="blocked", m_k=64, m_v=64, patch_dim=128, paged=True,
        page_size=16, n_pool_pages=4096, pos_mode="grid3", grid_w=32,
        patch_from_layer=40, seed=1008),
    # a mid-size paged recall: 16 frame chunks on a 32-layer model, rank 32
    "gqa32l_16x1024_m32_mrope_paged": Workload(
        name="gqa32l_16x1024_m32_mrope_paged", kind="rehydrate", n_chunks=16,
        n_layers=32, n_heads=8, head_dim=128, n_tokens=1024, theta=1e6,
        rope_dim=128, pairing=NEOX, sections=(16, 24, 24),
        section_order="blocked", m_k=32, m_v=32, patch_dim=128, paged=True,
        page_size=16, n_pool_pages=1024, pos_mode="grid3", grid_w=32,
        seed=1009),
}

# order in which the workloads are listed (smallest first)
WORKLOAD_ORDER: List[str] = [
    "gqa1l_256tok_m8",
    "gqa28l_8x1024_m16_reorder",
    "mha32l_window16x512_shift",
    "mla27l_4x2048_m32",
    "gqa80l_64x1024_m64_mrope_paged",
]

# workloads of the operator's other modes (relocation with a removal patch,
# a second rank on the MLA rope band, deep-half factors) and a mid-size recall
EXTRA_WORKLOADS: List[str] = [
    "gqa36l_15x1024_survivor_m64",
    "mla27l_4x2048_m32_pe16",
    "gqa80l_64x1024_m64_mrope_paged_deephalf",
    "gqa32l_16x1024_m32_mrope_paged",
]


# ----------------------------------------------------------------------------
# Host-side per-chunk metadata (integers only)
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class ChunkMeta:
    """Per-chunk integers of one call, drawn from ``numpy.random.default_rng(seed)``.

    pos[c] = (a, b, c3): for linear placement (p0, p0, p0); for grid placement
    the (t, h, w) of the chunk's first patch.  row_base[c]: first output row of
    chunk c in a dense output.  page_table[c][k]: pool page of tokens
    [k*P, (k+1)*P) of chunk c.  delta[c]: (dt, dh, dw) move for a shift.
    """

    pos: np.ndarray                      # int32 [C, 3]
    row_base: np.ndarray                 # int32 [C]
    page_table: Optional[np.ndarray]     # int32 [C, pages_per_chunk]
    delta: np.ndarray                    # int32 [C, 3]
    order: Optional[np.ndarray] = None   # slot -> chunk permutation (reorder)


def chunk_meta(w: Workload, seed: Optional[int] = None) -> ChunkMeta:
    rng = np.random.default_rng(w.seed if seed is None else seed)
    C, n = w.n_chunks, w.n_tokens
    order = None
    pos = np.zeros((C, 3), dtype=np.int32)
    row_base = np.zeros(C, dtype=np.int32)
    delta = np.zeros((C, 3), dtype=np.int32)
    page_table = None
    if w.name == "gqa1l_256tok_m8":
        pos[:] = 1000
        delta[:] = w.delta
    elif w.name == "gqa28l_8x1024_m16_reorder":
        # slot s holds chunk order[s]; contiguous target offsets 1024*s
        order = rng.permutation(C).astype(np.int32)
        for s, c in enumerate(order):
            pos[c, :] = n * s
            row_base[c] = n * s
    elif w.name in ("mla27l_4x2048_m32", "mla27l_4x2048_m32_pe16"):
        p0 = rng.integers(0, 32768 - n + 1, size=C)
        pos[:] = p0[:, None]
        row_base[:] = np.arange(C) * n
    elif w.name == "gqa36l_15x1024_survivor_m64":
        # survivor k sat at slot k + 1 of the window (frame origin 1024*(k+1) on
        # every coordinate) and moves to slot k: all three coordinates by delta
        pos[:] = (n * np.arange(C))[:, None]
        delta[:] = w.delta
    elif w.name in ("gqa80l_64x1024_m64_mrope_paged", "gqa80l_64x1024_m64_mrope_paged_deephalf",
                    "gqa32l_16x1024_m32_mrope_paged"):
        s = rng.integers(1, 4097, size=C)          # temporal delta in [1, 4096]
        pos[:] = s[:, None]                        # all three coordinates advance together
        pages = (n + w.page_size - 1) // w.page_size
        perm = rng.permutation(w.n_pool_pages)[: C * pages]
        page_table = perm.reshape(C, pages).astype(np.int32)
    elif w.kind == "shift":
        delta[:] = w.delta
    else:
        row_base[:] = np.arange(C) * n
    return ChunkMeta(pos=pos, row_base=row_base, page_table=page_table,
                     delta=delta, order=order)


def window_survivor_slots(w: Workload, slide: int) -> np.ndarray:
    """Ring-deque window: at slide k the oldest slot k % S is evicted; the other
    S-1 slots (oldest first) are the survivors that move by ``w.delta``."""
    S = w.window_slots
    evict = slide % S
    return np.array([(evict + 1 + k) % S for k in range(S - 1)], dtype=np.int32)


# ----------------------------------------------------------------------------
# Bulk tensors
# ----------------------------------------------------------------------------

def randn_bf16_numpy(shape, std: float, rng: np.random.Generator) -> np.ndarray:
    """N(0, std^2) rounded to bf16, returned as uint16 bit patterns (CPU tests)."""
    import torch

    x = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std)
    return torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def randn_bf16_device(shape, std: float, gen, device, slab_dim: int = 0, out=None):
    """N(0, std^2) bf16 tensor drawn on the device in slabs along ``slab_dim``
    (keeps the fp32 temporary small for tens-of-GB tensors); fills ``out``
    (shape ``shape``) when given."""
    import torch

    if out is None:
        out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    assert tuple(out.shape) == tuple(shape)
    if len(shape) == 0 or shape[slab_dim] == 0:
        return out
    for k in range(shape[slab_dim]):
        sl = out.select(slab_dim, k)
        tmp = torch.randn(sl.shape, generator=gen, device=device, dtype=torch.float32)
        if std != 1.0:
            tmp.mul_(std)
        sl.copy_(tmp)
        del tmp
    return out
