"""Plain fp64 CPU reference for Kamera's chunk-reuse operator.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code, tables or helpers with the HIP
library; both sides only receive the same seeded inputs.

What it computes (Kamera, Eq. ``eq:operator`` in Sec. 1 and the operator of
Sec. 3; the serve step of App. A):

* rehydrate:  K' = R(pos) . (K + U_k W_k)   on the rope band (patch first, in
  the position-free frame, then rotation), V' = V + U_v W_v;
* shift:      K' = R(delta) . K             (relocation of already-rotated keys,
  valid because R(delta) R(p) = R(p + delta), Sec. 1 and Sec. 3);
* scatter:    a bit copy of dense token rows into the slots a page table names
  (the "clean-view overwrite" of App. E is a copy with no arithmetic; the
  reconstructed KV is written into the paged pool, Sec. 6).

RoPE itself is only cited by the paper (RoFormer); the reading used here is the
standard one: pair j has frequency theta**(-2j/rope_dim) and is rotated by the
angle position * frequency, counter-clockwise, x' = x cos - y sin,
y' = x sin + y cos.  NeoX pairing couples columns (j, j + rope_dim/2);
interleaved pairing couples (2j, 2j+1).  Sectioned multimodal RoPE gives each
pair one of the token's (t, h, w) coordinates (Sec. 3, Fig. ``fig:unify``).

Everything is evaluated in float64: bf16 inputs widen exactly, products of two
bf16 values are exact in fp64 and the rank-m sums carry ~1e-16 relative error.
``round_bf16`` (round to nearest, ties to even) turns a result into the bf16 bit
pattern a correctly rounded implementation would store.

Parity pins: every function here is pinned by tests under ``tests/`` marked
``not gpu`` (closed forms, group properties, Eckart-Young, brute force loops,
independent formulations of RoPE).  Absolute output values of the operator are
not printed anywhere in the paper, so no paper number pins them.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np

NEOX = "neox"
INTERLEAVED = "interleaved"
BLOCKED = "blocked"


# ----------------------------------------------------------------------------
# bf16 <-> float64 (the stored dtype of the cached KV, App. A serve listing)
# ----------------------------------------------------------------------------

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) to float64 exactly.

    A bf16 value is the upper half of an IEEE binary32 pattern, so placing the
    16 bits in the high half of a uint32 and reinterpreting gives the exact
    value, which float64 then holds exactly.
    """
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 bit patterns, nearest-even, from the definition.

    bf16 keeps 8 significant bits.  Instead of bit tricks this works on the
    value: pick the exponent e with 2**e <= |x| < 2**(e+1), the grid spacing
    is 2**(e-7) (the subnormal spacing 2**-133 below the normal range), round
    |x|/spacing to the nearest integer with ties to even (``np.rint``), and
    encode sign, biased exponent and the 7 stored significand bits.  Overflow
    past the largest finite bf16 gives infinity.  NaN is not expected.
    """
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    sign = np.where(np.signbit(x), 0x8000, 0).astype(np.int64)
    a = np.where(np.isfinite(a), a, 0.0) + np.where(np.isinf(x), np.inf, 0.0)
    _, e2 = np.frexp(np.where(np.isinf(a), 1.0, a))  # a = f * 2**e2, 0.5 <= f < 1
    e = np.maximum(e2.astype(np.int64) - 1, -126)
    spacing = np.ldexp(1.0, (e - 7).astype(np.int32))
    q = np.rint(np.where(np.isinf(a), 0.0, a) / spacing)  # exact: < 2**9, ties to even
    up = q >= 256.0                         # rounded into the next binade
    e = np.where(up, e + 1, e)
    q = np.where(up, q / 2.0, q).astype(np.int64)
    normal = q >= 128
    bits = np.where(normal, ((e + 127) << 7) | (q - 128), q)
    bits = np.where(e > 127, 0x7F80, bits)  # overflow -> inf
    bits = np.where(np.isinf(a), 0x7F80, bits)
    bits = np.where(a == 0.0, 0, bits)
    return (sign | bits).astype(np.uint16)


# ----------------------------------------------------------------------------
# RoPE description
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Rope:
    """Which columns rotate and how (Sec. 3 "content | RoPE" split).

    rope_offset, rope_dim: the rotated band is columns [rope_offset,
    rope_offset + rope_dim) of the row (the whole GQA/MHA key, or the 64-dim
    decoupled k_pe behind the 512-dim MLA latent).
    sections: None for 1-D RoPE, else pair counts of the (t, h, w) sections
    (multimodal RoPE, Fig. ``fig:unify``).
    section_order: "blocked" (t pairs first, then h, then w) or "interleaved"
    (pairs cycle t, h, w while each section still has pairs left; the
    remaining pairs take t).
    """

    theta: float
    rope_dim: int
    pairing: str = NEOX
    rope_offset: int = 0
    sections: Optional[Sequence[int]] = None
    section_order: str = BLOCKED


def inv_freq(theta: float, rope_dim: int) -> np.ndarray:
    """Per-pair angular frequency theta**(-2j/rope_dim), j = 0 .. rope_dim/2 - 1."""
    j = np.arange(rope_dim // 2, dtype=np.float64)
    return np.power(np.float64(theta), -2.0 * j / rope_dim)


def pair_coordinate(rope: Rope) -> np.ndarray:
    """Index (0 = t, 1 = h, 2 = w) of the position coordinate that pair j uses."""
    half = rope.rope_dim // 2
    if rope.sections is None:
        return np.zeros(half, dtype=np.int64)
    st, sh, sw = (int(s) for s in rope.sections)
    assert st + sh + sw == half, "sections must cover every pair"
    coord = np.zeros(half, dtype=np.int64)
    if rope.section_order == BLOCKED:
        coord[st:st + sh] = 1
        coord[st + sh:] = 2
    else:
        # cycle t, h, w; a coordinate whose section is used up is skipped
        left = [st, sh, sw]
        j = 0
        while j < half:
            for s in range(3):
                if j < half and left[s] > 0:
                    coord[j] = s
                    left[s] -= 1
                    j += 1
    return coord


def pair_columns(rope: Rope):
    """Column indices (x_j, y_j) of every rotated pair, relative to the row."""
    half = rope.rope_dim // 2
    j = np.arange(half)
    if rope.pairing == NEOX:
        x, y = j, j + half
    else:
        x, y = 2 * j, 2 * j + 1
    return rope.rope_offset + x, rope.rope_offset + y


# ----------------------------------------------------------------------------
# Positions of a chunk's tokens
# ----------------------------------------------------------------------------

def positions_linear(p0: int, n: int) -> np.ndarray:
    """Token i of a chunk placed at offset p0 sits at p0 + i on every coordinate."""
    p = np.int64(p0) + np.arange(n, dtype=np.int64)
    return np.stack([p, p, p], axis=1)


def positions_grid3(base: Sequence[int], grid_w: int, n: int) -> np.ndarray:
    """Frame patches on a grid: token i is at (t0, h0 + i // grid_w, w0 + i % grid_w)."""
    i = np.arange(n, dtype=np.int64)
    t = np.full(n, np.int64(base[0]))
    h = np.int64(base[1]) + i // grid_w
    w = np.int64(base[2]) + i % grid_w
    return np.stack([t, h, w], axis=1)


# ----------------------------------------------------------------------------
# The operator
# ----------------------------------------------------------------------------

def rope_angles(rope: Rope, pos3: np.ndarray) -> np.ndarray:
    """angle[i, j] = pos[i, coord(j)] * theta**(-2j/rope_dim), in float64."""
    f = inv_freq(rope.theta, rope.rope_dim)
    coord = pair_coordinate(rope)
    pos = np.asarray(pos3, dtype=np.float64)
    return pos[:, coord] * f[None, :]


def rotate(rows: np.ndarray, rope: Rope, angles: np.ndarray) -> np.ndarray:
    """Rotate every pair of the rope band of each row by its angle.

    rows: [n, D] float64; angles: [n, rope_dim/2].  Columns outside the band
    are returned unchanged.
    """
    out = np.array(rows, dtype=np.float64, copy=True)
    xc, yc = pair_columns(rope)
    x = rows[:, xc]
    y = rows[:, yc]
    c = np.cos(angles)
    s = np.sin(angles)
    out[:, xc] = x * c - y * s
    out[:, yc] = x * s + y * c
    return out


def add_patch(rows: np.ndarray, U: Optional[np.ndarray], W: Optional[np.ndarray],
              patch_offset: int = 0) -> np.ndarray:
    """rows + U W on columns [patch_offset, patch_offset + W.shape[1]).

    U is the n x m per-token coefficient matrix with the singular values folded
    in, W the m x d basis (the top-m right singular vectors), as the compile
    step of App. A returns them; m = 0 (or None) leaves the rows unchanged.
    """
    out = np.array(rows, dtype=np.float64, copy=True)
    if U is None or W is None or U.shape[1] == 0:
        return out
    U = np.asarray(U, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    out[:, patch_offset:patch_offset + W.shape[1]] += U @ W
    return out


def rehydrate_k(K: np.ndarray, U, W, rope: Rope, pos3: np.ndarray,
                patch_offset: int = 0, patch_after_rope: bool = False) -> np.ndarray:
    """Rebuild one (chunk, layer, head) key block at the given token positions.

    Default reading: K' = R(pos) (K + U W) -- the patch lives in the stored,
    position-free frame so the same patch serves every target position
    (Sec. 3).  ``patch_after_rope`` gives the literal form of Eq.
    ``eq:operator``, K' = R(pos) K + U W, which coincides wherever the patched
    columns are not rotated (V, the MLA latent).
    """
    ang = rope_angles(rope, pos3)
    if patch_after_rope:
        return add_patch(rotate(np.asarray(K, np.float64), rope, ang), U, W, patch_offset)
    return rotate(add_patch(K, U, W, patch_offset), rope, ang)


def rehydrate_v(V: np.ndarray, U, W, patch_offset: int = 0) -> np.ndarray:
    """V' = V + U_v W_v: values carry no rotary phase, only the patch (Sec. 3)."""
    return add_patch(V, U, W, patch_offset)


def shift_k(K: np.ndarray, rope: Rope, delta3: Sequence[int]) -> np.ndarray:
    """K' = R(delta) K for already-rotated keys; every token moves by delta.

    delta3 gives the move of each (t, h, w) coordinate; 1-D RoPE uses
    delta3[0] for every pair.
    """
    n = K.shape[0]
    d = np.asarray(delta3, dtype=np.int64).reshape(1, 3).repeat(n, axis=0)
    return rotate(np.asarray(K, np.float64), rope, rope_angles(rope, d))


def relocate_k(K: np.ndarray, U, W, rope: Rope, pos3_target: np.ndarray, delta3: Sequence[int],
               patch_offset: int = 0, patch_after_rope: bool = False) -> np.ndarray:
    """Move already-rotated keys by delta and add a patch (survivor removal patch).

    Survivors of a window slide keep their conditioned keys, stored rotated at
    their old positions; they move by delta (Sec. 5), and where the evicted
    chunk's influence must be removed a low-rank removal patch is added (Sec. 5,
    Table ``tab:evict``).  K' = R(delta) K + R(pos) U W with pos the target
    position (the patch kept in the position-free frame, as for rehydrate), or
    K' = R(delta) K + U W when the patch lives in the rotated frame.
    """
    moved = shift_k(K, rope, delta3)
    if U is None or W is None or np.asarray(U).shape[1] == 0:
        return moved
    patch = add_patch(np.zeros_like(moved), U, W, patch_offset)
    if not patch_after_rope:
        patch = rotate(patch, rope, rope_angles(rope, pos3_target))
    return moved + patch


def form_patch(delta: np.ndarray, m: int):
    """Stored rank-m patch of a deficit Delta (n x d): the compile step of App. A
    keeps the top-m singular triplets, returning U[:, :m] * S[:m] (n x m, the
    singular values folded into the per-token coefficients) and Vt[:m] (m x d,
    the basis).  U W is then the best rank-m approximation of Delta
    (Eckart-Young).  float64, via numpy's SVD."""
    Uf, S, Vt = np.linalg.svd(np.asarray(delta, dtype=np.float64), full_matrices=False)
    return Uf[:, :m] * S[None, :m], Vt[:m], S


def orbit_patch(deltas, m: int):
    """One stored patch for every ordering of a cached chunk set (Sec. 5,
    reorder): the deficits of the orbit's orderings (K x n x d, the held-out
    ordering left out by the caller) are averaged and the mean is truncated to
    rank m as in ``form_patch``.  Because the sum over the orbit of
    ||Delta_k - P||^2 equals K ||mean - P||^2 plus a term free of P, this is
    the rank-m patch with the least total squared error over the orbit."""
    mean = np.mean(np.asarray(deltas, dtype=np.float64), axis=0)
    return form_patch(mean, m)


def paged_slot(page_table_row: np.ndarray, i: int, page_size: int) -> int:
    """Physical pool slot of a chunk's token i: page_table[i // P] * P + i % P."""
    return int(page_table_row[i // page_size]) * page_size + i % page_size


def scatter_paged(src_rows: np.ndarray, page_table_row: np.ndarray, page_size: int,
                  pool: np.ndarray) -> np.ndarray:
    """Copy token rows of one (chunk, layer) into their pool slots, bit for bit.

    src_rows: [n, ...] any dtype; pool: [n_slots, ...] same dtype.  Returns a
    new pool; slots the page table does not name keep their contents.
    """
    out = np.array(pool, copy=True)
    for i in range(src_rows.shape[0]):
        out[paged_slot(page_table_row, i, page_size)] = src_rows[i]
    return out
