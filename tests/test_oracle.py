"""The fp64 reference against its pins, and the pins against planted mistakes."""

from __future__ import annotations

import contextlib

import numpy as np
import pytest

import oracle.kamera_ref as ref
from tests import oracle_pins

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(ref)


# ---------------------------------------------------------------------------
# mutants: plausible mistakes planted in the reference (on the CPU only)
# ---------------------------------------------------------------------------

def _rotate_wrong_sign(rows, rope, angles):
    out = np.array(rows, dtype=np.float64, copy=True)
    xc, yc = ref.pair_columns(rope)
    x, y = rows[:, xc], rows[:, yc]
    c, s = np.cos(angles), np.sin(angles)
    out[:, xc] = x * c + y * s
    out[:, yc] = -x * s + y * c
    return out


def _pair_columns_swapped(rope):
    half = rope.rope_dim // 2
    j = np.arange(half)
    if rope.pairing == ref.NEOX:
        x, y = 2 * j, 2 * j + 1
    else:
        x, y = j, j + half
    return rope.rope_offset + x, rope.rope_offset + y


def _inv_freq_half_exponent(theta, rope_dim):
    j = np.arange(rope_dim // 2, dtype=np.float64)
    return np.power(np.float64(theta), -1.0 * j / rope_dim)


def _add_patch_dropped(rows, U, W, patch_offset=0):
    return np.array(rows, dtype=np.float64, copy=True)


def _add_patch_wrong_token(rows, U, W, patch_offset=0):
    out = np.array(rows, dtype=np.float64, copy=True)
    if U is None or W is None or U.shape[1] == 0:
        return out
    out[:, patch_offset:patch_offset + W.shape[1]] += (np.asarray(U) @ np.asarray(W))[::-1]
    return out


def _rehydrate_rotate_first(K, U, W, rope, pos3, patch_offset=0, patch_after_rope=False):
    ang = ref.rope_angles(rope, pos3)
    return ref.add_patch(ref.rotate(np.asarray(K, np.float64), rope, ang), U, W, patch_offset)


def _grid_swapped(base, grid_w, n):
    i = np.arange(n, dtype=np.int64)
    return np.stack([np.full(n, base[0]), base[1] + i % grid_w, base[2] + i // grid_w], axis=1)


def _pair_coordinate_off_by_one(rope):
    c = _orig["pair_coordinate"](rope)
    if rope.sections is not None:
        st = rope.sections[0]
        c = c.copy()
        c[st] = 0
    return c


def _round_ties_away(x):
    x = np.asarray(x, dtype=np.float64)
    bits = _orig["round_bf16"](x)
    # re-round exact ties away from zero
    lo = ref.bf16_to_f64(bits)
    a = np.abs(x)
    spacing = np.abs(ref.bf16_to_f64(bits + np.uint16(1)) - lo)
    tie = np.isclose(np.abs(a - np.abs(lo)), spacing / 2, rtol=0, atol=0) & (np.abs(lo) < a)
    return np.where(tie, bits + np.uint16(1), bits).astype(np.uint16)


def _round_truncate(x):
    x = np.asarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _slot_wrong(page_table_row, i, page_size):
    return int(page_table_row[i // page_size]) * page_size + i // page_size


def _relocate_patch_at_old_position(K, U, W, rope, pos3_target, delta3, patch_offset=0, patch_after_rope=False):
    moved = ref.shift_k(K, rope, delta3)
    if U is None or W is None or np.asarray(U).shape[1] == 0:
        return moved
    patch = ref.add_patch(np.zeros_like(moved), U, W, patch_offset)
    old = np.asarray(pos3_target) - np.asarray(delta3)[None, :]
    return moved + ref.rotate(patch, rope, ref.rope_angles(rope, old))


def _form_patch_unscaled(delta, m):
    Uf, S, Vt = np.linalg.svd(np.asarray(delta, dtype=np.float64), full_matrices=False)
    return Uf[:, :m], Vt[:m], S


def _form_patch_smallest(delta, m):
    Uf, S, Vt = np.linalg.svd(np.asarray(delta, dtype=np.float64), full_matrices=False)
    return Uf[:, -m:] * S[None, -m:], Vt[-m:], S


def _orbit_sum(deltas, m):
    return ref.form_patch(np.sum(np.asarray(deltas, dtype=np.float64), axis=0), m)


def _orbit_first(deltas, m):
    return ref.form_patch(np.asarray(deltas, dtype=np.float64)[0], m)


def _shift_negated(K, rope, delta3):
    return _orig["shift_k"](K, rope, [-int(v) for v in delta3])


_orig = {k: getattr(ref, k) for k in ("pair_coordinate", "round_bf16", "shift_k")}

MUTANTS = {
    "rotation sign flipped": ("rotate", _rotate_wrong_sign),
    "NeoX/interleaved partners swapped": ("pair_columns", _pair_columns_swapped),
    "frequency exponent -j/d": ("inv_freq", _inv_freq_half_exponent),
    "patch term dropped": ("add_patch", _add_patch_dropped),
    "patch rows on the wrong token": ("add_patch", _add_patch_wrong_token),
    "rotation before patch": ("rehydrate_k", _rehydrate_rotate_first),
    "grid h/w swapped": ("positions_grid3", _grid_swapped),
    "section boundary off by one": ("pair_coordinate", _pair_coordinate_off_by_one),
    "bf16 ties away from zero": ("round_bf16", _round_ties_away),
    "bf16 truncation": ("round_bf16", _round_truncate),
    "page slot offset i // P": ("paged_slot", _slot_wrong),
    "shift direction negated": ("shift_k", _shift_negated),
    "removal patch rotated to the old position": ("relocate_k", _relocate_patch_at_old_position),
    "patch forming without the singular values": ("form_patch", _form_patch_unscaled),
    "patch forming keeps the smallest components": ("form_patch", _form_patch_smallest),
    "orbit patch sums instead of averaging": ("orbit_patch", _orbit_sum),
    "orbit patch from one ordering only": ("orbit_patch", _orbit_first),
}


@contextlib.contextmanager
def _planted(attr, fn):
    saved = getattr(ref, attr)
    setattr(ref, attr, fn)
    try:
        yield
    finally:
        setattr(ref, attr, saved)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    attr, fn = MUTANTS[name]
    caught = []
    with _planted(attr, fn):
        for pin in oracle_pins.ALL_PINS:
            try:
                pin(ref)
            except AssertionError:
                caught.append(pin.__name__)
            except Exception:  # a shape error is also a catch
                caught.append(pin.__name__ + " (error)")
    assert caught, f"no pin catches the planted mistake: {name}"
