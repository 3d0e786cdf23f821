"""Pins of the fp64 reference against what the mathematics and the paper fix.

Each ``pin_*`` takes the reference module and asserts; ``test_oracle.py`` runs
them on the real module and on deliberately broken copies (a flipped sign, a
wrong pair partner, a dropped term...) to show every planted mistake trips at
least one pin.  Nothing here re-types the reference's own formulas: RoPE is
checked through complex multiplication, the "rotate half" form, an explicit
rotation matrix and scalar loops over math.cos/math.sin; the patch through the
SVD (Eckart-Young) and an identity basis.
"""

from __future__ import annotations

import cmath
import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rng(seed):
    return np.random.default_rng(seed)


def _lin_pos(p0, n):
    p = np.arange(n, dtype=np.int64) + p0
    return np.stack([p, p, p], axis=1)


# ---------------------------------------------------------------------------
# independent formulations of a RoPE rotation
# ---------------------------------------------------------------------------

def _freqs(theta, rd):
    # written out per pair with math.pow, not numpy's vector power
    return [math.pow(theta, -2.0 * j / rd) for j in range(rd // 2)]


def complex_rope_interleaved(band, pos, theta):
    """Interleaved RoPE as complex multiplication: (x + iy) * exp(i p f_j)."""
    n, rd = band.shape
    f = _freqs(theta, rd)
    z = band[:, 0::2] + 1j * band[:, 1::2]
    ph = np.exp(1j * np.outer(pos.astype(np.float64), f))
    w = z * ph
    out = np.empty_like(band)
    out[:, 0::2] = w.real
    out[:, 1::2] = w.imag
    return out


def rotate_half_neox(band, pos, theta):
    """NeoX RoPE in the "rotate half" form: x*cos + rotate_half(x)*sin, where
    rotate_half(x) = [-x2, x1] and cos/sin repeat over both halves."""
    n, rd = band.shape
    f = np.array(_freqs(theta, rd))
    ang = np.outer(pos.astype(np.float64), f)
    cos = np.concatenate([np.cos(ang), np.cos(ang)], axis=1)
    sin = np.concatenate([np.sin(ang), np.sin(ang)], axis=1)
    x1, x2 = band[:, : rd // 2], band[:, rd // 2:]
    rot = np.concatenate([-x2, x1], axis=1)
    return band * cos + rot * sin


def rope_matrix(p, theta, rd, pairing):
    """Explicit rd x rd block rotation matrix R(p); rows act on column vectors."""
    R = np.zeros((rd, rd))
    f = _freqs(theta, rd)
    for j in range(rd // 2):
        a, b = (j, j + rd // 2) if pairing == "neox" else (2 * j, 2 * j + 1)
        c, s = math.cos(p * f[j]), math.sin(p * f[j])
        R[a, a] = c
        R[a, b] = -s
        R[b, a] = s
        R[b, b] = c
    return R


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------

def pin_inv_freq_golden(ref):
    for case in _golden("rope_closed_form.json")["inv_freq"]:
        f = ref.inv_freq(case["theta"], case["rope_dim"])
        assert f.shape == (case["rope_dim"] // 2,)
        assert abs(f[case["j"]] - case["value"]) <= 1e-15 * max(1.0, case["value"]), case


def pin_unit_rotation_golden(ref):
    for pairing in ("neox", "interleaved"):
        rope = ref.Rope(theta=10000.0, rope_dim=2, pairing=pairing)
        for case in _golden("rope_closed_form.json")["unit_rotation"]["cases"]:
            K = np.array([[1.0, 0.0]])
            out = ref.rehydrate_k(K, None, None, rope, _lin_pos(case["p"], 1))
            assert abs(out[0, 0] - case["x"]) < 1e-15 and abs(out[0, 1] - case["y"]) < 1e-15


def pin_bf16_golden(ref):
    cases = _golden("rope_closed_form.json")["bf16_round_nearest_even"]["cases"]
    x = np.array([c["x"] for c in cases])
    want = np.array([int(c["bits"], 16) for c in cases], dtype=np.uint16)
    got = ref.round_bf16(x)
    assert np.array_equal(got, want), (got, want)
    # and widening is exact: the rounded bits decode to the grid point
    assert ref.bf16_to_f64(np.array([0x3F82], np.uint16))[0] == 1.015625


def pin_bf16_vs_library(ref):
    """torch's float32 -> bfloat16 cast (round-nearest-even) is an independent
    implementation; on float32 inputs the two must agree bit for bit."""
    import torch

    rng = _rng(7)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-80, 80, 20000))).astype(np.float32)
    x[:4] = [0.0, -0.0, 1.00390625, -1.01171875]
    t = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ref.round_bf16(x.astype(np.float64)), t)
    back = ref.bf16_to_f64(t)
    assert np.array_equal(back, torch.from_numpy(t.view(np.int16)).view(torch.bfloat16).double().numpy())


def pin_rotation_complex_interleaved(ref):
    rng = _rng(11)
    for rd in (2, 8, 64):
        K = rng.standard_normal((9, rd))
        p0 = int(rng.integers(-5000, 40000))
        rope = ref.Rope(theta=10000.0, rope_dim=rd, pairing="interleaved")
        got = ref.rehydrate_k(K, None, None, rope, _lin_pos(p0, 9))
        want = complex_rope_interleaved(K, np.arange(9) + p0, 10000.0)
        assert np.max(np.abs(got - want)) < 1e-9


def pin_rotation_rotate_half_neox(ref):
    rng = _rng(12)
    for rd in (2, 16, 128):
        K = rng.standard_normal((7, rd))
        p0 = int(rng.integers(-3000, 33000))
        rope = ref.Rope(theta=1e6, rope_dim=rd, pairing="neox")
        got = ref.rehydrate_k(K, None, None, rope, _lin_pos(p0, 7))
        want = rotate_half_neox(K, np.arange(7) + p0, 1e6)
        assert np.max(np.abs(got - want)) < 1e-9


def pin_rotation_matrix_and_band(ref):
    """A band inside a wider row (the MLA k_pe behind the latent): only the band
    moves, by the explicit matrix; columns outside are untouched bit for bit."""
    rng = _rng(13)
    for pairing in ("neox", "interleaved"):
        D, off, rd = 20, 12, 8
        K = rng.standard_normal((5, D))
        rope = ref.Rope(theta=500.0, rope_dim=rd, pairing=pairing, rope_offset=off)
        p = np.array([3, -7, 100, 0, 12345])
        pos = np.stack([p, p, p], axis=1)
        got = ref.rehydrate_k(K, None, None, rope, pos)
        for i in range(5):
            want = rope_matrix(int(p[i]), 500.0, rd, pairing) @ K[i, off:off + rd]
            assert np.max(np.abs(got[i, off:off + rd] - want)) < 1e-12
        assert np.array_equal(got[:, :off], K[:, :off])
        assert np.array_equal(got[:, off + rd:], K[:, off + rd:])


def pin_composition(ref):
    """R(delta) R(p) = R(p + delta) (Sec. 1, Sec. 3): rotating to p then shifting
    by delta equals rotating straight to p + delta, also per M-RoPE coordinate."""
    rng = _rng(14)
    for rope in (ref.Rope(theta=1e6, rope_dim=128, pairing="neox"),
                 ref.Rope(theta=1e4, rope_dim=64, pairing="interleaved"),
                 ref.Rope(theta=1e6, rope_dim=128, pairing="neox", sections=(16, 24, 24))):
        K = rng.standard_normal((6, rope.rope_dim))
        base = np.array([[100, 7, 3], [100, 7, 4], [100, 8, 0], [5, 5, 5], [0, 0, 0], [999, 31, 31]])
        d3 = (-512, 40, -2) if rope.sections else (-512, -512, -512)
        a = ref.shift_k(ref.rehydrate_k(K, None, None, rope, base), rope, d3)
        b = ref.rehydrate_k(K, None, None, rope, base + np.array(d3)[None, :])
        assert np.max(np.abs(a - b)) < 1e-11


def pin_inverse(ref):
    rng = _rng(15)
    for pairing in ("neox", "interleaved"):
        rope = ref.Rope(theta=1e4, rope_dim=32, pairing=pairing)
        K = rng.standard_normal((10, 32))
        back = ref.shift_k(ref.shift_k(K, rope, (777, 777, 777)), rope, (-777, -777, -777))
        assert np.max(np.abs(back - K)) < 1e-12
        moved = ref.shift_k(K, rope, (777, 777, 777))
        assert np.max(np.abs(moved - K)) > 1e-3


def pin_shift_matches_matrix(ref):
    rng = _rng(16)
    rope = ref.Rope(theta=1e4, rope_dim=16, pairing="interleaved")
    K = rng.standard_normal((3, 16))
    got = ref.shift_k(K, rope, (-512, -512, -512))
    R = rope_matrix(-512, 1e4, 16, "interleaved")
    assert np.max(np.abs(got - K @ R.T)) < 1e-12


def pin_m0_is_pure_rope(ref):
    rng = _rng(17)
    rope = ref.Rope(theta=1e6, rope_dim=64, pairing="neox")
    K = rng.standard_normal((12, 64))
    empty_u, empty_w = np.zeros((12, 0)), np.zeros((0, 64))
    got = ref.rehydrate_k(K, empty_u, empty_w, rope, _lin_pos(1000, 12))
    assert np.max(np.abs(got - rotate_half_neox(K, np.arange(12) + 1000, 1e6))) < 1e-9
    V = rng.standard_normal((12, 64))
    assert np.array_equal(ref.rehydrate_v(V, empty_u, empty_w), V)


def pin_full_rank_patch(ref):
    """A full-rank patch reproduces an arbitrary Delta K exactly (U = Delta K,
    W = I), the SVD factors U_m = U S, W = V^T of the compile step rebuild it at
    m = rank, and below full rank the error is the Eckart-Young tail."""
    rng = _rng(18)
    n, d = 24, 16
    K = rng.standard_normal((n, d))
    dK = rng.standard_normal((n, d)) * 0.3
    rope = ref.Rope(theta=1e4, rope_dim=d, pairing="interleaved")
    got = ref.rehydrate_k(K, dK, np.eye(d), rope, _lin_pos(50, n))
    want = complex_rope_interleaved(K + dK, np.arange(n) + 50, 1e4)
    assert np.max(np.abs(got - want)) < 1e-10
    Us, S, Vt = np.linalg.svd(dK, full_matrices=False)
    Um, Wm = Us * S[None, :], Vt
    Z = np.zeros((n, d))
    assert np.max(np.abs(ref.rehydrate_v(Z, Um, Wm) - dK)) < 1e-12
    for m in (1, 4, 9):
        err = np.linalg.norm(ref.rehydrate_v(Z, Um[:, :m], Wm[:m]) - dK)
        assert abs(err - math.sqrt(float(np.sum(S[m:] ** 2)))) < 1e-10
    # patch confined to a column window (the MLA latent in front of the rope key)
    V = rng.standard_normal((n, 2 * d))
    out = ref.rehydrate_v(V, dK, np.eye(d), patch_offset=d)
    assert np.array_equal(out[:, :d], V[:, :d])
    assert np.max(np.abs(out[:, d:] - (V[:, d:] + dK))) < 1e-15


def pin_band_patch_composition(ref):
    """MLA row [latent | rope key]: a latent patch (rank m on the latent
    columns) and a separate rope-band patch (rank m_pe on the band, in the
    stored frame) applied in turn equal one patch with the block basis
    diag(W_lat, W_pe) and concatenated coefficients [U_lat | U_pe]; the latent
    columns never rotate and only the band carries R(p) (k_pe' =
    R(p)(k_pe + U_pe W_pe), checked by complex arithmetic)."""
    rng = _rng(31)
    n, dl, dr, m, mp = 9, 16, 8, 3, 2
    K = rng.standard_normal((n, dl + dr))
    Ul, Wl = rng.standard_normal((n, m)), rng.standard_normal((m, dl))
    Up, Wp = rng.standard_normal((n, mp)), rng.standard_normal((mp, dr))
    rope = ref.Rope(theta=1e4, rope_dim=dr, pairing="interleaved", rope_offset=dl)
    pos = _lin_pos(77, n)
    Wb = np.zeros((m + mp, dl + dr))
    Wb[:m, :dl] = Wl
    Wb[m:, dl:] = Wp
    one = ref.rehydrate_k(K, np.concatenate([Ul, Up], axis=1), Wb, rope, pos)
    staged = ref.rehydrate_k(ref.add_patch(K, Up, Wp, dl), Ul, Wl, rope, pos)
    assert np.max(np.abs(one - staged)) < 1e-12
    assert np.max(np.abs(one[:, :dl] - (K[:, :dl] + Ul @ Wl))) < 1e-12
    band = K[:, dl:] + Up @ Wp
    assert np.max(np.abs(one[:, dl:] - complex_rope_interleaved(band, np.arange(n) + 77, 1e4))) < 1e-10


def pin_identity_index(ref):
    """Position 0 and no patch: cos 0 = 1, sin 0 = 0, so the stored bits come
    back unchanged."""
    rng = _rng(19)
    bits = (rng.integers(0, 2 ** 16, size=(8, 32)) & 0xBFFF).astype(np.uint16)  # finite values
    bits[(bits & 0x7F80) == 0x7F80] = 0x3F80
    K = ref.bf16_to_f64(bits)
    for pairing in ("neox", "interleaved"):
        rope = ref.Rope(theta=1e4, rope_dim=32, pairing=pairing)
        out = ref.rehydrate_k(K, None, None, rope, np.zeros((8, 3), dtype=np.int64))
        assert np.array_equal(ref.round_bf16(out), bits)


def pin_sectioned(ref):
    """Fig. ``fig:unify``: with t = h = w the sectioned rotation is the 1-D one,
    whatever the section layout; a uniform move of all three coordinates is a
    1-D shift."""
    rng = _rng(20)
    K = rng.standard_normal((9, 128))
    p = np.arange(9) * 37 - 50
    pos = np.stack([p, p, p], axis=1)
    one_d = ref.rehydrate_k(K, None, None, ref.Rope(theta=1e6, rope_dim=128), pos)
    for order in ("blocked", "interleaved"):
        r3 = ref.Rope(theta=1e6, rope_dim=128, sections=(16, 24, 24), section_order=order)
        assert np.max(np.abs(ref.rehydrate_k(K, None, None, r3, pos) - one_d)) < 1e-12
        a = ref.shift_k(K, r3, (300, 300, 300))
        b = ref.shift_k(K, ref.Rope(theta=1e6, rope_dim=128), (300, 300, 300))
        assert np.max(np.abs(a - b)) < 1e-12


def pin_pair_coordinate(ref):
    c = ref.pair_coordinate(ref.Rope(theta=1e6, rope_dim=128, sections=(16, 24, 24)))
    assert list(np.bincount(c, minlength=3)) == [16, 24, 24]
    assert c[15] == 0 and c[16] == 1 and c[39] == 1 and c[40] == 2 and c[63] == 2
    ci = ref.pair_coordinate(ref.Rope(theta=1e6, rope_dim=128, sections=(16, 24, 24),
                                      section_order="interleaved"))
    assert list(np.bincount(ci, minlength=3)) == [16, 24, 24]
    assert list(ci[:6]) == [0, 1, 2, 0, 1, 2]
    # t runs out after 16 cycles (pairs 0..47); the rest alternate h, w
    assert list(ci[45:52]) == [0, 1, 2, 1, 2, 1, 2]


def pin_sectioned_grid_brute(ref):
    """Scalar loops with math.cos/sin over a tiny M-RoPE grid chunk."""
    rng = _rng(21)
    rd, gw, n = 12, 3, 7
    sections = (2, 2, 2)
    K = rng.standard_normal((n, rd))
    base = (40, 5, 9)
    rope = ref.Rope(theta=100.0, rope_dim=rd, pairing="neox", sections=sections)
    got = ref.rehydrate_k(K, None, None, rope, ref.positions_grid3(base, gw, n))
    for i in range(n):
        t, h, w = base[0], base[1] + i // gw, base[2] + i % gw
        for j in range(rd // 2):
            coord = t if j < 2 else (h if j < 4 else w)
            a = coord * math.pow(100.0, -2.0 * j / rd)
            x, y = K[i, j], K[i, j + rd // 2]
            assert abs(got[i, j] - (x * math.cos(a) - y * math.sin(a))) < 1e-12
            assert abs(got[i, j + rd // 2] - (x * math.sin(a) + y * math.cos(a))) < 1e-12


def pin_grid_positions(ref):
    g = ref.positions_grid3((7, 100, 200), 32, 70)
    assert tuple(g[0]) == (7, 100, 200)
    assert tuple(g[31]) == (7, 100, 231)
    assert tuple(g[33]) == (7, 101, 201)
    assert tuple(g[69]) == (7, 102, 205)
    lp = ref.positions_linear(-3, 4)
    assert lp.tolist() == [[-3, -3, -3], [-2, -2, -2], [-1, -1, -1], [0, 0, 0]]


def pin_interleaved_vs_neox(ref):
    """interleaved(x) = P^T neox(P x) with P gathering even columns, then odd."""
    rng = _rng(22)
    K = rng.standard_normal((5, 32))
    perm = np.concatenate([np.arange(0, 32, 2), np.arange(1, 32, 2)])
    pos = _lin_pos(321, 5)
    a = ref.rehydrate_k(K, None, None, ref.Rope(theta=1e4, rope_dim=32, pairing="interleaved"), pos)
    b = ref.rehydrate_k(K[:, perm], None, None, ref.Rope(theta=1e4, rope_dim=32, pairing="neox"), pos)
    back = np.empty_like(b)
    back[:, perm] = b
    assert np.max(np.abs(a - back)) < 1e-12


def pin_norm_and_linearity(ref):
    rng = _rng(23)
    rope = ref.Rope(theta=1e6, rope_dim=64, pairing="neox")
    K = rng.standard_normal((11, 64))
    U = rng.standard_normal((11, 5))
    W = rng.standard_normal((5, 64))
    pos = _lin_pos(4000, 11)
    out = ref.rehydrate_k(K, U, W, rope, pos)
    pre = K + U @ W
    n_in = pre[:, :32] ** 2 + pre[:, 32:] ** 2
    n_out = out[:, :32] ** 2 + out[:, 32:] ** 2
    assert np.max(np.abs(n_in - n_out)) < 1e-10
    lin = ref.rehydrate_k(K, None, None, rope, pos) + ref.rehydrate_k(np.zeros_like(K), U, W, rope, pos)
    assert np.max(np.abs(out - lin)) < 1e-10


def pin_patch_order_reading(ref):
    """Patch in the stored frame, then rotate (default); the literal Eq. 1 form
    adds the patch after rotation.  They agree on unrotated columns and differ
    on the rotated ones."""
    rng = _rng(24)
    rope = ref.Rope(theta=1e4, rope_dim=8, pairing="neox", rope_offset=8)
    K = rng.standard_normal((4, 16))
    U = rng.standard_normal((4, 2))
    W = rng.standard_normal((2, 16))
    pos = _lin_pos(9, 4)
    pre = ref.rehydrate_k(K, U, W, rope, pos)
    post = ref.rehydrate_k(K, U, W, rope, pos, patch_after_rope=True)
    for i in range(4):
        R = rope_matrix(9 + i, 1e4, 8, "neox")
        want_pre = R @ (K[i, 8:] + U[i] @ W[:, 8:])
        want_post = R @ K[i, 8:] + U[i] @ W[:, 8:]
        assert np.max(np.abs(pre[i, 8:] - want_pre)) < 1e-12
        assert np.max(np.abs(post[i, 8:] - want_post)) < 1e-12
    assert np.max(np.abs(pre[:, :8] - post[:, :8])) < 1e-12


def pin_brute_force_tiny(ref):
    """Per-element scalar loops (plain Python floats) on tiny inputs."""
    rng = _rng(25)
    n, d, m = 5, 8, 3
    for pairing in ("neox", "interleaved"):
        K = rng.standard_normal((n, d))
        U = rng.standard_normal((n, m))
        W = rng.standard_normal((m, d))
        rope = ref.Rope(theta=50.0, rope_dim=d, pairing=pairing)
        p0 = 17
        got = ref.rehydrate_k(K, U, W, rope, _lin_pos(p0, n))
        for i in range(n):
            row = [float(K[i, c]) + sum(float(U[i, k]) * float(W[k, c]) for k in range(m))
                   for c in range(d)]
            want = list(row)
            for j in range(d // 2):
                a_idx, b_idx = (j, j + d // 2) if pairing == "neox" else (2 * j, 2 * j + 1)
                ang = (p0 + i) * 50.0 ** (-2.0 * j / d)
                z = complex(row[a_idx], row[b_idx]) * cmath.exp(1j * ang)
                want[a_idx], want[b_idx] = z.real, z.imag
            for c in range(d):
                assert abs(got[i, c] - want[c]) < 1e-12


def pin_paged_slot_and_scatter(ref):
    pt = np.array([5, 2, 9], dtype=np.int32)
    assert ref.paged_slot(pt, 0, 16) == 80
    assert ref.paged_slot(pt, 17, 16) == 33
    assert ref.paged_slot(pt, 47, 16) == 159
    rng = _rng(26)
    n, P, slots = 40, 16, 16 * 12
    src = rng.integers(0, 2 ** 16, size=(n, 6)).astype(np.uint16)
    pool = np.full((slots, 6), 0xDEAD, dtype=np.uint16)
    out = ref.scatter_paged(src, pt, P, pool)
    written = set()
    for i in range(n):
        page, off = int(pt[i // P]), i % P
        assert np.array_equal(out[page * P + off], src[i])
        written.add(page * P + off)
    for s in range(slots):
        if s not in written:
            assert np.all(out[s] == 0xDEAD)


def pin_relocate(ref):
    """Survivor relocation with a removal patch: a key rehydrated at p (no
    patch) and then moved by delta with the patch equals rehydrating it at
    p + delta with the patch, because R(delta) R(p) = R(p + delta) and the
    patch lives in the position-free frame; with no patch it is a plain shift;
    in the rotated frame the patch is added unrotated."""
    rng = _rng(27)
    for rope in (ref.Rope(theta=1e6, rope_dim=64, pairing="neox"),
                 ref.Rope(theta=1e4, rope_dim=32, pairing="interleaved", rope_offset=32),
                 ref.Rope(theta=1e6, rope_dim=64, pairing="neox", sections=(8, 12, 12))):
        D = rope.rope_offset + rope.rope_dim
        K0 = rng.standard_normal((6, D))
        U = rng.standard_normal((6, 3))
        W = rng.standard_normal((3, D))
        old = np.array([[50, 3, 4], [51, 3, 5], [52, 4, 0], [53, 4, 1], [54, 4, 2], [55, 5, 0]])
        d3 = np.array([-512, 7, -2]) if rope.sections else np.array([-512, -512, -512])
        stored = ref.rehydrate_k(K0, None, None, rope, old)
        got = ref.relocate_k(stored, U, W, rope, old + d3[None, :], d3)
        want = ref.rehydrate_k(K0, U, W, rope, old + d3[None, :])
        assert np.max(np.abs(got - want)) < 1e-11
        assert np.max(np.abs(ref.relocate_k(stored, None, None, rope, old + d3, d3) -
                             ref.shift_k(stored, rope, d3))) < 1e-13
        post = ref.relocate_k(stored, U, W, rope, old + d3, d3, patch_after_rope=True)
        assert np.max(np.abs(post - (ref.shift_k(stored, rope, d3) + U @ W))) < 1e-11
    # brute force, one NeoX pair per token
    K = rng.standard_normal((3, 2))
    U = rng.standard_normal((3, 1))
    W = rng.standard_normal((1, 2))
    rope = ref.Rope(theta=10.0, rope_dim=2)
    tgt = np.array([[5, 5, 5], [9, 9, 9], [-4, -4, -4]])
    got = ref.relocate_k(K, U, W, rope, tgt, (3, 3, 3))
    for i in range(3):
        zk = complex(K[i, 0], K[i, 1]) * cmath.exp(1j * 3.0)
        zp = complex(U[i, 0] * W[0, 0], U[i, 0] * W[0, 1]) * cmath.exp(1j * float(tgt[i, 0]))
        z = zk + zp
        assert abs(got[i, 0] - z.real) < 1e-12 and abs(got[i, 1] - z.imag) < 1e-12


def pin_form_patch(ref):
    """The compile step's factors: U W is the rank-m truncation (Eckart-Young
    residual), W has orthonormal rows, U = Delta W^T (singular values folded
    in), a planted rank-r Delta is rebuilt exactly at m = r, and the factors
    rehydrate Delta back through the patch path."""
    rng = _rng(28)
    n, d = 40, 12
    delta = rng.standard_normal((n, d))
    for m in (1, 5, d):
        U, W, S = ref.form_patch(delta, m)
        assert U.shape == (n, m) and W.shape == (m, d)
        err = np.linalg.norm(delta - U @ W)
        assert abs(err - math.sqrt(float(np.sum(S[m:] ** 2)))) < 1e-10
        assert np.max(np.abs(W @ W.T - np.eye(m))) < 1e-12
        assert np.max(np.abs(U - delta @ W.T)) < 1e-12
        # singular values come out in descending order and match the Gram matrix eigenvalues
        ev = np.sort(np.linalg.eigvalsh(delta.T @ delta))[::-1]
        assert np.max(np.abs(S ** 2 - ev)) < 1e-9
    A = rng.standard_normal((n, 3))
    B = rng.standard_normal((3, d))
    U, W, S = ref.form_patch(A @ B, 3)
    assert np.max(np.abs(U @ W - A @ B)) < 1e-11
    assert S[3] < 1e-12
    K = rng.standard_normal((n, d))
    assert np.max(np.abs(ref.rehydrate_v(K, U, W) - (K + A @ B))) < 1e-11


def pin_orbit_patch(ref):
    """The orbit patch: an orbit of identical deficits gives that deficit's own
    patch; for a real orbit its total squared error over the members is below
    that of every member's own patch, of the mean's rank-m truncation by any
    other rank-m subspace tried, and it equals the decomposition
    K ||mean - P||^2 + sum ||Delta_k - mean||^2."""
    rng = _rng(29)
    n, d, m, K = 30, 10, 3, 4
    base = rng.standard_normal((n, d))
    U1, W1, _ = ref.form_patch(base, m)
    Uo, Wo, _ = ref.orbit_patch(np.stack([base] * K), m)
    assert np.max(np.abs(Uo @ Wo - U1 @ W1)) < 1e-11
    # a shared low-rank core plus an ordering-dependent part
    core = rng.standard_normal((n, m)) @ rng.standard_normal((m, d)) * 3.0
    deltas = np.stack([core + rng.standard_normal((n, d)) for _ in range(K)])
    Uo, Wo, _ = ref.orbit_patch(deltas, m)
    P = Uo @ Wo

    def total(Q):
        return float(sum(np.sum((dk - Q) ** 2) for dk in deltas))

    mean = deltas.mean(axis=0)
    spread = float(sum(np.sum((dk - mean) ** 2) for dk in deltas))
    assert abs(total(P) - (K * np.sum((mean - P) ** 2) + spread)) < 1e-8 * total(P)
    for dk in deltas:
        Uk, Wk, _ = ref.form_patch(dk, m)
        assert total(P) < total(Uk @ Wk)
    for _ in range(20):
        Q, _r = np.linalg.qr(rng.standard_normal((d, m)))
        assert total(P) <= total(mean @ Q @ Q.T) + 1e-9
    # the orbit mean of K scaled copies c_k Delta is the patch of mean(c_k) Delta
    cs = np.array([0.5, 1.0, 2.0, 4.5])
    Uo, Wo, _ = ref.orbit_patch(cs[:, None, None] * base[None], m)
    assert np.max(np.abs(Uo @ Wo - cs.mean() * (U1 @ W1))) < 1e-10


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
