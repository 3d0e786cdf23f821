"""HIP library vs the fp64 reference on small seeded cases (several 16-token
tiles, ragged tails, every RoPE variant, ranks 0..128, dense and paged)."""

from __future__ import annotations

import zlib

import numpy as np
import pytest

import oracle as ref
import synth
from tests.gpu_util import (SENTINEL, TOL, RehydrateCase, assert_close, bits, dev, dev_i32, oracle_rope,
                            require_gpu, run_rehydrate)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def device():
    return require_gpu()


REHYDRATE_CASES = {
    "gqa_neox_m16": RehydrateCase(),
    "gqa_neox_m0": RehydrateCase(m_k=0, m_v=0, seed=1),
    "gqa_neox_m8": RehydrateCase(m_k=8, m_v=8, n=37, seed=2),
    "gqa_neox_m32_m64": RehydrateCase(m_k=32, m_v=64, seed=3),
    "gqa_full_rank_128": RehydrateCase(m_k=128, m_v=128, n=48, C=1, L=1, H=2, seed=4),
    "gqa_odd_rank_5_33": RehydrateCase(m_k=5, m_v=33, n=50, seed=5),
    "gqa_interleaved": RehydrateCase(pairing="interleaved", theta=1e4, seed=6),
    "gqa_large_positions": RehydrateCase(p0_range=(1 << 20, (1 << 20) + 5000), seed=7),
    "gqa_negative_positions": RehydrateCase(p0_range=(-70000, -1000), seed=8),
    "gqa_one_token": RehydrateCase(n=1, seed=9),
    "gqa_ragged": RehydrateCase(ragged=True, n=90, C=4, seed=10),
    "gqa_post_rope_frame": RehydrateCase(post_rope=True, seed=11),
    "gqa_shared_basis": RehydrateCase(shared_w=True, C=3, seed=12),
    "gqa_partial_rotary": RehydrateCase(rope_dim=64, rope_offset=64, pairing="neox", patch=(32, 64), seed=13),
    "gqa_d256": RehydrateCase(D=256, rope_dim=128, rope_offset=128, patch=(0, 256), n=40, seed=14),
    "mla_interleaved": RehydrateCase(D=576, H=1, rope_dim=64, rope_offset=512, pairing="interleaved",
                                     theta=1e4, patch=(0, 512), m_k=32, has_v=False, n=77, seed=15),
    "mla_neox": RehydrateCase(D=576, H=1, rope_dim=64, rope_offset=512, pairing="neox", theta=1e4,
                              patch=(0, 512), m_k=32, has_v=False, n=50, seed=16),
    "mrope_blocked_grid_paged": RehydrateCase(sections=(16, 24, 24), pos_mode="grid3", grid_w=32,
                                              paged=True, m_k=64, m_v=64, n=96, p0_range=(1, 4097),
                                              seed=17),
    "mrope_interleaved_grid7_paged": RehydrateCase(sections=(24, 20, 20), section_order="interleaved",
                                                   pos_mode="grid3", grid_w=7, paged=True, page_size=5,
                                                   n=61, seed=18),
    "explicit_positions": RehydrateCase(sections=(16, 24, 24), pos_mode="explicit", n=45, seed=19),
    "paged_page_size_1": RehydrateCase(paged=True, page_size=1, n=20, seed=20),
    # survivors: keys already rotated, moved by delta with a removal patch
    "relocate_neox_m64": RehydrateCase(reloc=True, m_k=64, m_v=64, n=70, seed=21),
    "relocate_interleaved_post_frame": RehydrateCase(reloc=True, pairing="interleaved", theta=1e4,
                                                     post_rope=True, seed=22),
    "relocate_mrope_grid_paged": RehydrateCase(reloc=True, sections=(16, 24, 24), pos_mode="grid3",
                                               paged=True, m_k=32, m_v=0, seed=23),
    "relocate_no_patch": RehydrateCase(reloc=True, m_k=0, m_v=0, seed=24),
    # MLA with a second, separate patch on the rope key band
    "mla_band_patch": RehydrateCase(D=576, H=1, rope_dim=64, rope_offset=512, pairing="interleaved",
                                    theta=1e4, patch=(0, 512), m_k=32, m_pe=16, has_v=False, n=77, seed=25),
    "mla_band_patch_reloc_paged": RehydrateCase(D=576, H=1, rope_dim=64, rope_offset=512, pairing="neox",
                                                theta=1e4, patch=(0, 512), m_k=32, m_pe=8, has_v=False,
                                                reloc=True, paged=True, n=40, seed=26),
    # deep-half patch: no factors on the shallow layers, odd ranks on others
    "max_row_4096": RehydrateCase(D=4096, H=1, C=1, L=2, n=20, rope_dim=128, rope_offset=2048, m_k=8, m_v=8,
                                  patch=(0, 4096), seed=29),
    "relocate_layer_rank_post_frame": RehydrateCase(reloc=True, post_rope=True, L=3, layer_rank=(0, 32, 7), m_k=32,
                                                    m_v=32, seed=40),
    "post_rope_grid_paged_shared": RehydrateCase(post_rope=True, sections=(16, 24, 24), pos_mode="grid3", grid_w=8,
                                                 paged=True, shared_w=True, C=3, seed=41),
    "mla_band_patch_layer_rank_shared": RehydrateCase(D=576, H=1, rope_dim=64, rope_offset=512, pairing="interleaved",
                                                      theta=1e4, patch=(0, 512), has_v=False, m_k=32, m_v=0, m_pe=16,
                                                      L=3, layer_rank=(16, 0, 48), shared_w=True, seed=42),
    "explicit_ragged_paged_rank_100": RehydrateCase(pos_mode="explicit", sections=(24, 20, 20),
                                                    section_order="interleaved", ragged=True, paged=True,
                                                    page_size=7, m_k=100, m_v=3, n=77, C=3, seed=43),
    "layer_rank_deep_half": RehydrateCase(L=4, layer_rank=(0, 0, 16, 16), m_k=16, m_v=16, seed=27),
    "layer_rank_odd": RehydrateCase(L=3, layer_rank=(5, 64, 33), m_k=64, m_v=48, seed=28),
    # the row-group kernel (all heads of a token row per workgroup), requested on
    # small shapes, and requests it cannot serve (they fall back to the per-head kernel)
    "rows_h8_mrope_grid_paged_m64": RehydrateCase(H=8, n=100, sections=(16, 24, 24), pos_mode="grid3", grid_w=32,
                                                  paged=True, m_k=64, m_v=64, p0_range=(1, 4097),
                                                  kernel=2, plan=2, seed=50),
    "rows_h3_interleaved_page24_ragged": RehydrateCase(pairing="interleaved", theta=1e4, paged=True, page_size=24,
                                                       ragged=True, C=4, n=90, m_k=40, m_v=8, kernel=2, plan=3, seed=51),
    "rows_h1_dense_rope_only": RehydrateCase(H=1, row_base=False, m_k=0, m_v=0, kernel=2, plan=3, seed=52),
    "rows_h8_dense_in_place": RehydrateCase(H=8, row_base=False, in_place=True, m_k=32, m_v=16, n=70,
                                            kernel=2, plan=2, seed=53),
    "rows_layer_rank_odd_paged": RehydrateCase(L=3, layer_rank=(20, 0, 64), m_k=64, m_v=64, paged=True,
                                               kernel=2, plan=3, seed=54),
    "rows_post_rope_unit_major": RehydrateCase(H=4, post_rope=True, unit_major=True, paged=True, kernel=2, plan=3, seed=55),
    "rows_unit_major_long_blocks": RehydrateCase(H=8, C=1, L=1, n=1100, unit_major=True, paged=True, m_k=64,
                                                 m_v=64, sections=(16, 24, 24), pos_mode="grid3",
                                                 kernel=2, plan=2, seed=56),
    "rows_shared_basis_v_patch_only": RehydrateCase(H=2, shared_w=True, C=3, m_k=0, m_v=24, paged=True,
                                                    kernel=2, plan=3, seed=57),
    "rows_one_token": RehydrateCase(H=8, n=1, paged=True, kernel=2, plan=2, seed=58),
    "rows_k_only": RehydrateCase(H=8, has_v=False, row_base=False, m_k=48, n=33, kernel=2, plan=2, seed=59),
    "rows_row_base_m64": RehydrateCase(H=8, m_k=64, m_v=64, kernel=2, plan=2, seed=60),
    "rows_row_base_h4_ragged": RehydrateCase(H=4, ragged=True, C=3, n=130, m_k=16, m_v=16, kernel=2, plan=3, seed=64),
    # 8-head rows in two 4-head groups (the mid-size grids' form)
    "rows4_h8_row_base_ragged": RehydrateCase(H=8, ragged=True, C=3, n=130, m_k=64, m_v=32, kernel=3, plan=3,
                                              seed=66),
    "rows4_h8_mrope_grid_paged": RehydrateCase(H=8, n=100, sections=(16, 24, 24), pos_mode="grid3", grid_w=32,
                                               paged=True, m_k=64, m_v=64, kernel=3, plan=3, seed=67),
    "rows4_h8_in_place": RehydrateCase(H=8, row_base=False, in_place=True, m_k=16, m_v=16, n=70,
                                                  kernel=3, plan=3, seed=68),
    "rows4_h6_post_rope_paged": RehydrateCase(H=6, post_rope=True, pairing="interleaved", theta=1e4, paged=True,
                                              page_size=8, kernel=3, plan=3, seed=69),
    "rows_reloc_h8_m64": RehydrateCase(H=8, reloc=True, m_k=64, m_v=64, n=70, kernel=2, plan=2, seed=65),
    "rows4_reloc_mrope_grid_paged_post_frame": RehydrateCase(H=8, reloc=True, post_rope=True, sections=(24, 20, 20),
                                                             section_order="interleaved", pos_mode="grid3",
                                                             paged=True, m_k=32, m_v=0, kernel=3, plan=3,
                                                             seed=70),
    "rows_reloc_in_place_no_patch": RehydrateCase(H=4, reloc=True, row_base=False, in_place=True, m_k=0, m_v=0,
                                                  kernel=2, plan=3, seed=71),
    # K and V written into one tensor with their rows interleaved ([L, slot, K|V, H, D])
    "rows4_kv_interleaved_pool": RehydrateCase(H=8, paged=True, m_k=64, m_v=64, sections=(16, 24, 24),
                                               pos_mode="grid3", grid_w=32, n=100, kernel=3, plan=3, seed=72,
                                               kv_interleaved=True),
    "rows_kv_interleaved_dense": RehydrateCase(H=8, row_base=False, m_k=32, m_v=16, n=70, kernel=2, plan=2,
                                               seed=73, kv_interleaved=True),
    "per_head_kv_interleaved_row_base_ragged": RehydrateCase(H=4, ragged=True, C=3, n=130, m_k=16, m_v=8,
                                                             kernel=1, plan=1, seed=74, kv_interleaved=True),
    "rows4_reloc_kv_interleaved_in_place": RehydrateCase(H=8, reloc=True, row_base=False, in_place=True, m_k=64,
                                                         m_v=64, n=70, sections=(24, 20, 20),
                                                         section_order="interleaved", pos_mode="grid3",
                                                         kernel=3, plan=3, seed=75, kv_interleaved=True),
    "per_head_kv_interleaved_in_place": RehydrateCase(row_base=False, in_place=True, m_k=16, m_v=16, n=90,
                                                      kernel=1, plan=1, seed=76, kv_interleaved=True),
    # relocation with interleaved pairing, and with a layer of rank 0 (the patch
    # term, and with it the per-token rotation, is absent there)
    "rows4_reloc_interleaved_pairing": RehydrateCase(H=8, reloc=True, pairing="interleaved", theta=1e4,
                                                     m_k=16, m_v=16, n=50, paged=True, kernel=3, plan=3,
                                                     seed=77, kv_interleaved=True),
    "rows4_reloc_layer_rank_0_64": RehydrateCase(H=4, reloc=True, L=2, layer_rank=(0, 64), m_k=64, m_v=64,
                                                 sections=(16, 24, 24), pos_mode="grid3", n=40, kernel=3,
                                                 plan=3, seed=78),
    "per_head_explicit_paged": RehydrateCase(H=8, pos_mode="explicit", paged=True, kernel=2, plan=1, seed=61),
    "per_head_rank_72_paged": RehydrateCase(H=8, m_k=72, m_v=8, paged=True, kernel=2, plan=1, seed=62),
    "per_head_9_heads_paged": RehydrateCase(H=9, paged=True, kernel=2, plan=1, seed=63),
    # few workgroups: each walks many tiles, crossing (chunk, layer) units,
    # ragged chunk ends and the 1024-token segment limit
    "rows4_few_workgroups_paged": RehydrateCase(H=8, C=3, L=3, n=300, ragged=True, paged=True, m_k=64, m_v=32,
                                                sections=(16, 24, 24), pos_mode="grid3", grid_w=20, kernel=3,
                                                plan=3, max_workgroups=6, sched=1, seed=84),
    "rows8_two_workgroups_long_chunk": RehydrateCase(H=8, C=2, L=2, n=1500, unit_major=True, m_k=16, m_v=16,
                                                     kernel=2, plan=2, max_workgroups=2, sched=1, seed=85),
    "rows4_reloc_few_workgroups": RehydrateCase(H=4, C=3, L=2, n=200, reloc=True, m_k=64, m_v=64, kernel=3,
                                                plan=3, max_workgroups=3, sched=1, seed=86),
    "rows4_one_workgroup_per_lane": RehydrateCase(H=8, C=2, L=3, n=130, m_k=32, m_v=0, paged=True, kernel=3,
                                                  plan=3, max_workgroups=4, sched=1, seed=87),
    # the block schedule (one workgroup per token block, handed out by the
    # hardware) on small shapes: blocks shrink to 64 tokens here, so units
    # split into several blocks, the last one short, and ragged chunks end
    # inside a block
    "rows4_blocks_paged_ragged_grid": RehydrateCase(H=8, C=3, L=3, n=300, ragged=True, paged=True, m_k=64, m_v=32,
                                                    sections=(16, 24, 24), pos_mode="grid3", grid_w=20, kernel=3,
                                                    plan=3, schedule=2, sched=2, seed=92),
    "rows8_blocks_long_chunk": RehydrateCase(H=8, C=2, L=2, n=1500, unit_major=True, m_k=16, m_v=16, kernel=2,
                                             plan=2, schedule=2, sched=2, seed=93),
    "rows4_blocks_reloc_kv_in_place": RehydrateCase(H=8, reloc=True, row_base=False, in_place=True, m_k=64, m_v=64,
                                                    n=200, sections=(24, 20, 20), section_order="interleaved",
                                                    pos_mode="grid3", kernel=3, plan=3, schedule=2, sched=2,
                                                    seed=94, kv_interleaved=True),
    "rows4_blocks_layer_rank_row_base": RehydrateCase(H=8, L=3, layer_rank=(0, 64, 20), m_k=64, m_v=64, n=130,
                                                      ragged=True, C=3, kernel=3, plan=3, schedule=2, sched=2,
                                                      seed=95),
    "rows4_blocks_reloc_post_frame_paged": RehydrateCase(H=4, reloc=True, post_rope=True, paged=True, m_k=32,
                                                         m_v=0, n=90, pairing="interleaved", theta=1e4, kernel=3,
                                                         plan=3, schedule=2, sched=2, seed=96),
    "rows4_blocks_kv_interleaved_pool_rank_0": RehydrateCase(H=8, paged=True, m_k=0, m_v=0, n=100, kernel=3,
                                                             plan=3, schedule=2, sched=2, seed=97,
                                                             kv_interleaved=True),
    "rows4_auto_small_is_persistent": RehydrateCase(H=8, paged=True, m_k=16, m_v=16, n=100, kernel=3, plan=3,
                                                    sched=1, seed=98),
    "per_head_few_workgroups_mla_band": RehydrateCase(D=576, H=1, C=2, L=3, n=300, rope_dim=64, rope_offset=512,
                                                      pairing="interleaved", theta=1e4, patch=(0, 512), m_k=32,
                                                      m_pe=8, has_v=False, kernel=1, plan=1, max_workgroups=3,
                                                      seed=88),
    "per_head_few_workgroups_layer_rank": RehydrateCase(H=3, L=4, layer_rank=(0, 64, 5, 33), m_k=64, m_v=40,
                                                        ragged=True, C=3, n=150, paged=True, kernel=1, plan=1,
                                                        max_workgroups=5, seed=89),
    "per_head_one_workgroup": RehydrateCase(H=2, C=2, L=2, n=90, sections=(16, 24, 24), pos_mode="grid3", grid_w=9,
                                            kernel=1, plan=1, max_workgroups=1, seed=90),
    "per_head_reloc_two_workgroups": RehydrateCase(H=5, C=2, L=2, n=120, reloc=True, m_k=16, m_v=24, kernel=1,
                                                   plan=1, max_workgroups=2, seed=91),
    # relocation above rank 64 on the per-head kernel: the two-rotation form
    # R(p)(R(delta - p) K + U W) (rank steps of 4 x 32), both frames
    "relocate_rank_72_per_head": RehydrateCase(reloc=True, m_k=72, m_v=8, n=70, kernel=1, plan=1, seed=80),
    "relocate_rank_72_post_frame_paged": RehydrateCase(reloc=True, m_k=72, m_v=72, post_rope=True, paged=True,
                                                       pairing="interleaved", theta=1e4, n=50, kernel=1, plan=1,
                                                       seed=81),
    "relocate_rank_128_per_head": RehydrateCase(reloc=True, m_k=128, m_v=128, n=48, C=1, L=1, H=2, kernel=1, plan=1,
                                                seed=82),
    "relocate_rank_128_post_frame_mrope": RehydrateCase(reloc=True, m_k=128, m_v=100, post_rope=True,
                                                        sections=(16, 24, 24), pos_mode="grid3", grid_w=8, n=40,
                                                        C=2, L=1, H=2, kernel=1, plan=1, seed=83),
}


@pytest.mark.parametrize("name", sorted(REHYDRATE_CASES))
def test_rehydrate_matches_oracle(device, name):
    print(f"[case] rehydrate {name}", flush=True)
    run_rehydrate(REHYDRATE_CASES[name], device)


def test_rehydrate_identity_is_bit_exact(device):
    """Position 0 with no patch reproduces the stored bits at the page slots."""
    import paper_2606_23581_amd as km
    import torch

    print("[case] rehydrate identity", flush=True)
    rng = np.random.default_rng(30)
    C, L, n, H, D, P = 3, 2, 45, 2, 128, 16
    K = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)
    pages = (n + P - 1) // P
    pt = rng.permutation(C * pages + 2)[: C * pages].reshape(C, pages).astype(np.int32)
    slots = (C * pages + 2) * P
    for pairing in ("neox", "interleaved"):
        pool = dev(np.full((L, slots, H, D), SENTINEL, np.uint16), device)
        # every token at position 0 (explicit positions; a linear p0 = 0 puts token i at i)
        km.rehydrate(dev(K, device), pool, rope=km.RopeSpec(theta=1e4, rope_dim=128, pairing=pairing),
                     pos_mode=km.POS_EXPLICIT, explicit_pos=dev_i32(np.zeros((C, n, 3)), device),
                     page_table=dev_i32(pt, device), page_size=P, n_pool_pages=C * pages + 2)
        torch.cuda.synchronize()
        out = bits(pool)
        for c in range(C):
            for i in range(n):
                s = ref.paged_slot(pt[c], i, P)
                assert np.array_equal(out[:, s], K[c, :, i]), (pairing, c, i)


@pytest.mark.parametrize("mla", [False, True])
def test_rehydrate_exactly_in_place(device, mla):
    """Keys and values rebuilt in their own storage (same base and strides):
    ragged chunks, the tokens past each chunk's count keep their bits; for MLA
    the latent and the rope band are two planes in place on one tensor."""
    import paper_2606_23581_amd as km
    import torch

    print(f"[case] rehydrate in place mla={mla}", flush=True)
    rng = np.random.default_rng(31 + mla)
    C, L, n = 3, 2, 70
    H, D = (1, 576) if mla else (2, 128)
    K = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)
    V = None if mla else synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)
    pd = 512 if mla else D
    m = 16
    Uk = synth.randn_bf16_numpy((C, L, H, n, m), 0.1, rng)
    Wk = synth.randn_bf16_numpy((C, L, H, m, pd), 0.1, rng)
    n_c = np.array([n, 33, 0], dtype=np.int32)
    p0 = rng.integers(0, 30000, size=C)
    pos = np.repeat(p0[:, None], 3, axis=1).astype(np.int32)
    if mla:
        rs = km.RopeSpec(theta=1e4, rope_dim=64, rope_offset=512, pairing="interleaved")
    else:
        rs = km.RopeSpec(theta=1e6, rope_dim=128)
    kt = dev(K, device)
    kw = dict(rope=rs, chunk_pos=dev_i32(pos, device), chunk_tokens=dev_i32(n_c, device),
              u_k=dev(Uk, device), w_k=dev(Wk, device), k_patch=(0, pd))
    if mla:
        Upe = synth.randn_bf16_numpy((C, L, H, n, 8), 0.1, rng)
        Wpe = synth.randn_bf16_numpy((C, L, H, 8, 64), 0.1, rng)
        kw.update(u_pe=dev(Upe, device), w_pe=dev(Wpe, device))
        km.rehydrate(kt, kt, **kw)
    else:
        Uv = synth.randn_bf16_numpy((C, L, H, n, m), 0.1, rng)
        Wv = synth.randn_bf16_numpy((C, L, H, m, D), 0.1, rng)
        vt = dev(V, device)
        km.rehydrate(kt, kt, v_in=vt, v_out=vt, u_v=dev(Uv, device), w_v=dev(Wv, device), v_patch=(0, D), **kw)
    torch.cuda.synchronize()
    kb = bits(kt)
    vb = None if mla else bits(vt)
    orope = oracle_rope(rs)
    for c in range(C):
        nc = int(n_c[c])
        assert np.array_equal(kb[c, :, nc:], K[c, :, nc:]), "tokens past the chunk's count were written"
        if not mla:
            assert np.array_equal(vb[c, :, nc:], V[c, :, nc:])
        p3 = ref.positions_linear(int(p0[c]), nc)
        for l in range(L):
            for h in range(H):
                u = ref.bf16_to_f64(Uk[c, l, h, :nc])
                w = ref.bf16_to_f64(Wk[c, l, h])
                if mla:
                    wf = np.zeros((m + 8, D))
                    wf[:m, :512] = w
                    wf[m:, 512:] = ref.bf16_to_f64(Wpe[c, l, h])
                    u, w = np.concatenate([u, ref.bf16_to_f64(Upe[c, l, h, :nc])], axis=1), wf
                want = ref.rehydrate_k(ref.bf16_to_f64(K[c, l, :nc, h]), u, w, orope, p3)
                assert_close(kb[c, l, :nc, h], want, f"in-place K c{c} l{l} h{h}")
                if not mla:
                    want = ref.rehydrate_v(ref.bf16_to_f64(V[c, l, :nc, h]), ref.bf16_to_f64(Uv[c, l, h, :nc]),
                                           ref.bf16_to_f64(Wv[c, l, h]))
                    assert_close(vb[c, l, :nc, h], want, f"in-place V c{c} l{l} h{h}")


def test_rehydrate_empty_call_writes_nothing(device):
    import paper_2606_23581_amd as km
    import torch

    print("[case] rehydrate empty", flush=True)
    K = dev(np.zeros((2, 1, 0, 2, 128), np.uint16), device)
    out = dev(np.full((2, 1, 4, 2, 128), SENTINEL, np.uint16), device)
    km.rehydrate(K, out, rope=km.RopeSpec(theta=1e4, rope_dim=128), chunk_pos=dev_i32(np.zeros((2, 3)), device))
    torch.cuda.synchronize()
    assert np.all(bits(out) == SENTINEL)


@pytest.mark.parametrize("kernel", ["per_head", "row_group"])
def test_rehydrate_bad_page_is_flagged_not_written(device, kernel):
    """A page number outside the pool is skipped by the kernel and flagged
    (explicit positions take the per-head kernel, linear ones the row-group
    kernel)."""
    import paper_2606_23581_amd as km
    import torch

    print(f"[case] rehydrate bad page {kernel}", flush=True)
    rng = np.random.default_rng(31)
    C, L, n, H, D, P = 1, 1, 32, 2, 128, 16
    K = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)
    pt = np.array([[1, 7]], dtype=np.int32)       # page 7 is outside a 3-page pool
    pool = dev(np.full((L, 3 * P, H, D), SENTINEL, np.uint16), device)
    status = dev_i32(np.zeros(1), device)
    rs = km.RopeSpec(theta=1e4, rope_dim=128)
    if kernel == "per_head":
        pos = dict(pos_mode=km.POS_EXPLICIT, explicit_pos=dev_i32(np.zeros((C, n, 3)), device))
    else:
        pos = dict(pos_mode=km.POS_LINEAR, chunk_pos=dev_i32(np.zeros((C, 3)), device))
    prep = km.prepare_rehydrate(dev(K, device), pool, rope=rs, page_table=dev_i32(pt, device), page_size=P,
                                n_pool_pages=3, status=status, kernel=km.KERNEL_ROW_GROUP, **pos)
    assert km.rehydrate_plan(prep) == (km.PLAN_PER_HEAD if kernel == "per_head" else km.PLAN_ROW_GROUP4)
    prep.launch()
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) & km.STATUS_BAD_PAGE
    out = bits(pool)
    if kernel == "per_head":
        assert np.array_equal(out[0, P:2 * P], K[0, 0, :P])     # page 1 written (position 0: identity)
    else:
        for h in range(H):                                      # page 1 holds tokens 0..15 at positions 0..15
            want = ref.rehydrate_k(ref.bf16_to_f64(K[0, 0, :P, h]), None, None, oracle_rope(rs),
                                   ref.positions_linear(0, P))
            assert_close(out[0, P:2 * P, h], want, f"page 1 h{h}")
    assert np.all(out[0, :P] == SENTINEL) and np.all(out[0, 2 * P:] == SENTINEL)


# ---------------------------------------------------------------------------
# shift
# ---------------------------------------------------------------------------

SHIFT_CASES = {
    "interleaved_5d": dict(pairing="interleaved", theta=1e4, rope_dim=128, D=128, layout="5d"),
    "neox_rowbase": dict(pairing="neox", theta=1e6, rope_dim=128, D=128, layout="rowbase"),
    "neox_partial_band": dict(pairing="neox", theta=1e6, rope_dim=64, rope_offset=64, D=128, layout="5d"),
    "mla_band": dict(pairing="interleaved", theta=1e4, rope_dim=64, rope_offset=512, D=576, H=1, layout="5d"),
    "mrope_sections_paged": dict(pairing="neox", theta=1e6, rope_dim=128, D=128, sections=(16, 24, 24),
                                 layout="paged"),
    "interleaved_rd48_ragged": dict(pairing="interleaved", theta=1e4, rope_dim=48, rope_offset=16, D=64,
                                    layout="5d", ragged=True),
}


@pytest.mark.parametrize("name", sorted(SHIFT_CASES))
def test_shift_matches_oracle(device, name):
    import paper_2606_23581_amd as km
    import torch

    print(f"[case] shift {name}", flush=True)
    cfg = dict(SHIFT_CASES[name])
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    C, L, n = 3, 2, 70
    H = cfg.get("H", 3)
    D = cfg["D"]
    rs = km.RopeSpec(theta=cfg["theta"], rope_dim=cfg["rope_dim"], pairing=cfg["pairing"],
                     rope_offset=cfg.get("rope_offset", 0), sections=cfg.get("sections"))
    orope = oracle_rope(rs)
    delta = rng.integers(-9000, 9000, size=(C, 3)).astype(np.int32)
    if cfg.get("sections") is None:
        delta[:, 1:] = delta[:, :1]
    n_c = rng.integers(0, n + 1, size=C).astype(np.int32) if cfg.get("ragged") else np.full(C, n, np.int32)
    status = dev_i32(np.zeros(1), device)
    layout = cfg["layout"]
    if layout == "5d":
        Kb = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)
        kt = dev(Kb, device)
        km.shift(kt, dev_i32(delta, device), rope=rs, status=status,
                 chunk_tokens=dev_i32(n_c, device) if cfg.get("ragged") else None)
        torch.cuda.synchronize()
        out = bits(kt)
        for c in range(C):
            for l in range(L):
                for h in range(H):
                    nc = int(n_c[c])
                    want = ref.shift_k(ref.bf16_to_f64(Kb[c, l, :nc, h]), orope, delta[c])
                    assert_close(out[c, l, :nc, h], want, f"c{c} l{l} h{h}")
                    assert np.array_equal(out[c, l, nc:, h], Kb[c, l, nc:, h])
        band = slice(rs.rope_offset, rs.rope_offset + rs.rope_dim)
        outside = np.ones(D, bool)
        outside[band] = False
        assert np.array_equal(out[..., outside], Kb[..., outside]), "columns outside the band changed"
    else:
        P = 16
        pages = (n + P - 1) // P
        rows = C * n + 11 if layout == "rowbase" else (C * pages + 2) * P
        Wb = synth.randn_bf16_numpy((L, rows, H, D), 1.0, rng)
        wt = dev(Wb, device)
        if layout == "rowbase":
            rb = (rng.permutation(C) * n + 5).astype(np.int32)
            km.shift(wt, dev_i32(delta, device), rope=rs, n_chunks=C, n_tokens=n,
                     row_base=dev_i32(rb, device), status=status)
            dst = [rb[c] + np.arange(n) for c in range(C)]
        else:
            npp = rows // P
            pt = rng.permutation(npp)[: C * pages].reshape(C, pages).astype(np.int32)
            km.shift(wt, dev_i32(delta, device), rope=rs, n_chunks=C, n_tokens=n,
                     page_table=dev_i32(pt, device), page_size=P, n_pool_pages=npp, status=status)
            dst = [np.array([ref.paged_slot(pt[c], i, P) for i in range(n)]) for c in range(C)]
        torch.cuda.synchronize()
        out = bits(wt)
        touched = np.zeros((rows,), bool)
        for c in range(C):
            touched[dst[c]] = True
            for l in range(L):
                for h in range(H):
                    want = ref.shift_k(ref.bf16_to_f64(Wb[l, dst[c], h]), orope, delta[c])
                    assert_close(out[l, dst[c], h], want, f"c{c} l{l} h{h}")
        assert np.array_equal(out[:, ~touched], Wb[:, ~touched]), "rows of other chunks changed"
    assert int(status.cpu()[0]) == 0


def test_shift_round_trip(device):
    """Shift by delta then -delta returns the keys within two bf16 roundings."""
    import paper_2606_23581_amd as km
    import torch

    print("[case] shift round trip", flush=True)
    rng = np.random.default_rng(40)
    Kb = synth.randn_bf16_numpy((2, 2, 64, 4, 128), 1.0, rng)
    kt = dev(Kb, device)
    rs = km.RopeSpec(theta=1e4, rope_dim=128, pairing="interleaved")
    d = np.array([[-512] * 3, [3000] * 3], dtype=np.int32)
    km.shift(kt, dev_i32(d, device), rope=rs)
    km.shift(kt, dev_i32(-d, device), rope=rs)
    torch.cuda.synchronize()
    got = ref.bf16_to_f64(bits(kt))
    want = ref.bf16_to_f64(Kb)
    assert np.max(np.abs(got - want) / np.maximum(1, np.abs(want))) <= 2 * TOL


# ---------------------------------------------------------------------------
# scatter
# ---------------------------------------------------------------------------

def test_scatter_is_bit_exact(device):
    import paper_2606_23581_amd as km
    import torch

    print("[case] scatter", flush=True)
    rng = np.random.default_rng(50)
    C, L, n, H, D, P = 4, 3, 53, 2, 128, 16
    src = rng.integers(0, 1 << 16, size=(C, L, n, H, D)).astype(np.uint16)
    pages = (n + P - 1) // P
    npp = C * pages + 7
    pt = rng.permutation(npp)[: C * pages].reshape(C, pages).astype(np.int32)
    n_c = np.array([n, 0, 17, 40], dtype=np.int32)
    pool = dev(np.full((L, npp * P, H, D), SENTINEL, np.uint16), device)
    status = dev_i32(np.zeros(1), device)
    km.scatter_paged(dev(src, device), pool, dev_i32(pt, device), page_size=P, n_pool_pages=npp,
                     chunk_tokens=dev_i32(n_c, device), status=status)
    torch.cuda.synchronize()
    out = bits(pool)
    want = np.full((L, npp * P, H, D), SENTINEL, np.uint16)
    for c in range(C):
        for l in range(L):
            want[l] = ref.scatter_paged(src[c, l, : n_c[c]], pt[c], P, want[l])
    assert np.array_equal(out, want)
    assert int(status.cpu()[0]) == 0


def test_gather_is_bit_exact_inverse(device):
    """Gather reads the page-table slots back into dense rows bit for bit;
    scatter then gather returns the original rows."""
    import paper_2606_23581_amd as km
    import torch

    print("[case] gather", flush=True)
    rng = np.random.default_rng(51)
    C, L, n, H, D, P = 3, 2, 45, 2, 128, 16
    pages = (n + P - 1) // P
    npp = C * pages + 3
    pt = rng.permutation(npp)[: C * pages].reshape(C, pages).astype(np.int32)
    pool_np = rng.integers(0, 1 << 16, size=(L, npp * P, H, D)).astype(np.uint16)
    rows = dev(np.full((C, L, n, H, D), SENTINEL, np.uint16), device)
    km.gather_paged(rows, dev(pool_np, device), dev_i32(pt, device), page_size=P, n_pool_pages=npp)
    torch.cuda.synchronize()
    got = bits(rows)
    for c in range(C):
        for i in range(n):
            assert np.array_equal(got[c, :, i], pool_np[:, ref.paged_slot(pt[c], i, P)])
    pool2 = dev(np.zeros((L, npp * P, H, D), np.uint16), device)
    km.scatter_paged(rows, pool2, dev_i32(pt, device), page_size=P, n_pool_pages=npp)
    back = dev(np.zeros((C, L, n, H, D), np.uint16), device)
    km.gather_paged(back, pool2, dev_i32(pt, device), page_size=P, n_pool_pages=npp)
    torch.cuda.synchronize()
    assert np.array_equal(bits(back), got)


def test_conditioning_switch(device):
    """App. E: the clean view is the canonical at its position (no patch);
    re-conditioning adds R(p) U W in place (a relocation by delta = 0); turning
    it off again restores the clean view bit for bit."""
    import paper_2606_23581_amd as km
    import torch

    print("[case] conditioning switch", flush=True)
    rng = np.random.default_rng(52)
    C, L, n, H, D, m = 2, 2, 40, 2, 128, 16
    K = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)
    U = synth.randn_bf16_numpy((C, L, H, n, m), 0.1, rng)
    W = synth.randn_bf16_numpy((C, L, H, m, D), 0.1, rng)
    rs = km.RopeSpec(theta=1e6, rope_dim=128)
    p0 = np.array([[300] * 3, [7000] * 3], dtype=np.int32)
    clean = dev(np.zeros((C, L, n, H, D), np.uint16), device)
    km.rehydrate(dev(K, device), clean, rope=rs, chunk_pos=dev_i32(p0, device))
    conditioned = clean.clone()
    km.rehydrate(conditioned, conditioned, rope=rs, chunk_pos=dev_i32(p0, device), u_k=dev(U, device),
                 w_k=dev(W, device), delta=dev_i32(np.zeros((C, 3)), device))
    clean2 = dev(np.zeros((C, L, n, H, D), np.uint16), device)
    km.rehydrate(dev(K, device), clean2, rope=rs, chunk_pos=dev_i32(p0, device))
    torch.cuda.synchronize()
    assert np.array_equal(bits(clean2), bits(clean))
    orope = oracle_rope(rs)
    cb = bits(conditioned)
    for c in range(C):
        for l in range(L):
            for h in range(H):
                want = ref.rehydrate_k(ref.bf16_to_f64(K[c, l, :, h]), ref.bf16_to_f64(U[c, l, h]),
                                       ref.bf16_to_f64(W[c, l, h]), orope, ref.positions_linear(int(p0[c, 0]), n))
                got = ref.bf16_to_f64(cb[c, l, :, h])
                assert np.max(np.abs(got - want) / np.maximum(1, np.abs(want))) <= 2 * TOL


def test_scatter_bad_page_is_flagged(device):
    import paper_2606_23581_amd as km
    import torch

    print("[case] scatter bad page", flush=True)
    src = np.arange(2 * 16 * 8, dtype=np.uint16).reshape(1, 1, 32, 8)
    pool = dev(np.full((1, 32, 8), SENTINEL, np.uint16), device)
    status = dev_i32(np.zeros(1), device)
    km.scatter_paged(dev(src, device), pool, dev_i32([[1, -3]], device), page_size=16, n_pool_pages=2,
                     status=status)
    torch.cuda.synchronize()
    out = bits(pool)
    assert int(status.cpu()[0]) & km.STATUS_BAD_PAGE
    assert np.array_equal(out[0, 16:], src[0, 0, :16])
    assert np.all(out[0, :16] == SENTINEL)


# ---------------------------------------------------------------------------
# compile-side patch forming
# ---------------------------------------------------------------------------

def _check_patch(delta, Ub, Wb, sg, m, tag):
    """One unit's patch against the fp64 truncated SVD: product, singular
    values, W's orthonormal rows and the Eckart-Young residual.  U and W are
    stored in bf16 (unit roundoff 2^-8 each), so the product's relative
    Frobenius error is bounded by ~2 * 2^-8 plus the fp32 subspace error; the
    bound used is 2^-6."""
    Dl = delta.astype(np.float64)
    Ur, Wr, S = ref.form_patch(Dl, m)
    Ug, Wg = ref.bf16_to_f64(Ub), ref.bf16_to_f64(Wb)
    prod_ref = Ur @ Wr
    rel = np.linalg.norm(Ug @ Wg - prod_ref) / np.linalg.norm(prod_ref)
    assert rel <= 2.0 ** -6, (tag, rel)
    assert np.max(np.abs(sg - S[:m]) / S[:m]) <= 1e-4, (tag, sg[:4], S[:4])
    assert np.max(np.abs(Wg @ Wg.T - np.eye(m))) <= 2.0 ** -6, tag
    opt = np.linalg.norm(Dl - prod_ref)
    got = np.linalg.norm(Dl - Ug @ Wg)
    assert got <= opt + 2.0 ** -6 * np.linalg.norm(prod_ref), (tag, got, opt)


@pytest.mark.parametrize("n,d,m", [(100, 128, 16), (1024, 128, 64), (37, 64, 8), (50, 36, 1), (64, 32, 32),
                                   (7, 4, 2), (130, 16, 16), (2000, 128, 128), (300, 100, 40)])
def test_form_patch_matches_svd(device, n, d, m):
    """Planted deficits with a spectral gap at m (rank-m signal + small noise),
    through both eigensolvers (the tridiagonal default and block Jacobi): U W
    must match the fp64 truncated SVD's product, the singular values the fp64
    ones, W's rows must be orthonormal and the residual Eckart-Young's."""
    import paper_2606_23581_amd as km
    import torch

    rng = np.random.default_rng(n * 1000 + d + m)
    C, L, H = 2, 2, 2
    delta = np.empty((C, L, H, n, d), np.float32)
    for idx in np.ndindex(C, L, H):
        A = np.linalg.qr(rng.standard_normal((n, m)))[0]
        B = np.linalg.qr(rng.standard_normal((d, m)))[0]
        sig = np.linspace(10.0, 2.0, m)
        delta[idx] = (A * sig) @ B.T + 0.01 * rng.standard_normal((n, d))
    dt = torch.from_numpy(delta).to(device)
    for sweeps in (0, 12):
        print(f"[case] form_patch n{n} d{d} m{m} sweeps {sweeps}", flush=True)
        U = torch.zeros((C, L, H, n, m), dtype=torch.bfloat16, device=device)
        W = torch.zeros((C, L, H, m, d), dtype=torch.bfloat16, device=device)
        sigma = torch.zeros((C, L, H, m), dtype=torch.float32, device=device)
        done = torch.full((C, L, H), -1, dtype=torch.int32, device=device)
        km.form_patch(dt, U, W, sigma=sigma, sweeps=sweeps, sweeps_done=done)
        torch.cuda.synchronize()
        if sweeps == 0:
            assert (done == 0).all(), done.cpu().numpy()        # no Jacobi sweep with the tridiagonal solver
        else:
            # Jacobi converged within 12 sweeps, after at least one
            assert ((done >= 1) & (done < 12)).all(), done.cpu().numpy()
        Ub, Wb, sg = bits(U), bits(W), sigma.cpu().numpy()
        for idx in np.ndindex(C, L, H):
            _check_patch(delta[idx], Ub[idx], Wb[idx], sg[idx], m, (sweeps,) + idx)
    capped = torch.full((C, L, H), -1, dtype=torch.int32, device=device)
    km.form_patch(dt, torch.empty((C, L, H, n, m), dtype=torch.bfloat16, device=device),
                  torch.empty((C, L, H, m, d), dtype=torch.bfloat16, device=device), sweeps=1, sweeps_done=capped)
    torch.cuda.synchronize()
    assert (capped == 1).all()


@pytest.mark.parametrize("sweeps", [0, 12])
def test_form_patch_degenerate_spectra(device, sweeps):
    """Spectra where the eigensolvers meet multiple or zero eigenvalues:
    the patch is still the truncation wherever that is unique, and W's rows
    stay orthonormal.
      * zero deficit: U = 0, sigma = 0;
      * m equal singular values over noise-free rank m: U W = Delta;
      * identical columns (rank 1, a (d-1)-fold zero eigenvalue): U W = Delta;
      * a decaying spectrum without a gap at m, s_k = (1 + k)^(-1/4), the
        shape of the benchmark's deficits: the Eckart-Young residual."""
    import paper_2606_23581_amd as km
    import torch

    print(f"[case] form_patch degenerate spectra sweeps {sweeps}", flush=True)
    rng = np.random.default_rng(4242)
    cases = []
    cases.append(("zero", np.zeros((64, 32)), 8))
    Aq = np.linalg.qr(rng.standard_normal((100, 8)))[0]
    Bq = np.linalg.qr(rng.standard_normal((32, 8)))[0]
    cases.append(("equal", (Aq * 5.0) @ Bq.T, 8))
    X = rng.standard_normal((50, 1))
    cases.append(("identical_columns", np.repeat(X, 16, axis=1), 4))
    A = rng.standard_normal((1024, 128))
    Q = np.linalg.qr(rng.standard_normal((128, 128)))[0]
    cases.append(("decaying", (A * (1.0 + np.arange(128)) ** -0.25) @ Q, 64))
    for name, D, m in cases:
        n, d = D.shape
        D32 = D.astype(np.float32)
        dt = torch.from_numpy(D32.reshape(1, 1, 1, n, d)).to(device)
        U = torch.zeros((1, 1, 1, n, m), dtype=torch.bfloat16, device=device)
        W = torch.zeros((1, 1, 1, m, d), dtype=torch.bfloat16, device=device)
        sigma = torch.full((1, 1, 1, m), -1.0, dtype=torch.float32, device=device)
        km.form_patch(dt, U, W, sigma=sigma, sweeps=sweeps)
        torch.cuda.synchronize()
        Ug, Wg, sg = ref.bf16_to_f64(bits(U)[0, 0, 0]), ref.bf16_to_f64(bits(W)[0, 0, 0]), sigma.cpu().numpy()[0, 0, 0]
        assert np.all(np.isfinite(Ug)) and np.all(np.isfinite(Wg)) and np.all(np.isfinite(sg)), name
        assert np.max(np.abs(Wg @ Wg.T - np.eye(m))) <= 2.0 ** -6, name
        Dl = D32.astype(np.float64)
        if name == "zero":
            assert np.all(Ug == 0) and np.all(sg == 0), name
        elif name in ("equal", "identical_columns"):
            rel = np.linalg.norm(Ug @ Wg - Dl) / np.linalg.norm(Dl)
            assert rel <= 2.0 ** -6, (name, rel)
            # the square root of an fp32 eigenvalue of G near zero carries an
            # absolute error ~ sqrt(d u) sigma_1 (u = 2^-24): 2^-9 sigma_1 at d <= 32
            S = np.linalg.svd(Dl, compute_uv=False)[:m]
            assert np.max(np.abs(sg - S)) <= 2.0 ** -9 * S[0], (name, sg, S)
        else:
            Ur, Wr, S = ref.form_patch(Dl, m)
            prod_ref = Ur @ Wr
            opt = np.linalg.norm(Dl - prod_ref)
            got = np.linalg.norm(Dl - Ug @ Wg)
            assert got <= opt + 2.0 ** -6 * np.linalg.norm(prod_ref), (name, got, opt)
            assert np.max(np.abs(sg - S[:m]) / S[:m]) <= 1e-4, (name, sg[:4], S[:4])


@pytest.mark.parametrize("K,n,d,m", [(3, 200, 128, 16), (6, 64, 64, 8), (1, 90, 128, 32)])
def test_orbit_patch_matches_reference(device, K, n, d, m):
    """Orbit patch (Sec. 5, reorder): the K orderings' deficits share a
    rank-m core with a gap; the GPU's patch must match the fp64 truncation of
    the orbit mean, and a one-member orbit must give the plain call's bits."""
    import paper_2606_23581_amd as km
    import torch

    print(f"[case] orbit_patch K{K} n{n} d{d} m{m}", flush=True)
    rng = np.random.default_rng(K * 100 + m)
    C, L, H = 2, 1, 3
    deltas = np.empty((K, C, L, H, n, d), np.float32)
    for idx in np.ndindex(C, L, H):
        A = np.linalg.qr(rng.standard_normal((n, m)))[0]
        B = np.linalg.qr(rng.standard_normal((d, m)))[0]
        core = (A * np.linspace(10.0, 3.0, m)) @ B.T
        for k in range(K):
            deltas[(k,) + idx] = core + 0.05 * rng.standard_normal((n, d))
    dt = torch.from_numpy(deltas).to(device)
    U = torch.zeros((C, L, H, n, m), dtype=torch.bfloat16, device=device)
    W = torch.zeros((C, L, H, m, d), dtype=torch.bfloat16, device=device)
    km.form_patch(dt, U, W)
    torch.cuda.synchronize()
    Ub, Wb = bits(U), bits(W)
    for idx in np.ndindex(C, L, H):
        Ur, Wr, _ = ref.orbit_patch(deltas[(slice(None),) + idx].astype(np.float64), m)
        prod_ref = Ur @ Wr
        got = ref.bf16_to_f64(Ub[idx]) @ ref.bf16_to_f64(Wb[idx])
        rel = np.linalg.norm(got - prod_ref) / np.linalg.norm(prod_ref)
        assert rel <= 2.0 ** -6, (idx, rel)
    if K == 1:
        U2 = torch.zeros_like(U)
        W2 = torch.zeros_like(W)
        km.form_patch(dt[0], U2, W2)
        torch.cuda.synchronize()
        assert np.array_equal(bits(U2), Ub) and np.array_equal(bits(W2), Wb)


@pytest.mark.parametrize("kernel", [1, 3])
def test_form_patch_then_rehydrate_in_both_frames(device, kernel):
    """The compile step feeds the serve step (App. A): a key deficit is
    planted, its patch formed on the GPU and applied by kamera_rehydrate.

    * rotated frame (App. A takes the deficit against R(p) K): a rank-m
      Delta_post, formed as is and applied with KAMERA_PATCH_POST_ROPE,
      rebuilds R(p) K + Delta_post;
    * stored frame: a deficit that is rank m before rotation, handed over as
      App. A would see it (R(p) Delta_pre) and turned back per token by
      R(-p_i) before forming, applied with KAMERA_PATCH_PRE_ROPE, rebuilds
      R(p)(K + Delta_pre);
    * rotated-frame factors applied in the stored frame rotate the patch
      twice and miss the target.

    Each output is checked element by element against the oracle run on the
    GPU-formed factors (the parity bar), and against the target keys within
    2 x 2^-7 (the output's bf16 rounding plus that of the two factors)."""
    import paper_2606_23581_amd as km
    import torch

    print(f"[case] form_patch -> rehydrate frames kernel {kernel}", flush=True)
    rng = np.random.default_rng(4242 + kernel)
    C, L, H, n, D, m = 2, 2, 4, 256, 128, 16
    rs = km.RopeSpec(theta=1e6, rope_dim=D, pairing="neox")
    orope = oracle_rope(rs)
    p0 = rng.integers(0, 30000, size=C)
    pos = np.zeros((C, 3), np.int32)
    pos[:, 0] = p0
    pos3 = [ref.positions_linear(int(p0[c]), n) for c in range(C)]
    K = synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng)

    def planted():
        A = np.linalg.qr(rng.standard_normal((n, m)))[0]
        B = np.linalg.qr(rng.standard_normal((D, m)))[0]
        return (A * np.linspace(12.0, 4.0, m)) @ B.T          # entries ~0.3

    d_post = np.empty((C, L, H, n, D))
    d_pre = np.empty((C, L, H, n, D))
    d_pre_rotated = np.empty((C, L, H, n, D))                 # what App. A would hand over
    for c, l, h in np.ndindex(C, L, H):
        d_post[c, l, h] = planted()
        d_pre[c, l, h] = planted()
        d_pre_rotated[c, l, h] = ref.rotate(d_pre[c, l, h], orope, ref.rope_angles(orope, pos3[c]))
    # the caller's conversion to the stored frame: R(-p_i) per token
    d_back = np.empty_like(d_pre_rotated)
    for c, l, h in np.ndindex(C, L, H):
        d_back[c, l, h] = ref.rotate(d_pre_rotated[c, l, h], orope, ref.rope_angles(orope, -pos3[c]))

    kin = dev(K, device)
    cpos = dev_i32(pos, device)

    def form(deficit):
        U = torch.zeros((C, L, H, n, m), dtype=torch.bfloat16, device=device)
        W = torch.zeros((C, L, H, m, D), dtype=torch.bfloat16, device=device)
        km.form_patch(torch.from_numpy(deficit.astype(np.float32)).to(device), U, W)
        return U, W

    def apply(U, W, frame):
        out = dev(np.full((C, L, n, H, D), SENTINEL, np.uint16), device)
        km.rehydrate(kin, out, rope=rs, chunk_pos=cpos, u_k=U, w_k=W, patch_frame=frame, kernel=kernel)
        torch.cuda.synchronize()
        return bits(out), bits(U), bits(W)

    cases = {
        "rotated frame, POST_ROPE": (d_post, km.PATCH_POST_ROPE, True),
        "stored frame, PRE_ROPE": (d_back, km.PATCH_PRE_ROPE, False),
    }
    for what, (deficit, frame, post) in cases.items():
        got, Ub, Wb = apply(*form(deficit), frame)
        for c, l, h in np.ndindex(C, L, H):
            Kf = ref.bf16_to_f64(K[c, l, :, h])
            Ug, Wg = ref.bf16_to_f64(Ub[c, l, h]), ref.bf16_to_f64(Wb[c, l, h])
            want = ref.rehydrate_k(Kf, Ug, Wg, orope, pos3[c], patch_after_rope=post)
            assert_close(got[c, l, :, h], want, f"{what} c{c} l{l} h{h}")
            rotated = ref.rehydrate_k(Kf, None, None, orope, pos3[c])
            target = rotated + (d_post[c, l, h] if post else d_pre_rotated[c, l, h])
            err = np.abs(ref.bf16_to_f64(got[c, l, :, h]) - target) / np.maximum(1.0, np.abs(target))
            assert err.max() <= 2 * TOL, (what, c, l, h, float(err.max()))
    # the hazard the frame flag guards against
    got, _, _ = apply(*form(d_post), km.PATCH_PRE_ROPE)
    worst = 0.0
    for c, l, h in np.ndindex(C, L, H):
        target = ref.rehydrate_k(ref.bf16_to_f64(K[c, l, :, h]), None, None, orope, pos3[c]) + d_post[c, l, h]
        err = np.abs(ref.bf16_to_f64(got[c, l, :, h]) - target) / np.maximum(1.0, np.abs(target))
        worst = max(worst, float(err.max()))
    assert worst > 8 * TOL, worst


# ---------------------------------------------------------------------------
# graph capture
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("form", ["per_head", "row_group_interleaved_pool"])
def test_graph_capture_replays_match_eager(device, form):
    """The entry points allocate, free and synchronise nothing and clear
    nothing with a memset, so a serving loop can capture them: a rehydrate
    into a paged pool followed by a shift of the same pages, captured in one
    graph, replayed three times with eager work and synchronisations between
    the replays; every replay gives the eager result bit for bit.  Once with
    the per-head kernel and separate pools, once with 4-head row groups into
    one K|V-interleaved pool."""
    import paper_2606_23581_amd as km
    import torch

    print(f"[case] graph capture rehydrate + shift ({form})", flush=True)
    rows = form != "per_head"
    rng = np.random.default_rng(61)
    C, L, n, H, D, m, P = (2, 2, 64, 8, 128, 64, 16) if rows else (2, 2, 64, 2, 128, 16, 16)
    pages = n // P
    npp = C * pages + 3
    K = dev(synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng), device)
    V = dev(synth.randn_bf16_numpy((C, L, n, H, D), 1.0, rng), device)
    Uk = dev(synth.randn_bf16_numpy((C, L, H, n, m), 0.1, rng), device)
    Wk = dev(synth.randn_bf16_numpy((C, L, H, m, D), 0.1, rng), device)
    pt = dev_i32(rng.permutation(npp)[: C * pages].reshape(C, pages), device)
    pos = dev_i32(np.repeat(rng.integers(0, 20000, size=(C, 1)), 3, axis=1), device)
    delta = dev_i32(np.full((C, 3), -777), device)
    rs = km.RopeSpec(theta=1e6, rope_dim=128)

    def pools():
        if rows:
            kv = torch.zeros((L, npp * P, 2, H, D), dtype=torch.bfloat16, device=device)
            return kv[:, :, 0], kv[:, :, 1]
        return (torch.zeros((L, npp * P, H, D), dtype=torch.bfloat16, device=device),
                torch.zeros((L, npp * P, H, D), dtype=torch.bfloat16, device=device))

    def calls(kp, vp):
        kernel = km.KERNEL_ROW_GROUP4 if rows else km.KERNEL_AUTO
        reh = km.prepare_rehydrate(K, kp, v_in=V, v_out=vp, rope=rs, chunk_pos=pos, u_k=Uk, w_k=Wk,
                                   page_table=pt, page_size=P, n_pool_pages=npp, kernel=kernel)
        assert km.rehydrate_plan(reh) == (km.PLAN_ROW_GROUP4 if rows else km.PLAN_PER_HEAD)
        return (reh,
                km.prepare_shift(kp, delta, rope=rs, n_chunks=C, n_tokens=n, page_table=pt, page_size=P,
                                 n_pool_pages=npp))

    ke, ve = pools()
    for call in calls(ke, ve):
        call.launch()
    torch.cuda.synchronize()
    want_k, want_v = bits(ke), bits(ve)

    kg, vg = pools()
    prepared = calls(kg, vg)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for call in prepared:          # warm-up launch outside the capture
            call.launch(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        for call in prepared:
            call.launch(side)
    for rep in range(3):
        kg.zero_()
        vg.zero_()
        scratch = torch.randn(1 << 20, device=device) * rep   # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(kg), want_k), f"replay {rep}: keys differ from the eager run"
        assert np.array_equal(bits(vg), want_v), f"replay {rep}: values differ from the eager run"
        del scratch
