"""Device set-up of the operator workloads in ``synth.WORKLOADS``.

Builds the seeded device tensors of a workload and a prepared library call
that performs one pass of it (the unit the benchmark times and the full-size
parity tests check).  It draws inputs and lays them out; every number the
operator produces comes from the HIP library.
"""

from __future__ import annotations

import dataclasses
from typing import Callable, Dict, List, Optional

import numpy as np

from . import WORKLOADS, Workload, chunk_meta, randn_bf16_device, window_survivor_slots


@dataclasses.dataclass
class Prepared:
    workload: Workload
    tensors: Dict[str, object]          # device tensors by name
    meta: object                        # synth.ChunkMeta
    step: Callable[[], None]            # one pass of the hot path (one launch)
    bytes_per_step: int                 # algorithmic bytes (K/V in + U, W + K/V out)
    chunks_per_step: int
    extra: Dict[str, object] = dataclasses.field(default_factory=dict)


def algorithmic_bytes(w: Workload) -> int:
    """K/V rows read + patch factors read + K/V rows written, bf16.

    rehydrate, per (chunk, layer, head): 2 planes x (n*D read + n*D written)
    plus, per patched plane, U (n*m) and W (m*patch_dim).  The page table and
    positions are excluded.  shift: the rope band of every survivor row read
    and written.
    """
    n, D = w.n_tokens, w.head_dim
    if w.kind == "shift":
        return w.n_chunks * w.n_layers * w.n_heads * n * w.rope_dim * 2 * 2
    planes = 2 if w.has_v else 1
    rows = planes * 2 * n * D * 2
    factors = 0
    for m in ((w.m_k, w.m_v) if w.has_v else (w.m_k,)):
        if m > 0:
            factors += (n * m + m * w.patch_dim) * 2
    if w.m_pe > 0:
        factors += (n * w.m_pe + w.m_pe * w.rope_dim) * 2
    patched_layers = w.n_layers - w.patch_from_layer
    per_layer_units = w.n_chunks * w.n_heads
    return per_layer_units * (w.n_layers * rows + patched_layers * factors)


def _rope_spec(w: Workload):
    import paper_2606_23581_amd as km

    return km.RopeSpec(theta=w.theta, rope_dim=w.rope_dim, pairing=w.pairing,
                       rope_offset=w.rope_offset, sections=w.sections,
                       section_order=w.section_order)


class _Arena:
    """The large tensors of one workload carved from one device allocation,
    each at a 2 MiB boundary, as a serving engine reserves one region for its
    KV store (``nbytes`` = 0: every tensor allocated on its own)."""

    ALIGN = 2 << 20

    def __init__(self, nbytes: int, device):
        import torch

        self.device = device
        self.off = 0
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=device) if nbytes > 0 else None

    def empty(self, shape):
        import torch

        if self.buf is None:
            return torch.empty(shape, dtype=torch.bfloat16, device=self.device)
        nb = 2 * int(np.prod(shape))
        at = -(-self.off // self.ALIGN) * self.ALIGN
        if at + nb > self.buf.numel():
            raise RuntimeError("workload arena too small")
        self.off = at + nb
        return self.buf[at:at + nb].view(torch.bfloat16).view(shape)

    def zeros(self, shape):
        t = self.empty(shape)
        t.zero_()
        return t

    def randn(self, shape, std, gen, slab_dim: int = 0):
        return randn_bf16_device(shape, std, gen, self.device, slab_dim=slab_dim, out=self.empty(shape))


def _arena_bytes(w: Workload, meta) -> int:
    """Upper bound of the arena of one workload: its inputs, factors and outputs
    (bf16), each rounded up to the alignment, plus one alignment each."""
    C, L, H, n, D = w.n_chunks, w.n_layers, w.n_heads, w.n_tokens, w.head_dim
    planes = 2 if (w.kind == "rehydrate" and w.has_v) else 1
    sizes = []
    if w.kind == "shift":
        sizes.append(L * w.window_slots * n * H * D)
    else:
        if w.reloc:
            sizes += [w.window_slots * L * n * H * D] * planes
        else:
            sizes += [C * L * n * H * D] * planes
        for m in ((w.m_k, w.m_v) if w.has_v else (w.m_k,)):
            if m > 0:
                sizes += [C * L * H * n * m, C * L * H * m * w.patch_dim]
        if w.m_pe > 0:
            sizes += [C * L * H * n * w.m_pe, C * L * H * w.m_pe * w.rope_dim]
        if not w.reloc:
            rows = w.n_pool_pages * w.page_size if w.paged else int(meta.row_base.max()) + n
            sizes += [L * rows * H * D] * planes
    A = _Arena.ALIGN
    return sum(-(-2 * s // A) * A + A for s in sizes)


def _kv_rows(shape, gen, arena: _Arena, unit_major: bool):
    """K/V of one workload, [C, L, n, H, D] as the operator sees it.  With
    ``unit_major`` the memory is [C, L, H, n, D]: every (chunk, layer, head)
    unit is one contiguous run of rows."""
    C, L, n, H, D = shape
    if unit_major:
        return arena.randn((C, L, H, n, D), 1.0, gen).permute(0, 1, 3, 2, 4)
    return arena.randn(shape, 1.0, gen)


def _u_rows(shape, std, gen, arena: _Arena, token_major: bool):
    """Patch factors U of one workload, [C, L, H, n, m] as the operator sees
    it.  With ``token_major`` the memory is [C, L, n, H, m]: the factors of
    every head of a token row are adjacent, like the rows themselves."""
    C, L, H, n, m = shape
    if token_major:
        return arena.randn((C, L, n, H, m), std, gen).permute(0, 1, 3, 2, 4)
    return arena.randn(shape, std, gen)


def prepare(name: str, device="cuda", seed: Optional[int] = None, unit_major: bool = True,
            pool_head_major: bool = False, u_token_major: bool = False,
            separate_pools: bool = False, arena: bool = True, kernel: int = 0) -> Prepared:
    """Device tensors and the prepared call of one workload.  The paged pool
    and the relocation window hold K and V interleaved by rows (one tensor
    [.., slot or token, K|V, H, D]) unless ``separate_pools``; the inputs,
    factors and outputs are carved from one allocation unless not ``arena``.
    ``kernel`` is the rehydrate kernel requested (0: the library's choice)."""
    import torch

    import paper_2606_23581_amd as km

    w = WORKLOADS[name]
    meta = chunk_meta(w, seed)
    gen = torch.Generator(device=device)
    gen.manual_seed(w.seed if seed is None else seed)
    C, L, H, n, D = w.n_chunks, w.n_layers, w.n_heads, w.n_tokens, w.head_dim
    rope = _rope_spec(w)
    T: Dict[str, object] = {}
    A = _Arena(_arena_bytes(w, meta) if arena else 0, device)

    if w.kind == "shift":
        # ring window of S chunk slots [L, S*n, H, D], already rotated keys
        S = w.window_slots
        T["window"] = A.randn((L, S * n, H, D), 1.0, gen, slab_dim=0)
        T["delta"] = torch.from_numpy(meta.delta).to(device)
        state = {"slide": 0}
        T["row_base"] = torch.zeros(C, dtype=torch.int32, device=device)

        def set_slide(k):
            slots = window_survivor_slots(w, k)
            T["row_base"].copy_(torch.from_numpy((slots * n).astype(np.int32)))
            state["slide"] = k

        set_slide(0)
        call = km.prepare_shift(T["window"], T["delta"], rope=rope, n_chunks=C, n_tokens=n,
                                row_base=T["row_base"])

        def step():
            call.launch()

        p = Prepared(w, T, meta, step, algorithmic_bytes(w), C)
        p.extra["set_slide"] = set_slide
        p.extra["call"] = call
        p.extra["arena"] = A.buf
        return p

    if w.reloc:
        # the window's K/V, chunk-major [slot][L][n][H][D]; survivors are slots
        # 1..15, rotated and moved in place (input = output)
        S = w.window_slots
        if w.has_v and not separate_pools:
            # one window [slot][L][n][K|V][H][D]: the K and V rows of a token adjacent
            T["kv_window"] = A.randn((S, L, n, 2, H, D), 1.0, gen)
            T["k_window"], T["v_window"] = T["kv_window"][:, :, :, 0], T["kv_window"][:, :, :, 1]
        else:
            T["k_window"] = A.randn((S, L, n, H, D), 1.0, gen)
            if w.has_v:
                T["v_window"] = A.randn((S, L, n, H, D), 1.0, gen)
        T["k_in"] = T["k_window"][1:1 + C]
        if w.has_v:
            T["v_in"] = T["v_window"][1:1 + C]
    else:
        T["k_in"] = _kv_rows((C, L, n, H, D), gen, A, unit_major)
        if w.has_v:
            T["v_in"] = _kv_rows((C, L, n, H, D), gen, A, unit_major)
    if w.m_k > 0:
        T["u_k"] = _u_rows((C, L, H, n, w.m_k), w.u_std, gen, A, u_token_major)
        T["w_k"] = A.randn((C, L, H, w.m_k, w.patch_dim), w.w_std, gen)
    if w.has_v and w.m_v > 0:
        T["u_v"] = _u_rows((C, L, H, n, w.m_v), w.u_std, gen, A, u_token_major)
        T["w_v"] = A.randn((C, L, H, w.m_v, w.patch_dim), w.w_std, gen)
    if w.m_pe > 0:
        T["u_pe"] = A.randn((C, L, H, n, w.m_pe), w.u_std, gen)
        T["w_pe"] = A.randn((C, L, H, w.m_pe, w.rope_dim), w.w_std, gen)
    T["chunk_pos"] = torch.from_numpy(meta.pos).to(device)
    kw = dict(rope=rope, chunk_pos=T["chunk_pos"], u_k=T.get("u_k"), w_k=T.get("w_k"),
              k_patch=(w.patch_offset, w.patch_dim),
              pos_mode=km.POS_GRID3 if w.pos_mode == "grid3" else km.POS_LINEAR, grid_w=w.grid_w)
    if w.reloc:
        T["delta"] = torch.from_numpy(meta.delta).to(device)
        kw["delta"] = T["delta"]
    if w.m_pe > 0:
        kw.update(u_pe=T["u_pe"], w_pe=T["w_pe"])
    if w.patch_from_layer > 0:
        ranks = np.array([0 if l < w.patch_from_layer else max(w.m_k, w.m_v, w.m_pe) for l in range(L)],
                         dtype=np.int32)
        T["layer_rank"] = torch.from_numpy(ranks).to(device)
        kw.update(k_layer_rank=T["layer_rank"], v_layer_rank=T["layer_rank"], pe_layer_rank=T["layer_rank"])
    if w.reloc:
        k_out = T["k_in"]
        if w.has_v:
            v_out = T["v_in"]
    elif w.paged:
        slots = w.n_pool_pages * w.page_size
        if w.has_v and not pool_head_major and not separate_pools:
            # one pool [L, slots, K|V, H, D]: the K and V rows of a slot are
            # adjacent, so a 16-token page of both planes is one 64 KiB run
            T["kv_pool"] = A.zeros((L, slots, 2, H, D))
            T["k_pool"], T["v_pool"] = T["kv_pool"][:, :, 0], T["kv_pool"][:, :, 1]
        elif pool_head_major:   # [L, H, slots, D] memory, [L, slots, H, D] view
            T["k_pool"] = A.zeros((L, H, slots, D)).transpose(1, 2)
            if w.has_v:
                T["v_pool"] = A.zeros((L, H, slots, D)).transpose(1, 2)
        else:
            T["k_pool"] = A.zeros((L, slots, H, D))
            if w.has_v:
                T["v_pool"] = A.zeros((L, slots, H, D))
        T["page_table"] = torch.from_numpy(meta.page_table).to(device)
        kw.update(page_table=T["page_table"], page_size=w.page_size, n_pool_pages=w.n_pool_pages)
        k_out = T["k_pool"]
        if w.has_v:
            v_out = T["v_pool"]
    else:
        rows = int(meta.row_base.max()) + n
        T["k_out_rows"] = A.zeros((L, rows, H, D))
        k_out = T["k_out_rows"].unsqueeze(0).expand(C, L, rows, H, D)
        T["row_base"] = torch.from_numpy(meta.row_base).to(device)
        kw["row_base"] = T["row_base"]
        if w.has_v:
            T["v_out_rows"] = A.zeros((L, rows, H, D))
            v_out = T["v_out_rows"].unsqueeze(0).expand(C, L, rows, H, D)
    if w.has_v:
        kw.update(v_in=T["v_in"], v_out=v_out, u_v=T.get("u_v"), w_v=T.get("w_v"),
                  v_patch=(w.patch_offset, w.patch_dim))
    call = km.prepare_rehydrate(T["k_in"], k_out, kernel=kernel, **kw)

    def step():
        call.launch()

    p = Prepared(w, T, meta, step, algorithmic_bytes(w), C)
    p.extra["call"] = call
    p.extra["arena"] = A.buf
    return p


def sample_units(w: Workload, k: int, seed: int = 0) -> List[tuple]:
    """k distinct (chunk, layer, head) units, always including the first and last."""
    rng = np.random.default_rng(seed)
    total = w.n_chunks * w.n_layers * w.n_heads
    idx = set([0, total - 1])
    while len(idx) < min(k, total):
        idx.add(int(rng.integers(0, total)))
    out = []
    for u in sorted(idx):
        c, rem = divmod(u, w.n_layers * w.n_heads)
        l, h = divmod(rem, w.n_heads)
        out.append((c, l, h))
    return out


def form_deficits(w: Workload, device, planes, orbit: int = 1, chunks: Optional[int] = None):
    """Synthetic fp32 deficits for patch forming on workload w: for each plane
    name, a tensor [C, L, H, n, d] (or [K, C, L, H, n, d] for an orbit of K
    orderings) of N(0, 1) token coefficients on the decaying spectrum
    sigma_k = (1 + k)^(-1/4) in one random orthonormal basis per plane, so that
    about 90% of the energy sits in the top ~80% of the components and the
    spectrum has no gap at the rank.  chunks: generate only the first few
    chunks (the rest of the tensor is left uninitialised)."""
    import torch

    dev = torch.device(device)
    C, L, H, n, d = w.n_chunks, w.n_layers, w.n_heads, w.n_tokens, w.head_dim
    K = max(1, orbit)
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed + 7)
    sig = (1.0 + torch.arange(d, device=dev, dtype=torch.float32)) ** -0.25
    out = {}
    for name in planes:
        q, _ = torch.linalg.qr(torch.randn((d, d), generator=gen, device=dev, dtype=torch.float32))
        D = torch.empty((K, C, L, H, n, d) if K > 1 else (C, L, H, n, d), dtype=torch.float32, device=dev)
        Dv = D.view(K * C, L, H, n, d)
        for c in range(K * C if chunks is None else min(K * C, chunks)):
            a = torch.randn((L, H, n, d), generator=gen, device=dev, dtype=torch.float32)
            torch.matmul(a * sig, q.contiguous(), out=Dv[c])
            del a
        out[name] = D
    return out

