"""Element-complete checks of whole workloads against the fp64 reference.

The GPU's inputs and outputs are streamed to the host one layer at a time
into numpy memory-mapped files (double-buffered: the next layer is copied
while worker processes check the current one), and a pool of spawned,
single-threaded worker processes runs the reference on every (chunk, layer,
head) unit of the layer and compares every element.  Workers never touch the
GPU; they are started with the "spawn" method, so nothing of the parent's GPU
state is inherited.
"""

from __future__ import annotations

import dataclasses
import multiprocessing as mp
import os
import shutil
import tempfile
import time
from typing import Dict, List, Optional, Tuple

import numpy as np

TOL = 2.0 ** -7
SENTINEL = 0x7FC1


# ---------------------------------------------------------------------------
# worker side
# ---------------------------------------------------------------------------

_OPEN: Dict[str, np.ndarray] = {}


def _worker_init():
    for var in ("OPENBLAS_NUM_THREADS", "OMP_NUM_THREADS", "MKL_NUM_THREADS", "BLIS_NUM_THREADS"):
        os.environ[var] = "1"
    try:
        from threadpoolctl import threadpool_limits

        threadpool_limits(1)
    except Exception:  # pragma: no cover
        pass


def _arr(path: str, gen: int) -> np.ndarray:
    key = f"{path}@{gen}"
    a = _OPEN.get(key)
    if a is None:
        for k in [k for k in _OPEN if k.startswith(path + "@")]:
            del _OPEN[k]
        a = np.load(path, mmap_mode="r")
        _OPEN[key] = a
    return a


def _compare(got_bits: np.ndarray, want: np.ndarray) -> Tuple[int, float]:
    import oracle as ref

    got = ref.bf16_to_f64(got_bits)
    err = np.abs(got - want)
    bound = TOL * np.maximum(1.0, np.abs(want))
    bad = ~(err <= bound)
    ratio = err / bound
    return int(bad.sum()), float(np.nanmax(np.where(np.isnan(ratio), np.inf, ratio))) if ratio.size else 0.0


def check_rehydrate_layer(job: dict) -> dict:
    """Every unit (c, l, h) of chunks [c0, c1) of one layer: keys and values
    against the reference, read from the layer's host copies."""
    import oracle as ref

    g = job["gen"]
    A = {k: _arr(p, g) for k, p in job["paths"].items()}
    rope = ref.Rope(**job["rope"])
    n, H, l = job["n"], job["H"], job["layer"]
    patched = l >= job["patch_from_layer"]
    bad, worst, units = 0, 0.0, 0
    first = None
    for c in range(job["c0"], job["c1"]):
        if job["pos_mode"] == "grid3":
            p3 = ref.positions_grid3(job["pos"][c], job["grid_w"], n)
        else:
            p3 = ref.positions_linear(int(job["pos"][c][0]), n)
        if job["paged"]:
            dst = np.array([ref.paged_slot(job["page_table"][c], i, job["page_size"]) for i in range(n)])
        else:
            dst = int(job["row_base"][c]) + np.arange(n)
        for h in range(H):
            K = ref.bf16_to_f64(A["k_in"][c, :, h])
            U = W = None
            off = job["patch_offset"]
            if patched and job["m_k"]:
                U = ref.bf16_to_f64(A["u_k"][c, h])
                W = ref.bf16_to_f64(A["w_k"][c, h])
            if patched and job["m_pe"]:
                # latent patch and rope-band patch on disjoint columns = one block patch
                up = ref.bf16_to_f64(A["u_pe"][c, h])
                wp = ref.bf16_to_f64(A["w_pe"][c, h])
                Wf = np.zeros((U.shape[1] + up.shape[1], job["D"]))
                Wf[:U.shape[1], off:off + W.shape[1]] = W
                Wf[U.shape[1]:, rope.rope_offset:rope.rope_offset + rope.rope_dim] = wp
                U, W, off = np.concatenate([U, up], axis=1), Wf, 0
            if job["reloc"]:
                want = ref.relocate_k(K, U, W, rope, p3, job["delta"][c], off)
            else:
                want = ref.rehydrate_k(K, U, W, rope, p3, off)
            nb, wr = _compare(A["k_out"][dst, h] if not job["reloc"] else A["k_out"][c, :, h], want)
            units += 1
            if nb and first is None:
                first = ("K", c, l, h)
            bad += nb
            worst = max(worst, wr)
            if job["has_v"]:
                V = ref.bf16_to_f64(A["v_in"][c, :, h])
                Uv = Wv = None
                if patched and job["m_v"]:
                    Uv = ref.bf16_to_f64(A["u_v"][c, h])
                    Wv = ref.bf16_to_f64(A["w_v"][c, h])
                want = ref.rehydrate_v(V, Uv, Wv, job["patch_offset"])
                nb, wr = _compare(A["v_out"][dst, h] if not job["reloc"] else A["v_out"][c, :, h], want)
                units += 1
                if nb and first is None:
                    first = ("V", c, l, h)
                bad += nb
                worst = max(worst, wr)
    return {"bad": bad, "worst": worst, "units": units, "first": first}


def check_shift_layer(job: dict) -> dict:
    """Every survivor unit (chunk, head) of one layer of a window slide: the
    band moved by delta, against the reference on the layer before the slide."""
    import oracle as ref

    g = job["gen"]
    before = _arr(job["paths"]["before"], g)
    after = _arr(job["paths"]["after"], g)
    rope = ref.Rope(**job["rope"])
    n = job["n"]
    bad, worst, units, first = 0, 0.0, 0, None
    for j, slot in enumerate(job["slots"]):
        rows = slice(slot * n, (slot + 1) * n)
        for h in range(job["H"]):
            want = ref.shift_k(ref.bf16_to_f64(before[rows, h]), rope, job["delta"])
            nb, wr = _compare(after[rows, h], want)
            units += 1
            if nb and first is None:
                first = ("K", j, job["layer"], h)
            bad += nb
            worst = max(worst, wr)
    return {"bad": bad, "worst": worst, "units": units, "first": first}


# ---------------------------------------------------------------------------
# parent side
# ---------------------------------------------------------------------------

def bits(t) -> np.ndarray:
    import torch

    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16)


def _scratch_dir(need_bytes: int) -> str:
    """A directory for the layer files: /dev/shm when it has room, else the
    system temporary directory."""
    for base in ("/dev/shm", None):
        try:
            d = tempfile.mkdtemp(prefix="kamera_full_", dir=base)
        except OSError:
            continue
        st = os.statvfs(d)
        if st.f_bavail * st.f_frsize >= need_bytes * 1.2:
            return d
        shutil.rmtree(d, ignore_errors=True)
    raise RuntimeError(f"no scratch space for {need_bytes / 1e9:.1f} GB of layer copies")


@dataclasses.dataclass
class Result:
    bad: int = 0
    worst: float = 0.0
    units: int = 0
    first: Optional[tuple] = None
    seconds: float = 0.0
    workers: int = 0

    def add(self, r: dict):
        self.bad += r["bad"]
        self.worst = max(self.worst, r["worst"])
        self.units += r["units"]
        if self.first is None and r["first"] is not None:
            self.first = r["first"]


class LayerStreamer:
    """Double-buffered host copies of per-layer arrays and a spawned worker pool."""

    def __init__(self, layer_bytes: int, n_workers: Optional[int] = None):
        self.n_workers = n_workers or max(1, min(16, len(os.sched_getaffinity(0))))
        self.dir = _scratch_dir(2 * layer_bytes)
        self.pool = mp.get_context("spawn").Pool(self.n_workers, initializer=_worker_init)
        self.gen = 0

    def write(self, slot: int, arrays: Dict[str, np.ndarray]) -> Dict[str, str]:
        paths = {}
        for name, a in arrays.items():
            path = os.path.join(self.dir, f"{name}_{slot}.npy")
            mm = np.lib.format.open_memmap(path, mode="w+", dtype=a.dtype, shape=a.shape)
            mm[...] = a
            mm.flush()
            del mm
            paths[name] = path
        return paths

    def close(self):
        self.pool.close()
        self.pool.join()
        shutil.rmtree(self.dir, ignore_errors=True)


def run_layers(n_layers: int, layer_bytes: int, fetch, make_jobs, worker, label: str) -> Result:
    """For l in range(n_layers): fetch(l) -> {name: host array}; the arrays go
    to the layer files; make_jobs(l, paths, gen) -> jobs for `worker` in the pool.
    Layer l + 1 is fetched while layer l is being checked."""
    res = Result()
    t0 = time.perf_counter()
    st = LayerStreamer(layer_bytes)
    res.workers = st.n_workers
    try:
        pending: List[tuple] = []           # (slot, AsyncResult)
        for l in range(n_layers):
            slot = l % 2
            # the slot's previous layer must be checked before its files are rewritten
            while pending and any(p[0] == slot for p in pending):
                s, ar = pending.pop(0)
                for r in ar.get():
                    res.add(r)
            st.gen += 1
            paths = st.write(slot, fetch(l))
            jobs = make_jobs(l, paths, st.gen)
            pending.append((slot, st.pool.map_async(worker, jobs, chunksize=1)))
            if l % 8 == 0 or l == n_layers - 1:
                print(f"[full] {label}: layer {l + 1}/{n_layers} queued, {res.units} units checked, "
                      f"{time.perf_counter() - t0:.1f} s", flush=True)
        for _, ar in pending:
            for r in ar.get():
                res.add(r)
    finally:
        st.close()
    res.seconds = time.perf_counter() - t0
    return res
