"""Seeded synthetic SparSTAR workloads (inputs only; none of the method's arithmetic).

Both the HIP path and the CPU oracle read what this module produces; neither
computes anything here.  It stands in for InfinityStar's late-scale Q/K/V, which
need the model weights and prompts and are not available.

Key layout follows Eq. (1): K = Concat(K_ref, K_text, K_cur) with
L_k = L_ref + L_text + L_q (the "listed" layout [text | ref | cur] is also
available).  Values are drawn in float32, then rounded to bf16 with
round-to-nearest-even; every consumer reads those bf16 bits.

Planted block structure (per batch element and head):
  1. Q, K, V base values ~ N(0, 1).
  2. Every key block j gets an offset o_j = 2 * u_j / |u_j|, u_j ~ N(0, I_D),
     added to all of its tokens.
  3. Every query block i picks `aligned` key blocks uniformly without
     replacement among the blocks lying wholly outside the text segment (and
     outside its band, if any) and adds 1.5 * sum of their offsets to all of its
     tokens.
  4. Optionally (`band` > 0): a local spatial band, adding band_weight * sum of
     o_{c0+i+d}, |d| <= band, where c0 is the first current-segment block,
     clipped to the current segment.

Random streams are keyed by (seed, batch, head, stream) so that any head can be
regenerated alone.  Per-head densities for a sweep are drawn from their own
stream (seed + 1000).
"""
from __future__ import annotations

import dataclasses

import numpy as np

_STREAM_K, _STREAM_Q, _STREAM_V, _STREAM_PLANT = 0, 1, 2, 3


# --------------------------------------------------------------------------
# bf16 storage
# --------------------------------------------------------------------------
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); returns the
    16-bit patterns as uint16.  Inputs here are finite."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    t = u >> np.uint32(16)
    t &= np.uint32(1)
    t += np.uint32(0x7FFF)
    t += u
    t >>= np.uint32(16)
    return t.astype(np.uint16)


def _add_per_block(x: np.ndarray, per_block: np.ndarray, block: int) -> None:
    """x[t] += per_block[t // block] in place (x: [L, D] float32)."""
    n_full = x.shape[0] // block
    if n_full:
        x[: n_full * block].reshape(n_full, block, -1)[...] += per_block[:n_full, None, :]
    if x.shape[0] > n_full * block:
        x[n_full * block:] += per_block[n_full]


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact float32 values of bf16 bit patterns."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return bf16_to_f32(bits).astype(np.float64)


# --------------------------------------------------------------------------
# Workload description
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    heads: int
    head_dim: int
    block: int
    lq: int
    l_text: int
    l_ref: int
    density: float
    aligned: int
    seed: int
    batch: int = 1
    band: int = 0
    band_weight: float = 0.5
    layout: str = "eq1"          # "eq1": [ref | text | cur]; "listed": [text | ref | cur]
    density_spread: float = 0.0  # per-head densities ~ U[(1-s)rho, (1+s)rho] when > 0

    @property
    def lk(self) -> int:
        return self.l_ref + self.l_text + self.lq

    def segments(self) -> dict[str, tuple[int, int]]:
        """Half-open token ranges of the three key segments."""
        if self.layout == "eq1":
            ref = (0, self.l_ref)
            text = (self.l_ref, self.l_ref + self.l_text)
        elif self.layout == "listed":
            text = (0, self.l_text)
            ref = (self.l_text, self.l_text + self.l_ref)
        else:
            raise ValueError(self.layout)
        cur = (self.l_ref + self.l_text, self.lk)
        return {"ref": ref, "text": text, "cur": cur}

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads: a tiny CPU-checkable case, a mid pyramid scale, the 720p
# final scale (72,000 queries; Section 1 and the supplement's scale table), the
# density sweep at that shape, and a five-scale clip pyramid.
TINY = Workload("tiny", heads=2, head_dim=64, block=64, lq=512, l_text=128, l_ref=512,
                density=0.25, aligned=3, seed=41)
MID = Workload("mid", heads=24, head_dim=128, block=64, lq=11_520, l_text=512, l_ref=72_000,
               density=0.25, aligned=8, seed=42)
P720 = Workload("720p", heads=24, head_dim=128, block=64, lq=72_000, l_text=512, l_ref=72_000,
                density=0.25, aligned=16, seed=43, band=2)
SWEEP_DENSITIES = (0.10, 0.25, 0.50)
SWEEP = P720.with_(name="sweep", seed=44, density_spread=0.5)
PYRAMID_GRIDS = ((9, 16), (18, 32), (27, 48), (36, 64), (45, 80))
PYRAMID_T = 20


def pyramid_scales(density: float = 0.25) -> list[tuple[Workload, bool]]:
    """The five clip-pyramid scales (T = 20 frames), each as (workload, sparse?):
    dense on the first three, sparse on the last two."""
    out = []
    for s, (h, w) in enumerate(PYRAMID_GRIDS):
        lq = PYRAMID_T * h * w
        wl = P720.with_(name=f"pyramid_s{s + 1}", lq=lq, seed=45 + 10 * s, density=density)
        out.append((wl, s >= 3))
    return out


# --------------------------------------------------------------------------
# Generation
# --------------------------------------------------------------------------
def _rng(w: Workload, b: int, h: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([w.seed, b, h, stream])


def _nblocks(length: int, block: int) -> int:
    return -(-length // block)


def _plant_candidates(w: Workload) -> np.ndarray:
    """Key blocks lying wholly outside the text segment."""
    t0, t1 = w.segments()["text"]
    n_k = _nblocks(w.lk, w.block)
    j = np.arange(n_k)
    outside = ((j + 1) * w.block <= t0) | (j * w.block >= t1)
    return j[outside]


def _band_blocks(w: Workload, i: int) -> np.ndarray:
    if w.band <= 0:
        return np.zeros(0, dtype=np.int64)
    c_begin, c_end = w.segments()["cur"]
    c0 = c_begin // w.block
    c_last = (c_end - 1) // w.block
    idx = np.arange(c0 + i - w.band, c0 + i + w.band + 1)
    return idx[(idx >= c0) & (idx <= c_last)]


def generate_head(w: Workload, b: int = 0, h: int = 0):
    """Q [L_q, D], K [L_k, D], V [L_k, D] of one (batch, head) as bf16 bit patterns."""
    d, blk = w.head_dim, w.block
    n_q, n_k = _nblocks(w.lq, blk), _nblocks(w.lk, blk)

    rk = _rng(w, b, h, _STREAM_K)
    kx = rk.standard_normal((w.lk, d), dtype=np.float32)
    u = rk.standard_normal((n_k, d), dtype=np.float32).astype(np.float64)
    offs = 2.0 * u / np.linalg.norm(u, axis=1, keepdims=True)          # [n_k, D]
    _add_per_block(kx, offs.astype(np.float32), blk)

    rq = _rng(w, b, h, _STREAM_Q)
    qx = rq.standard_normal((w.lq, d), dtype=np.float32)
    rp = _rng(w, b, h, _STREAM_PLANT)
    cand = _plant_candidates(w)
    qoff = np.zeros((n_q, d), dtype=np.float64)
    for i in range(n_q):
        band = _band_blocks(w, i)
        pool = np.setdiff1d(cand, band, assume_unique=True) if band.size else cand
        m = min(w.aligned, pool.size)
        if m:
            chosen = rp.choice(pool, size=m, replace=False)
            qoff[i] += 1.5 * offs[chosen].sum(axis=0)
        if band.size:
            qoff[i] += w.band_weight * offs[band].sum(axis=0)
    _add_per_block(qx, qoff.astype(np.float32), blk)

    rv = _rng(w, b, h, _STREAM_V)
    vx = rv.standard_normal((w.lk, d), dtype=np.float32)
    return bf16_bits(qx), bf16_bits(kx), bf16_bits(vx)


def _shm_worker(job):
    """Process-pool worker: generate one (batch, head) into shared memory."""
    from multiprocessing import shared_memory

    names, shapes, w, b, hi, h = job
    blocks = [shared_memory.SharedMemory(name=n) for n in names]
    try:
        arrs = [np.ndarray(shp, dtype=np.uint16, buffer=blk.buf) for shp, blk in zip(shapes, blocks)]
        for dst, src in zip(arrs, generate_head(w, b, h)):
            dst[b, hi] = src
        del arrs
    finally:
        for blk in blocks:
            blk.close()


def _may_spawn() -> bool:
    """Whether worker processes may be started: not under a profiler (its
    preloaded library would start GPU work in every child) and not after this
    process has initialised the GPU through torch."""
    import os
    import sys

    pre = os.environ.get("LD_PRELOAD", "")
    if "rocprof" in pre or any(k.startswith(("ROCPROF", "ROCP_")) for k in os.environ):
        return False
    torch = sys.modules.get("torch")
    if torch is not None:
        try:
            if torch.cuda.is_initialized():
                return False
        except Exception:  # pragma: no cover - a torch without cuda support
            return False
    return True


def generate(w: Workload, heads: list[int] | None = None, workers: int | None = None):
    """Q [B, H', L_q, D], K and V [B, H', L_k, D] as bf16 bit patterns (uint16),
    for all heads or the listed ones (H' = len(heads)).

    Large workloads are generated by spawned worker processes (numpy's
    generators hold the GIL) writing into shared memory, unless a profiler is
    attached or this process has already initialised the GPU: then everything
    is generated in-process.  The result does not depend on the number of
    workers."""
    import os

    hs = list(range(w.heads)) if heads is None else list(heads)
    shapes = [(w.batch, len(hs), w.lq, w.head_dim), (w.batch, len(hs), w.lk, w.head_dim),
              (w.batch, len(hs), w.lk, w.head_dim)]
    jobs = [(b, hi, h) for b in range(w.batch) for hi, h in enumerate(hs)]
    total = sum(int(np.prod(s)) for s in shapes) * 2
    if workers is None:
        workers = min(16, len(os.sched_getaffinity(0)), len(jobs))
    if workers <= 1 or total < (256 << 20) or not _may_spawn():
        out = [np.empty(s, dtype=np.uint16) for s in shapes]
        for b, hi, h in jobs:
            for dst, src in zip(out, generate_head(w, b, h)):
                dst[b, hi] = src
        return tuple(out)

    import multiprocessing as mp
    from multiprocessing import shared_memory

    blocks = [shared_memory.SharedMemory(create=True, size=int(np.prod(s)) * 2) for s in shapes]
    try:
        names = [blk.name for blk in blocks]
        ctx = mp.get_context("spawn")
        with ctx.Pool(processes=workers) as pool:
            pool.map(_shm_worker, [(names, shapes, w, b, hi, h) for b, hi, h in jobs], chunksize=1)
        out = tuple(np.ndarray(s, dtype=np.uint16, buffer=blk.buf).copy() for s, blk in zip(shapes, blocks))
    finally:
        for blk in blocks:
            blk.close()
            blk.unlink()
    return out


def head_densities(w: Workload, density: float | None = None) -> np.ndarray:
    """Per-head densities: all equal to the nominal density, or, with a spread s,
    drawn ~ U[(1-s) rho, (1+s) rho] (float64, clamped to [0, 1])."""
    rho = w.density if density is None else float(density)
    if w.density_spread <= 0:
        return np.full(w.heads, rho, dtype=np.float64)
    r = np.random.default_rng([w.seed + 1000])
    lo, hi = (1.0 - w.density_spread) * rho, (1.0 + w.density_spread) * rho
    return np.clip(r.uniform(lo, hi, size=w.heads), 0.0, 1.0)
