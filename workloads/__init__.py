"""Seeded synthetic workloads for the packed causal conv1d and selective scan.

This module is shared by the fp64 oracle tests and by the HIP-path tests and
benchmark.  It holds none of the operators' arithmetic: only random draws,
sequential packing of sequence lengths into fixed-length rows, the
position-index layout, and exact rounding of fp32 draws to bf16 storage.

Packing follows PackMamba §3.1: ``pack()`` concatenates sequences along the
sequence dimension and records, for every token, its 0-based position inside
its own sequence (``position_indices``); ``unpack()`` is its inverse.  Rows are
filled in arrival order and sealed when full (§5); the sequence that does not
fit is truncated to the space left, so rows carry no padding.

The paper's corpus (lengths 57..2048, mean 646, §4) is not available; the
log-normal length laws below stand in for it (mu=6, sigma=1 clipped to
[16, 4096] has a mean of about 648).
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Sequence

import numpy as np

__all__ = [
    "Config", "CONFIGS", "config", "draw_row_lengths", "positions_from_lengths",
    "make_inputs", "bf16_bits", "bf16_round", "pack", "unpack", "ACTIVATIONS", "draw_stream_lengths",
]

# Tensors stored in the path dtype (bf16 or fp32); everything else is fp32.
ACTIVATIONS = ("x", "z", "delta", "B", "C", "dout", "u")


@dataclasses.dataclass(frozen=True)
class Config:
    key: str
    name: str
    batch: int
    seqlen: int
    dim: int
    dstate: int
    width: int
    dtype: str          # "f32" or "bf16"
    lengths: tuple      # length law, see draw_row_lengths
    seed: int

    @property
    def tokens(self) -> int:
        return self.batch * self.seqlen

    @property
    def elements(self) -> int:
        return self.batch * self.dim * self.seqlen


CONFIGS: Dict[str, Config] = {
    # Tiny packed row: 5 sequences with lengths in U{16..96}, last one fills L.
    "0": Config("0", "tiny-fp32", 1, 256, 64, 16, 4, "f32", ("tiny5", 16, 96), 1000),
    # Mamba-130M layer shape (d_inner 1536).
    "1": Config("1", "mamba-130m", 4, 2048, 1536, 16, 4, "bf16", ("lognormal", 5.5, 1.0, 8, 2048), 1001),
    # Mamba-1.4B layer shape (d_inner 4096), pack length 4096: the headline workload.
    "2": Config("2", "mamba-1.4b", 8, 4096, 4096, 16, 4, "bf16", ("lognormal", 6.0, 1.0, 16, 4096), 1002),
    # Mamba-2.8B layer shape (d_inner 5120).
    "3": Config("3", "mamba-2.8b", 8, 4096, 5120, 16, 4, "bf16", ("lognormal", 6.0, 1.0, 16, 4096), 1003),
    # Boundary stress: many short sequences, starts forced onto tile edges.
    "4a": Config("4a", "edge-stress", 2, 8192, 2048, 16, 4, "bf16", ("edges", 1, 64), 1004),
    # One long row holding three long sequences (multi-chunk carry with resets).
    "4b": Config("4b", "long-row", 1, 65536, 2048, 16, 4, "bf16", ("long3", 10000, 30000), 1005),
}


def config(key, **overrides) -> Config:
    """Return a registered config, optionally with fields replaced (shape tweaks for tests)."""
    cfg = CONFIGS[str(key)]
    return dataclasses.replace(cfg, **overrides) if overrides else cfg


# --------------------------------------------------------------------------
# sequence lengths and position indices
# --------------------------------------------------------------------------

def _edge_starts(seqlen: int) -> List[int]:
    """Forced sequence starts for the boundary-stress rows.

    Odd multiples of 64 (so half of the 64-token edges reset and half carry
    state), the powers of two 256..4096 and their right/left neighbours, a run of
    six length-1 sequences, and a length-1 sequence on the last token.
    """
    s = {0}
    s.update(range(64, seqlen, 128))
    for e in (256, 512, 1024, 2048, 4096):
        for off in (-1, 0, 1):
            if 0 < e + off < seqlen:
                s.add(e + off)
    run0 = min(5000, seqlen - 8)
    if run0 > 0:
        s.update(range(run0, run0 + 7))
    s.add(seqlen - 1)
    return sorted(x for x in s if 0 <= x < seqlen)


def draw_stream_lengths(law: tuple, rng: np.random.Generator, count: int) -> np.ndarray:
    """``count`` sequence lengths of a stream (int64), drawn as the log-normal law of
    the workloads draws them, before any packing."""
    if law[0] != "lognormal":
        raise ValueError("stream lengths are drawn from a log-normal law")
    mu, sigma, lo, hi = law[1:]
    return np.clip(np.rint(np.exp(rng.normal(mu, sigma, size=count))), lo, hi).astype(np.int64)


def draw_row_lengths(law: tuple, rng: np.random.Generator, batch: int, seqlen: int) -> List[List[int]]:
    """Draw per-row sequence lengths; every row sums to ``seqlen``."""
    kind = law[0]
    rows: List[List[int]] = []
    if kind == "tiny5":
        lo, hi = law[1], law[2]
        for _ in range(batch):
            while True:
                first = rng.integers(lo, hi + 1, size=4)
                last = seqlen - int(first.sum())
                if 1 <= last <= hi:
                    break
            rows.append([int(v) for v in first] + [last])
    elif kind == "lognormal":
        mu, sigma, lo, hi = law[1:]
        for _ in range(batch):
            row, left = [], seqlen
            while left > 0:
                n = int(np.clip(np.rint(np.exp(rng.normal(mu, sigma))), lo, hi))
                n = min(n, left)          # sequential packing: truncate to fill the row
                row.append(n)
                left -= n
            rows.append(row)
    elif kind == "edges":
        lo, hi = law[1], law[2]
        starts = _edge_starts(seqlen)
        for _ in range(batch):
            row = []
            for a, b in zip(starts, starts[1:] + [seqlen]):
                left = b - a
                while left > 0:
                    n = min(int(rng.integers(lo, hi + 1)), left)
                    row.append(n)
                    left -= n
            rows.append(row)
    elif kind == "long3":
        lo, hi = law[1], law[2]
        for _ in range(batch):
            l1, l2 = (int(v) for v in rng.integers(lo, hi + 1, size=2))
            rows.append([l1, l2, seqlen - l1 - l2])
    elif kind == "arange":       # one sequence per row (single-sequence layout)
        rows = [[seqlen] for _ in range(batch)]
    else:
        raise ValueError(f"unknown length law {kind!r}")
    for row in rows:
        assert sum(row) == seqlen and min(row) >= 1, row
    return rows


def positions_from_lengths(rows: Sequence[Sequence[int]], seqlen: int) -> np.ndarray:
    """position_indices (batch, seqlen) int32: 0..len-1 for each packed sequence."""
    pos = np.empty((len(rows), seqlen), dtype=np.int32)
    for b, row in enumerate(rows):
        off = 0
        for n in row:
            pos[b, off:off + n] = np.arange(n, dtype=np.int32)
            off += n
        assert off == seqlen
    return pos


# --------------------------------------------------------------------------
# bf16 storage
# --------------------------------------------------------------------------

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); return the uint16 bit patterns."""
    bits = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (bits >> np.uint32(16)) & np.uint32(1)
    rounded = (bits + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """float32 array holding exactly the bf16-representable values nearest to ``a``."""
    return (bf16_bits(a).astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# inputs
# --------------------------------------------------------------------------

_BLOCK = 1 << 22   # elements per independent random block (fixed, so results do not depend on threads)


def _fill(seq: np.random.SeedSequence, shape, kind: str, lo: float = 0.0, hi: float = 1.0,
          round_bf16: bool = False) -> np.ndarray:
    """Draw a float32 array in fixed-size blocks, block i from child i of ``seq``; optionally round to bf16."""
    out = np.empty(int(np.prod(shape)), dtype=np.float32)
    nblk = (out.size + _BLOCK - 1) // _BLOCK
    children = seq.spawn(nblk)

    def work(i):
        g = np.random.Generator(np.random.PCG64(children[i]))
        sl = out[i * _BLOCK:(i + 1) * _BLOCK]
        if kind == "normal":
            g.standard_normal(sl.size, dtype=np.float32, out=sl)
        else:
            sl[:] = g.uniform(lo, hi, size=sl.size)
        if round_bf16:
            sl[:] = bf16_round(sl)

    threads = max(1, min(16, len(os.sched_getaffinity(0)), nblk))
    if threads == 1:
        for i in range(nblk):
            work(i)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(work, range(nblk)))
    return out.reshape(shape)


def make_inputs(cfg: Config, seed: int | None = None, variant: str = "paper") -> Dict[str, np.ndarray]:
    """Seeded inputs for one config.

    The root ``SeedSequence(cfg.seed)`` (or ``seed``) is split into one child per
    draw, in this order: sequence lengths, x, z, delta (raw), delta_bias, B, C,
    conv weight, dout, u, and (``variant="general"``) A, D, conv bias.  Large
    tensors are drawn in fixed 4M-element blocks from grandchildren, so the
    values do not depend on the number of threads.

    ``variant="paper"``: A[d,n] = -(n+1), D = 1, conv bias = 0 (the recipe of the
    workloads).  ``variant="general"``: A = -exp(N(0, 0.5)), D ~ N(0,1),
    conv bias ~ U(-0.5, 0.5), so that no value is special.

    Activations (x, z, delta, B, C, dout, u) are returned as float32 arrays
    already rounded to the path dtype, so both sides see identical values.
    """
    root = np.random.SeedSequence(cfg.seed if seed is None else seed)
    (s_len, s_x, s_z, s_dt, s_db, s_B, s_C, s_w, s_dout, s_u, s_A, s_D, s_bias) = root.spawn(13)
    Nb, Dn, L, N, W = cfg.batch, cfg.dim, cfg.seqlen, cfg.dstate, cfg.width
    if cfg.dtype not in ("f32", "bf16"):
        raise ValueError(cfg.dtype)
    rb = cfg.dtype == "bf16"
    rows = draw_row_lengths(cfg.lengths, np.random.Generator(np.random.PCG64(s_len)), Nb, L)
    pos = positions_from_lengths(rows, L)
    f32 = np.float32
    out: Dict[str, np.ndarray] = {}
    out["x"] = _fill(s_x, (Nb, Dn, L), "normal", round_bf16=rb)
    out["z"] = _fill(s_z, (Nb, Dn, L), "normal", round_bf16=rb)
    out["delta"] = _fill(s_dt, (Nb, Dn, L), "normal", round_bf16=rb)
    v = np.random.Generator(np.random.PCG64(s_db)).uniform(1e-3, 1e-1, size=Dn)
    out["delta_bias"] = np.log(np.expm1(v)).astype(f32)      # inverse softplus of U[1e-3, 1e-1]
    out["B"] = _fill(s_B, (Nb, N, L), "normal", round_bf16=rb)
    out["C"] = _fill(s_C, (Nb, N, L), "normal", round_bf16=rb)
    out["w"] = np.random.Generator(np.random.PCG64(s_w)).uniform(-0.5, 0.5, size=(Dn, W)).astype(f32)
    out["dout"] = _fill(s_dout, (Nb, Dn, L), "normal", round_bf16=rb)
    out["u"] = _fill(s_u, (Nb, Dn, L), "normal", round_bf16=rb)
    if variant == "paper":
        out["A"] = np.broadcast_to(-(np.arange(N, dtype=f32) + 1), (Dn, N)).copy()
        out["D"] = np.ones(Dn, dtype=f32)
        out["bias"] = np.zeros(Dn, dtype=f32)
    elif variant == "general":
        out["A"] = (-np.exp(np.random.Generator(np.random.PCG64(s_A)).normal(0.0, 0.5, size=(Dn, N)))).astype(f32)
        out["D"] = np.random.Generator(np.random.PCG64(s_D)).standard_normal(Dn, dtype=f32)
        out["bias"] = np.random.Generator(np.random.PCG64(s_bias)).uniform(-0.5, 0.5, size=Dn).astype(f32)
    else:
        raise ValueError(variant)
    out["pos"] = pos
    out["lengths"] = np.array([n for row in rows for n in row], dtype=np.int64)
    out["row_of_seq"] = np.array([b for b, row in enumerate(rows) for _ in row], dtype=np.int64)
    return out


# --------------------------------------------------------------------------
# pack / unpack (PackMamba §3.1)
# --------------------------------------------------------------------------

def pack(seqs: Sequence[np.ndarray]) -> tuple:
    """Concatenate sequences (each (..., len_i)) along the last axis into one row.

    Returns (packed (1, ..., sum len_i), position_indices (1, sum len_i) int32).
    """
    packed = np.concatenate(list(seqs), axis=-1)[None]
    pos = positions_from_lengths([[s.shape[-1] for s in seqs]], packed.shape[-1])
    return packed, pos


def unpack(packed: np.ndarray, lengths: Sequence[int]) -> List[np.ndarray]:
    """Inverse of :func:`pack` for one row: split the last axis back into sequences."""
    assert packed.shape[0] == 1
    cuts = np.cumsum([0] + list(lengths))
    assert cuts[-1] == packed.shape[-1]
    return [packed[0, ..., cuts[i]:cuts[i + 1]] for i in range(len(lengths))]
