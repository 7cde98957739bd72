"""Seeded synthetic workloads: sample lengths, fixed-token packs and bf16 tensors.

This module only *describes inputs*.  It holds none of the method's arithmetic
(no tile costs, no placement, no attention); the oracle under ``oracle/`` and
the HIP library each derive everything else (offsets, tiles, costs, outputs)
on their own from what is returned here.

Workloads stand in for the paper's private 256K / 1M production corpora
(Sec. 6.1, Fig. 2 is not reproducible): sample lengths are long-tailed with the
median the paper quotes (644 tokens, Sec. 1) and a few forced outliers of the
sizes the text names ("approaching one million" tokens).  Attention shapes
follow Table 1 (Qwen3-8B / 30B-A3B / 235B-A22B).

Length draw (one draw per sample, ``numpy.random.default_rng(seed)``, PCG64):

* a mixture component is chosen with ``u = rng.random()`` when the law is a
  mixture (lognormal if ``u < w_lognormal`` else Pareto);
* lognormal: ``max(1, round(median * exp(sigma * rng.standard_normal())))``;
* Pareto: ``floor(xmin / (1 - rng.random()) ** (1 / alpha))``;
* an optional cap clips the draw.

Fixed-token packing (Sec. 2.3): draws are appended, each clipped to the
remaining capacity, until the pack holds exactly ``L`` tokens, so the last
sample is truncated.  A forced sample of ``G`` tokens is appended *last*:
fillers fill ``L - G`` first.

Tensors: ``torch.Generator().manual_seed(1000 + seed)``; fp32 ``randn`` drawn in
the order Q, K, V, dO, then rounded to bf16 (round-to-nearest-even).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "LengthLaw", "Workload", "draw_length", "pack_lengths", "workload", "WORKLOADS",
    "W_4K", "W_32K", "W_POOL", "W_256K", "W_1M", "tensors", "tiny_random",
    "VRSP_WINDOWS", "vrsp_window",
]


@dataclass(frozen=True)
class LengthLaw:
    """A (mixture) sample-length law; see the module docstring."""
    median: float = 644.0
    sigma: float = 1.0
    w_lognormal: float = 1.0          # weight of the lognormal component
    pareto_alpha: float = 1.1
    pareto_xmin: float = 8192.0
    cap: Optional[int] = None


def draw_length(rng: np.random.Generator, law: LengthLaw) -> int:
    """One raw sample length (>= 1)."""
    use_lognormal = True
    if law.w_lognormal < 1.0:
        use_lognormal = rng.random() < law.w_lognormal
    if use_lognormal:
        n = max(1, int(round(law.median * math.exp(law.sigma * rng.standard_normal()))))
    else:
        n = int(math.floor(law.pareto_xmin / (1.0 - rng.random()) ** (1.0 / law.pareto_alpha)))
        n = max(1, n)
    if law.cap is not None:
        n = min(n, law.cap)
    return n


def pack_lengths(rng: np.random.Generator, law: LengthLaw, L: int,
                 forced: Sequence[int] = ()) -> List[int]:
    """Fill one fixed-token pack of exactly ``L`` tokens.

    Fillers drawn from ``law`` fill ``L - sum(forced)`` tokens (the last filler
    is truncated to fit), then the forced samples are appended in order.
    """
    room = L - int(sum(forced))
    if room < 0:
        raise ValueError("forced samples exceed the pack")
    out: List[int] = []
    while room > 0:
        n = min(draw_length(rng, law), room)
        out.append(n)
        room -= n
    out.extend(int(g) for g in forced)
    return out


@dataclass
class Workload:
    """One benchmark / parity workload.

    ``packs`` lists the sample lengths of each packed sequence of the pool, in
    pool order.  ``q_ranges`` (pool token coordinates, half-open) restrict the
    query rows that are present (a context-parallel rank's share); ``None``
    means every row.  The plan parameters (``B``, ``H``, ``CP``) and the number
    of virtual workers ``V = P * CP`` are part of the workload description.
    """
    name: str
    seed: int
    packs: List[List[int]]
    h_q: int
    h_kv: int
    d: int
    B: int
    H: int
    CP: int
    q_ranges: Optional[List[Tuple[int, int]]] = None
    backward: bool = True
    per_worker: bool = False      # run each virtual worker's tile set separately
    notes: List[str] = field(default_factory=list)

    @property
    def P(self) -> int:
        return len(self.packs)

    @property
    def V(self) -> int:
        return self.P * self.CP

    @property
    def lengths(self) -> List[int]:
        return [n for p in self.packs for n in p]

    @property
    def pack_tokens(self) -> List[int]:
        return [sum(p) for p in self.packs]

    @property
    def n_kv_rows(self) -> int:
        return sum(self.pack_tokens)

    @property
    def n_q_rows(self) -> int:
        if self.q_ranges is None:
            return self.n_kv_rows
        return sum(e - b for b, e in self.q_ranges)

    def q_positions(self) -> np.ndarray:
        """Global (pool) token position of every present query row, in row order."""
        if self.q_ranges is None:
            return np.arange(self.n_kv_rows, dtype=np.int64)
        return np.concatenate([np.arange(b, e, dtype=np.int64) for b, e in self.q_ranges])


# The five seeded workloads, by name (token counts, model whose attention
# shapes they take).
W_4K = "4K-h2-kv1-d64"
W_32K = "32K-qwen3-8b"
W_POOL = "pool8x64K-qwen3-30b-a3b"
W_256K = "256K-cp16-share-qwen3-235b-a22b"
W_1M = "1M-cp16-share-qwen3-30b-a3b"
WORKLOADS = (W_4K, W_32K, W_POOL, W_256K, W_1M)


def _share_ranges(L: int, cp: int, rank: int = 0) -> List[Tuple[int, int]]:
    """Head+tail (zigzag) chunks of one CP rank: chunks ``rank`` and ``2cp-1-rank``."""
    c = L // (2 * cp)
    a, b = rank, 2 * cp - 1 - rank
    return [(a * c, (a + 1) * c), (b * c, (b + 1) * c)]


def workload(name: str, scale: int = 1, rank: int = 0) -> Workload:
    """One of the five seeded workloads of ``WORKLOADS`` (the i-th uses length
    seed i + 1).

    ``scale`` > 1 divides every token count (pack size, forced sample, Pareto
    floor, cap, block size ``B``) by ``scale`` while keeping heads and ``H``;
    it builds the reduced replicas the parity tests check in full.  ``rank`` picks the CP
    rank whose head+tail share is measured in the two CP-share workloads.
    """
    if name not in WORKLOADS:
        raise ValueError(f"unknown workload {name!r}; one of {WORKLOADS}")
    k = WORKLOADS.index(name) + 1
    rng = np.random.default_rng(k)
    s = int(scale)
    if k == 1:
        law = LengthLaw(median=644, sigma=1.0)
        packs = [pack_lengths(rng, law, 4096 // s)]
        return Workload(W_4K, k, packs, 2, 1, 64, B=256 // s, H=2, CP=4,
                        backward=False)
    if k == 2:
        law = LengthLaw(median=644, sigma=1.5)
        packs = [pack_lengths(rng, law, 32768 // s, forced=[16384 // s])]
        return Workload(W_32K, k, packs, 32, 8, 128, B=2048 // s, H=2, CP=8)
    if k == 3:
        law = LengthLaw(median=644, sigma=1.5, w_lognormal=0.95, pareto_alpha=1.1,
                        pareto_xmin=8192 / s, cap=65536 // s)
        packs = [pack_lengths(rng, law, 65536 // s) for _ in range(8)]
        return Workload(W_POOL, k, packs, 32, 4, 128, B=4096 // s,
                        H=2, CP=1, per_worker=True)
    if k == 4:
        L = 262144 // s
        law = LengthLaw(median=644, sigma=1.5)
        packs = [pack_lengths(rng, law, L, forced=[200000 // s])]
        return Workload(W_256K, k, packs, 64, 4, 128,
                        B=4096 // s, H=2, CP=16, q_ranges=_share_ranges(L, 16, rank),
                        notes=["lognormal sigma=1.5 assumed", "V=16 assumed"])
    if k == 5:
        L = 1048576 // s
        law = LengthLaw(median=644, sigma=2.0, w_lognormal=0.95, pareto_alpha=1.05,
                        pareto_xmin=32768 / s)
        packs = [pack_lengths(rng, law, L, forced=[900000 // s])]
        return Workload(W_1M, k, packs, 32, 4, 128,
                        B=8192 // s, H=2, CP=16, q_ranges=_share_ranges(L, 16, rank),
                        notes=["mixture weights 0.95/0.05 assumed"])
    raise AssertionError(name)


# Optimizer-step windows of packed sequences (stand-ins for the 256K and 1M
# production datasets of Sec. 6.1): every pack is filled to exactly its
# token count from a long-tailed law (median 644, a Pareto tail reaching the
# pack size), so a few packs carry outliers and most carry many short samples.
VRSP_WINDOWS = {
    "256K": (262144, LengthLaw(median=644, sigma=1.5, w_lognormal=0.95, pareto_alpha=1.1,
                               pareto_xmin=8192, cap=262144)),
    "1M": (1048576, LengthLaw(median=644, sigma=2.0, w_lognormal=0.95, pareto_alpha=1.05,
                              pareto_xmin=32768, cap=1048576)),
}


def vrsp_window(kind: str, gbs: int, seed: int) -> List[List[int]]:
    """``gbs`` packed sequences (lists of raw-sample lengths) of one window."""
    L, law = VRSP_WINDOWS[kind]
    rng = np.random.default_rng(50_000 + int(seed))
    return [pack_lengths(rng, law, L) for _ in range(int(gbs))]


def tensors(seed: int, n_q: int, n_k: int, h_q: int, h_kv: int, d: int,
            with_dout: bool = True, zero_k: bool = False):
    """Seeded bf16 Q, K, V (and dO) on the CPU, THD layout ``[rows, heads, d]``.

    Returns ``(q, k, v, dout)``; ``dout`` is None when ``with_dout`` is false.
    ``zero_k`` replaces K by zeros after drawing it (the draw order is kept so
    V and dO are the same values as in the unmodified workload).
    """
    import torch
    g = torch.Generator().manual_seed(1000 + int(seed))
    q = torch.randn((n_q, h_q, d), generator=g, dtype=torch.float32).to(torch.bfloat16)
    k = torch.randn((n_k, h_kv, d), generator=g, dtype=torch.float32).to(torch.bfloat16)
    v = torch.randn((n_k, h_kv, d), generator=g, dtype=torch.float32).to(torch.bfloat16)
    do = None
    if with_dout:
        do = torch.randn((n_q, h_q, d), generator=g, dtype=torch.float32).to(torch.bfloat16)
    if zero_k:
        k = torch.zeros_like(k)
    return q, k, v, do


def tiny_random(seed: int, max_packs: int = 3, max_len: int = 40,
                heads: Sequence[Tuple[int, int]] = ((1, 1), (2, 1), (4, 2), (8, 2)),
                d_choices: Sequence[int] = (64, 128)) -> Workload:
    """A small random workload for exhaustive / brute-force checks.

    Pack sizes are multiples of ``2 * CP`` so that the head+tail CP layout
    exists; lengths are drawn uniformly so that ragged edges are common.
    """
    rng = np.random.default_rng(10_000 + seed)
    P = int(rng.integers(1, max_packs + 1))
    CP = int(rng.choice([1, 1, 2, 4]))
    h_q, h_kv = heads[int(rng.integers(0, len(heads)))]
    H_opts = [h for h in (1, 2, 4, 8) if h_q % h == 0 and (h_kv % h == 0 or h % h_kv == 0)]
    H = int(rng.choice(H_opts))
    d = int(rng.choice(list(d_choices)))
    unit = 2 * CP
    packs = []
    for _ in range(P):
        L = unit * int(rng.integers(1, max(2, max_len // unit) + 1))
        lens: List[int] = []
        room = L
        while room > 0:
            n = min(int(rng.integers(1, max(2, L // 2) + 1)), room)
            lens.append(n)
            room -= n
        packs.append(lens)
    B = int(rng.integers(1, max(2, max(sum(p) for p in packs)) + 1))
    return Workload(f"tiny{seed}", seed, packs, h_q, h_kv, d, B=B, H=H, CP=CP)


def small_random(seed: int) -> Workload:
    """A few-hundred-token random pool that spans several kernel tiles.

    Ragged sample and pack sizes, block sizes that are not multiples of the
    kernel's row or key blocks, and head layouts from MHA to 16-way GQA.
    """
    rng = np.random.default_rng(20_000 + seed)
    layouts = [(2, 1, 2), (4, 1, 2), (8, 2, 2), (8, 2, 4), (16, 2, 2), (32, 4, 2), (12, 4, 4),
               (4, 4, 1), (32, 2, 8), (6, 3, 3)]
    h_q, h_kv, H = layouts[int(rng.integers(0, len(layouts)))]
    d = int(rng.choice([64, 128]))
    CP = int(rng.choice([1, 2]))
    P = int(rng.integers(1, 4))
    packs = []
    for _ in range(P):
        L = 2 * CP * int(rng.integers(8, 160))
        lens: List[int] = []
        room = L
        while room > 0:
            n = min(int(rng.integers(1, 400)) if rng.random() < 0.8 else int(rng.integers(1, 8)),
                    room)
            lens.append(n)
            room -= n
        packs.append(lens)
    B = int(rng.integers(1, 300))
    return Workload(f"small{seed}", seed, packs, h_q, h_kv, d, B=B, H=H, CP=CP)
