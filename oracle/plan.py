"""Plan oracle (test infrastructure): SH-Tiles, tile costs and Algorithm 2.

Pure Python integers, written from Sec. 4.3 of the paper:

* Sec. 4.3.1, Eq. 5 -- a SH-Tile is (sequence block b, head shard h).  Each
  packed sequence is cut at global token positions into blocks of at most B
  tokens (no extra cuts at sample boundaries, the last block may be short);
  the h_q query heads are split into H equal shards.
* Eq. 6 -- tile work f_{b,h} = (h_q/H) * sum over intersected samples j of
  sum_{q=a_bj}^{e_bj-1} (q+1), with a_bj..e_bj-1 the sample-local query
  positions of sample j inside block b (the exact causal pair count).
* Eq. 7 -- K(t) = {(j, h) : sample j intersects tile t = (b, h)}.
* Sec. 4.3.2, Eq. 8 -- Delta_comm(t, r) = sum_{g in K(t) \\ C_r} V_g
  + [r != q(t)] * (V_Q(t) + V_O(t)).
* Algorithm 2 -- C = (1 + tau) * sum_t f_t / |W|; tiles in order of decreasing
  f_t then tile ID; among workers with L_r + f_t <= C take the minimum of
  (Delta_comm, L_r, r), otherwise the minimum over all workers of
  (L_r, Delta_comm, r); then L_r += f_t and C_r |= K(t).

Readings of points the paper leaves open (each one is listed with its reason
in the design notes):

* cost unit: f is the integer (h_q/H) * (causal pair count), diagonal included;
* tile ID: global_block * H + h, with the block index running over the whole
  pool, pack-major;
* tau is the exact rational tau_num/tau_den and the capacity test is
  evaluated exactly in integers, inclusive;
* Q-home q(t): the CP rank that holds the block's first token under the
  head+tail (zigzag) CP layout -- pack p is cut into 2*CP equal chunks, chunk c
  lives on rank c if c < CP else 2*CP-1-c, and worker ids are p*CP + rank;
* initial resident sets: C_r starts with every group (j, h) whose sample j
  lies wholly on worker r (fragments do not count);
* byte volumes: V_Q = rows * (h_q/H) * d * elem_bytes, V_O = V_Q, and
  V_g = l_j * kvh * d * elem_bytes * 2 (K and V) with kvh = max(1, h_kv/H);
* q_ranges (a CP rank's share) select whole blocks; absent blocks make no
  tiles but still count in the block index.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple


@dataclass
class PlanCfg:
    B: int                 # block tokens
    H: int                 # head shards
    P: int                 # packs in the pool
    CP: int                # context-parallel degree (workers per pack)
    h_q: int
    h_kv: int
    d: int
    elem_bytes: int = 2
    tau_num: int = 3
    tau_den: int = 100

    @property
    def V(self) -> int:
        return self.P * self.CP


@dataclass
class Tile:
    id: int
    pack: int
    q_begin: int
    q_end: int
    q_row: int
    cost: int
    head_begin: int
    head_end: int
    home: int
    worker: int = -1
    samples: Tuple[int, ...] = ()     # sample indices j of K(t)
    comm: int = 0                     # Delta_comm(t, worker) when it was placed (Eq. 8)


def sample_offsets(lengths: Sequence[int]) -> List[int]:
    """cu_seqlens: start of every sample in pool coordinates, plus the total."""
    out = [0]
    for n in lengths:
        out.append(out[-1] + int(n))
    return out


def zigzag_home(pos: int, pack: int, pack_start: int, pack_len: int, cp: int) -> int:
    """Worker holding token ``pos`` under the head+tail CP layout of its pack."""
    chunk = pack_len // (2 * cp)
    c = (pos - pack_start) // chunk
    rank = c if c < cp else 2 * cp - 1 - c
    return pack * cp + rank


def causal_pairs(a: int, e: int) -> int:
    """sum_{q=a}^{e-1} (q+1): causal query-key pairs of sample-local rows a..e-1."""
    return e * (e + 1) // 2 - a * (a + 1) // 2


def build_tiles(cfg: PlanCfg, lengths: Sequence[int], pack_tokens: Sequence[int],
                q_ranges: Optional[Sequence[Tuple[int, int]]] = None) -> List[Tile]:
    """SH-Tiles of the pool in tile-ID order, with Eq. 6 costs and K(t)."""
    assert cfg.h_q % cfg.H == 0
    assert len(pack_tokens) == cfg.P
    cu = sample_offsets(lengths)
    pack_cu = sample_offsets(pack_tokens)
    assert cu[-1] == pack_cu[-1]
    heads = cfg.h_q // cfg.H

    def present(lo: int, hi: int) -> bool:
        if q_ranges is None:
            return True
        return any(b <= lo and hi <= e for b, e in q_ranges)

    tiles: List[Tile] = []
    gb = 0          # pool-global block index
    q_row = 0       # next row of the Q buffer
    for p in range(cfg.P):
        off, end = pack_cu[p], pack_cu[p + 1]
        lo = off
        while lo < end:
            hi = min(end, lo + cfg.B)
            if present(lo, hi):
                pairs = 0
                js = []
                for j in range(len(lengths)):
                    s, t = cu[j], cu[j + 1]
                    if t <= lo or s >= hi:
                        continue
                    a = max(lo, s) - s
                    e = min(hi, t) - s
                    pairs += causal_pairs(a, e)
                    js.append(j)
                home = zigzag_home(lo, p, off, end - off, cfg.CP)
                for h in range(cfg.H):
                    tiles.append(Tile(id=gb * cfg.H + h, pack=p, q_begin=lo, q_end=hi,
                                      q_row=q_row, cost=heads * pairs,
                                      head_begin=h * heads, head_end=(h + 1) * heads,
                                      home=home, samples=tuple(js)))
                q_row += hi - lo
            gb += 1
            lo = hi
    return tiles


def initial_resident(cfg: PlanCfg, lengths: Sequence[int],
                     pack_tokens: Sequence[int]) -> List[set]:
    """C_r before placement: groups (j, h) of samples lying wholly on worker r."""
    cu = sample_offsets(lengths)
    pack_cu = sample_offsets(pack_tokens)
    C: List[set] = [set() for _ in range(cfg.V)]
    for j in range(len(lengths)):
        s, t = cu[j], cu[j + 1]
        p = max(i for i in range(cfg.P) if pack_cu[i] <= s)
        off, end = pack_cu[p], pack_cu[p + 1]
        homes = {zigzag_home(x, p, off, end - off, cfg.CP) for x in range(s, t)}
        if len(homes) == 1:
            r = homes.pop()
            for h in range(cfg.H):
                C[r].add((j, h))
    return C


def kv_group_bytes(cfg: PlanCfg, length: int) -> int:
    kvh = max(1, cfg.h_kv // cfg.H)
    return length * kvh * cfg.d * cfg.elem_bytes * 2


def q_bytes(cfg: PlanCfg, t: Tile) -> int:
    return (t.q_end - t.q_begin) * (cfg.h_q // cfg.H) * cfg.d * cfg.elem_bytes


def delta_comm(cfg: PlanCfg, t: Tile, r: int, C_r: set, lengths: Sequence[int]) -> int:
    """Eq. 8: bytes added by placing tile t on worker r."""
    h = t.id % cfg.H
    kv = sum(kv_group_bytes(cfg, lengths[j]) for j in t.samples if (j, h) not in C_r)
    qo = 0 if r == t.home else 2 * q_bytes(cfg, t)      # V_Q + V_O, V_O = V_Q
    return kv + qo


def place(cfg: PlanCfg, tiles: List[Tile], lengths: Sequence[int],
          pack_tokens: Sequence[int]) -> List[int]:
    """Algorithm 2; fills ``tile.worker`` and returns the loads L_r."""
    V = cfg.V
    L = [0] * V
    C = initial_resident(cfg, lengths, pack_tokens)
    S = sum(t.cost for t in tiles)
    order = sorted(tiles, key=lambda t: (-t.cost, t.id))
    for t in order:
        # L_r + f_t <= C  <=>  tau_den*V*(L_r + f_t) <= (tau_den + tau_num)*S
        feas = [r for r in range(V)
                if cfg.tau_den * V * (L[r] + t.cost) <= (cfg.tau_den + cfg.tau_num) * S]
        dc = [delta_comm(cfg, t, r, C[r], lengths) for r in range(V)]
        if feas:
            r_star = min(feas, key=lambda r: (dc[r], L[r], r))
        else:
            r_star = min(range(V), key=lambda r: (L[r], dc[r], r))
        t.worker = r_star
        t.comm = dc[r_star]
        L[r_star] += t.cost
        h = t.id % cfg.H
        for j in t.samples:
            C[r_star].add((j, h))
    return L


def plan(cfg: PlanCfg, lengths: Sequence[int], pack_tokens: Sequence[int],
         q_ranges: Optional[Sequence[Tuple[int, int]]] = None) -> Tuple[List[Tile], List[int]]:
    """Tiles (tile-ID order, ``worker`` set) and per-worker loads."""
    tiles = build_tiles(cfg, lengths, pack_tokens, q_ranges)
    loads = place(cfg, tiles, lengths, pack_tokens)
    return tiles, loads


def worker_comm(tiles: Sequence[Tile], V: int) -> List[int]:
    """Bytes each worker receives under the plan: the sum of Eq. 8 over the
    tiles placed on it, each taken when the tile was placed (KV groups it
    did not hold yet, plus the tile's Q rows and outputs when it is not the
    tile's Q-home)."""
    B = [0] * V
    for t in tiles:
        B[t.worker] += t.comm
    return B


def max_over_mean(loads: Sequence[int]) -> float:
    tot = sum(loads)
    return (len(loads) * max(loads) / tot) if tot else 1.0
