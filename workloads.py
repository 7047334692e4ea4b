"""Seeded synthetic workloads for the fused vocabulary-projection cross-entropy.

This module only *draws* inputs: hidden states ``H [T, d]``, the vocabulary
projection split into row shards ``W_p [V_p, d]`` (``lm_head`` layout, shard p
owns the global vocabulary ids ``[off_p, off_p + V_p)``), int64 targets with an
exact count of ``ignore_index`` positions, and the visiting order of the shards.
It holds none of the method's arithmetic and is the only code that both the
CPU oracle side (tests) and the HIP side (tests, bench) share.

Recipe (shapes and distributions of the paper's isolated vocabulary-projection
benchmark, Sec. 3.2 and its appendix table of the projection; sizes of the
named workloads below):

* one ``numpy.random.default_rng(seed)`` stream (PCG64), drawn in this order:
  ``H`` (float32 standard normal times ``h_scale``), ``W`` (float32 standard
  normal divided by ``sqrt(d)``, drawn row-chunk by row-chunk in vocabulary-id
  order), the targets, then the ignore mask (exactly ``round(frac * T)``
  positions, the first entries of ``rng.permutation(T)``);
* targets are uniform over ``[0, V)`` or a bounded Zipf law
  ``P(id = k) ~ (k + 1) ** -s`` sampled by inverse CDF (ids are not permuted, so
  the mass sits in the first shard);
* bf16 inputs are the float32 draws rounded to nearest-even; the same bits go to
  the GPU path and (widened exactly to float64) to the oracle.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import List, Optional, Sequence

import numpy as np

IGNORE_INDEX = -100


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    T: int
    d: int
    V: int
    P: int
    dtype: str  # "f32" or "bf16"
    seed: int
    h_scale: float
    target_law: str  # "uniform" or "zipf"
    zipf_s: float
    ignore_frac: float
    order: str  # "natural", "ring0" (rank 0's ring order), "ring0_reversed"


# The five workloads.  Names state what each one is.
WORKLOADS = {
    w.name: w
    for w in [
        Workload("tiny_f32_T256_d256_V2048_P8", 256, 256, 2048, 8, "f32", 0, 1.0,
                 "uniform", 0.0, 0.05, "natural"),
        Workload("bf16_T4096_d2880_V201088_P8", 4096, 2880, 201088, 8, "bf16", 0, 1.0,
                 "uniform", 0.0, 0.02, "natural"),
        Workload("longctx_bf16_T32768_d2880_V201088_P8_ring", 32768, 2880, 201088, 8, "bf16", 0,
                 1.0, "zipf", 1.1, 0.0, "ring0"),
        Workload("wide_bf16_T16384_d7168_V129280_P8", 16384, 7168, 129280, 8, "bf16", 0, 1.0,
                 "uniform", 0.0, 0.01, "natural"),
        # h_scale: a logit is ~N(0, h_scale^2); the expected max of |logit| over 2*T*V
        # draws is ~6.47*h_scale, so 6.18 puts it near 40.
        Workload("stress_bf16_T65536_d4096_V151936_P16_rev", 65536, 4096, 151936, 16, "bf16", 0,
                 6.18, "zipf", 1.3, 0.10, "ring0_reversed"),
        # The paper's own isolated vocabulary-projection benchmark (Sec. 3.2 table, App. C):
        # one rank's share, N = 16384 local tokens, hidden 7168, V = 200000 over P = 8
        # shards, FP32, move-weights ring order.
        Workload("paper_f32_T16384_d7168_V200000_P8_ring", 16384, 7168, 200000, 8, "f32", 0, 1.0,
                 "uniform", 0.0, 0.0, "ring0"),
    ]
}
WORKLOAD_LIST = list(WORKLOADS.values())


def shard_rows(V: int, P: int) -> List[int]:
    """Row counts of the P vocabulary shards: ceil(V/P) each, the last one shorter."""
    per = -(-V // P)
    rows = []
    left = V
    for _ in range(P):
        r = min(per, left)
        rows.append(r)
        left -= r
    return rows


def visiting_order(kind: str, P: int) -> List[int]:
    """Order in which the local tokens meet the shards.

    ``ring0`` is rank 0's order on a move-weights ring: its own shard, then
    ``(0 - i) mod P`` for ``i = 1..P-1``.  ``ring0_reversed`` is that list reversed.
    """
    if kind == "natural":
        return list(range(P))
    ring = [0] + [(-i) % P for i in range(1, P)]
    if kind == "ring0":
        return ring
    if kind == "ring0_reversed":
        return ring[::-1]
    raise ValueError(kind)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    u = u + (((u >> 16) & 1) + np.uint32(0x7FFF))
    return (u >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of a generated array (float32, or bf16 bits) to float64."""
    if dtype == "bf16":
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


@dataclasses.dataclass
class Inputs:
    workload: Workload
    T: int
    d: int
    V: int
    dtype: str
    H: np.ndarray  # [T, d] float32, or uint16 bf16 bits
    W_shards: List[np.ndarray]  # P arrays [V_p, d], same storage dtype as H
    targets: np.ndarray  # int64 [T]
    order: List[int]
    shard_rows: List[int]
    ignore_index: int = IGNORE_INDEX

    def sha256(self) -> str:
        h = hashlib.sha256()
        h.update(np.ascontiguousarray(self.H).tobytes())
        for w in self.W_shards:
            h.update(np.ascontiguousarray(w).tobytes())
        h.update(self.targets.tobytes())
        return h.hexdigest()


def _draw_targets(rng: np.random.Generator, w: Workload, T: int, V: int) -> np.ndarray:
    if w.target_law == "uniform":
        t = rng.integers(0, V, size=T, dtype=np.int64)
    elif w.target_law == "zipf":
        weights = np.arange(1, V + 1, dtype=np.float64) ** (-w.zipf_s)
        cdf = np.cumsum(weights)
        cdf /= cdf[-1]
        t = np.searchsorted(cdf, rng.random(T), side="right").astype(np.int64)
        np.minimum(t, V - 1, out=t)
    else:
        raise ValueError(w.target_law)
    n_ign = int(round(w.ignore_frac * T))
    if n_ign:
        t[rng.permutation(T)[:n_ign]] = IGNORE_INDEX
    return t


def make_inputs(w: Workload | str, T: Optional[int] = None, V: Optional[int] = None,
                d: Optional[int] = None, P: Optional[int] = None,
                seed: Optional[int] = None, row_chunk: int = 8192) -> Inputs:
    """Draw one workload's inputs (optionally with T, V, d, P or seed overridden)."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    T = w.T if T is None else T
    V = w.V if V is None else V
    d = w.d if d is None else d
    P = w.P if P is None else P
    rng = np.random.default_rng(w.seed if seed is None else seed)
    H = rng.standard_normal((T, d), dtype=np.float32)
    if w.h_scale != 1.0:
        H *= np.float32(w.h_scale)
    if w.dtype == "bf16":
        H = f32_to_bf16_bits(H)
    inv = np.float32(1.0 / np.sqrt(d))
    rows = shard_rows(V, P)
    W_shards = []
    for r in rows:
        parts = []
        done = 0
        while done < r:
            n = min(row_chunk, r - done)
            blk = rng.standard_normal((n, d), dtype=np.float32) * inv
            parts.append(f32_to_bf16_bits(blk) if w.dtype == "bf16" else blk)
            done += n
        if parts:
            W_shards.append(np.ascontiguousarray(np.concatenate(parts, axis=0)))
        else:
            W_shards.append(np.zeros((0, d), dtype=np.uint16 if w.dtype == "bf16" else np.float32))
    targets = _draw_targets(rng, w, T, V)
    return Inputs(w, T, d, V, w.dtype, H, W_shards, targets, visiting_order(w.order, P), rows)


def resplit(inp: Inputs, rows: Sequence[int], order: Optional[Sequence[int]] = None) -> Inputs:
    """The same vocabulary projection split into shards of the given row counts."""
    W = np.concatenate(inp.W_shards, axis=0)
    assert sum(rows) == W.shape[0]
    offs = np.cumsum([0] + list(rows))
    shards = [np.ascontiguousarray(W[offs[p]:offs[p + 1]]) for p in range(len(rows))]
    order = list(range(len(rows))) if order is None else list(order)
    return dataclasses.replace(inp, W_shards=shards, shard_rows=list(rows), order=order)


def random_grad_loss(T: int, seed: int, kind: str = "mean", targets: Optional[np.ndarray] = None,
                     ignore_index: int = IGNORE_INDEX) -> np.ndarray:
    """Upstream per-token gradient g [T] (float32): 'mean' (1/N_valid), 'sum' (1) or 'random'."""
    if kind == "sum":
        return np.ones(T, dtype=np.float32)
    if kind == "mean":
        n_valid = T if targets is None else int(np.count_nonzero(targets != ignore_index))
        return np.full(T, 0.0 if n_valid == 0 else 1.0 / n_valid, dtype=np.float32)
    if kind == "random":
        return np.random.default_rng(seed + 7919).uniform(0.5, 1.5, size=T).astype(np.float32)
    raise ValueError(kind)


def sample_rows(T: int, n: int, seed: int) -> np.ndarray:
    """A sorted seeded sample of row indices that always includes the first and last rows."""
    rng = np.random.default_rng(seed + 104729)
    n = min(n, T)
    rows = set(rng.choice(T, size=n, replace=False).tolist())
    rows.update({0, T - 1})
    return np.array(sorted(rows), dtype=np.int64)


def sample_vocab(V: int, rows: Sequence[int], n: int, seed: int, extra: Sequence[int] = ()) -> np.ndarray:
    """Seeded vocabulary ids: shard edges, ``extra`` ids (e.g. frequent targets) and random ids."""
    rng = np.random.default_rng(seed + 1299709)
    ids = set(int(x) for x in extra)
    off = 0
    for r in rows:
        if r:
            ids.update({off, off + r - 1})
        off += r
    ids.update(rng.choice(V, size=min(n, V), replace=False).tolist())
    return np.array(sorted(i for i in ids if 0 <= i < V), dtype=np.int64)
