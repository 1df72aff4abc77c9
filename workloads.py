"""Seeded synthetic inputs for YOSO attention, shared by the tests and the bench.

This module holds none of the method's arithmetic: it only draws the inputs that
the method consumes (unit-length queries and keys, values, upstream gradients and
the Gaussian hyperplane matrix of the sign-random-projection hash).  Both the GPU
path and the CPU oracle receive exactly these arrays.

Input recipe (stated once, used everywhere):
  * Q, K rows: N(0, I_d) in fp64, scaled to unit l2 norm (Sec. 4 preamble: the
    experiments l2-normalise queries and keys), then stored as fp32.  For the
    bf16 workload the unit rows are rounded to bf16 (round to nearest even).
  * "mixture" workloads (skewed buckets): per (batch, head) 16 random unit
    centres; every Q row and every K row independently picks a centre uniformly
    and adds N(0, 0.1^2) noise per coordinate before normalising.  Q and K share
    the centres of their head.
  * V, dY: N(0, 1), same storage dtype as Q.
  * R: N(0, 1) fp32 of shape [d, m*tau], one matrix shared by every head; column
    h*tau+b is hyperplane b of hash h (Sec. 3.2, "we sample a hash function").
  * signs: uniform random 64-bit masks of shape [ceil(m*tau/64), 3], the +-1
    diagonals D1, D2, D3 of the fast hash's pseudo-random rotations (Sec. 3.2
    "Speed-up"), one set shared by every head.

Every array comes from its own numpy PCG64 stream spawned from one seed, so any
subset of heads can be regenerated identically.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Sequence

import numpy as np

__all__ = ["Workload", "WORKLOADS", "make_inputs", "fast_hash_signs", "bf16_round", "bf16_bits"]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads: int
    n: int
    d: int
    tau: int
    m: int
    dtype: str  # "f32" or "bf16": storage type of Q, K, V, dY and outputs
    dist: str  # "gauss" or "mixture"
    seed: int

    @property
    def bh(self) -> int:
        return self.batch * self.heads

    @property
    def tokens(self) -> int:
        return self.batch * self.n

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


# The five shapes of the paper's workloads (Sec. 4: BERT-base at 512 tokens,
# LRA at 1K-4K tokens) plus two longer-context variants.  The seed of each is
# 211109714 plus its index.
WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in [
        Workload("single_head_n512", 1, 1, 512, 64, 8, 32, "f32", "gauss", 211109714 + 0),
        Workload("bert_base_n512", 32, 12, 512, 64, 8, 32, "f32", "gauss", 211109714 + 1),
        Workload("lra_n4096", 16, 2, 4096, 64, 8, 32, "f32", "gauss", 211109714 + 2),
        Workload("skewed_n16384", 4, 8, 16384, 64, 8, 16, "f32", "mixture", 211109714 + 3),
        Workload("bf16_n32768", 2, 12, 32768, 64, 9, 32, "bf16", "gauss", 211109714 + 4),
    ]
}


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32 holding them."""
    return bf16_bits_to_f32(bf16_bits(x))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The 16-bit patterns of fp32 values rounded to bf16 (ties to even). No NaN inputs."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def _unit_rows(a: np.ndarray) -> np.ndarray:
    return a / np.linalg.norm(a, axis=-1, keepdims=True)


def _head_streams(seed: int, bh: int):
    """One independent generator per (head, array) so head subsets are reproducible."""
    root = np.random.SeedSequence(seed)
    children = root.spawn(bh + 1)
    return children[0], children[1:]


def make_inputs(
    w: Workload,
    heads: Optional[Sequence[int]] = None,
    n: Optional[int] = None,
    n_k: Optional[int] = None,
) -> dict:
    """Draw Q, K, V, dY ([len(heads), n, d]) and R ([d, m*tau]) for workload ``w``.

    ``heads`` selects flattened (batch*head) indices (default: all);
    ``n`` / ``n_k`` override the query / key lengths (default: the workload's n).
    Returned arrays are fp32 holding exactly the stored values; for bf16
    workloads the raw 16-bit patterns are returned as well (``*_bits``).
    """
    n_q = w.n if n is None else n
    n_k = n_q if n_k is None else n_k
    heads = list(range(w.bh)) if heads is None else list(heads)
    r_seq, head_seqs = _head_streams(w.seed, w.bh)
    R = np.random.Generator(np.random.PCG64(r_seq)).standard_normal((w.d, w.m * w.tau)).astype(np.float32)

    out = {name: np.empty((len(heads), nn, w.d), np.float32)
           for name, nn in (("q", n_q), ("k", n_k), ("v", n_k), ("dy", n_q))}
    for slot, h in enumerate(heads):
        s_q, s_k, s_v, s_dy, s_mix = head_seqs[h].spawn(5)
        if w.dist == "gauss":
            q = _unit_rows(np.random.Generator(np.random.PCG64(s_q)).standard_normal((n_q, w.d)))
            k = _unit_rows(np.random.Generator(np.random.PCG64(s_k)).standard_normal((n_k, w.d)))
        elif w.dist == "mixture":
            g = np.random.Generator(np.random.PCG64(s_mix))
            centres = _unit_rows(g.standard_normal((16, w.d)))
            gq = np.random.Generator(np.random.PCG64(s_q))
            gk = np.random.Generator(np.random.PCG64(s_k))
            q = _unit_rows(centres[gq.integers(0, 16, n_q)] + 0.1 * gq.standard_normal((n_q, w.d)))
            k = _unit_rows(centres[gk.integers(0, 16, n_k)] + 0.1 * gk.standard_normal((n_k, w.d)))
        else:
            raise ValueError(f"unknown distribution {w.dist!r}")
        out["q"][slot] = q
        out["k"][slot] = k
        out["v"][slot] = np.random.Generator(np.random.PCG64(s_v)).standard_normal((n_k, w.d))
        out["dy"][slot] = np.random.Generator(np.random.PCG64(s_dy)).standard_normal((n_q, w.d))
    if w.dtype == "bf16":
        for name in ("q", "k", "v", "dy"):
            out[name + "_bits"] = bf16_bits(out[name])
            out[name] = bf16_bits_to_f32(out[name + "_bits"])
    out["R"] = R
    out["signs"] = fast_hash_signs(w)
    return out


def fast_hash_signs(w: Workload) -> np.ndarray:
    """The D1, D2, D3 masks of the fast hash for workload ``w`` (uint64 [ceil(m*tau/64), 3]).

    Drawn from the seed's child stream number bh + 1, after the bh + 1 streams of
    the other arrays, so adding them left every other array unchanged."""
    seq = np.random.SeedSequence(w.seed).spawn(w.bh + 2)[w.bh + 1]
    nrot = (w.m * w.tau + 63) // 64
    return np.random.Generator(np.random.PCG64(seq)).integers(0, 2**64, size=(nrot, 3), dtype=np.uint64)
