"""Seeded synthetic inputs for KV-cache migration runs.

This module only draws numbers: block tables, free lists, append counts,
request lengths and the 16-bit values that fill the pools.  It holds none of
the migration's own arithmetic (no planning, no block-count formula, no
copying), so both the GPU path's tests and the CPU oracle's tests can take
their inputs from it without sharing any of the method.

Every stream is a numpy PCG64 generator keyed by (seed, purpose), so that two
runs with one seed draw identical inputs whatever else they draw.  Values are
uniform in [-1, 1] rounded to fp16 or bf16 (round to nearest even), the
distribution of freshly computed K/V activations stated for the synthetic
pools.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# Purposes: each keys an independent sub-stream of a config's seed.
SRC_LAYOUT, DST_LAYOUT, SRC_VALUES, DST_VALUES, APPENDS, APPEND_VALUES, LENGTHS, EXTRA = range(8)

ELEM_BYTES = {"fp16": 2, "bf16": 2}


def stream(seed: int, purpose: int, sub: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(purpose, sub))))


@dataclass(frozen=True)
class PoolShape:
    num_layers: int
    num_blocks: int
    block_size: int
    kv_heads: int
    head_dim: int
    dtype: str = "fp16"

    @property
    def elem_bytes(self) -> int:
        return ELEM_BYTES[self.dtype]


@dataclass(frozen=True)
class Workload:
    """One synthetic migration workload.

    ``table_blocks`` is the number of source blocks the request's table
    holds: enough for the longest length the request can reach in this
    workload (initial length plus every append), a stated constant rather than
    something derived here."""
    name: str
    shape: PoolShape
    seed: int
    lengths: tuple                  # initial request length(s) in tokens
    table_blocks: int
    src_preoccupied: float = 0.0    # fraction of source blocks held by other requests
    dst_preoccupied: float = 0.0    # fraction of destination blocks held by other requests
    appends: int = 0                # number of seeded append batches (incremental stages)
    append_lo: int = 0
    append_hi: int = 0
    notes: str = field(default="", compare=False)


# The five workloads.  Shapes: LLaMA-7B has 32 layers of 32 heads x 128;
# LLaMA-30B has 60 layers of 52 heads x 128, so one of four tensor-parallel
# ranks holds 13 heads; the long-context GQA shape has 80 layers and 8 KV
# heads of 128.  Lengths: "1k" means 1,024 tokens (Llumnix §2, footnote).
TINY = Workload("tiny_single_stage", PoolShape(2, 256, 16, 4, 64, "fp16"), 1001,
                lengths=(200,), table_blocks=13)
LLAMA7B = Workload("llama7b_multistage", PoolShape(32, 4096, 16, 32, 128, "fp16"), 1002,
                   lengths=(8192,), table_blocks=528, src_preoccupied=0.4, dst_preoccupied=0.4,
                   appends=4, append_lo=16, append_hi=64,
                   notes="8192 + 4 x 64 tokens at most = 8448 tokens = 528 blocks")
LLAMA30B_TP4 = Workload("llama30b_tp_quarter", PoolShape(60, 8192, 16, 13, 128, "fp16"), 1003,
                        lengths=(1024, 4096, 16384), table_blocks=1040,
                        notes="16384 tokens plus up to 256 appended = 1040 blocks")
BATCHED = Workload("batched_fragmented", PoolShape(32, 0, 16, 32, 128, "bf16"), 1004,
                   lengths=(), table_blocks=0, src_preoccupied=0.5, dst_preoccupied=0.5,
                   notes="64 lognormal lengths; pools sized from the drawn lengths")
GQA_LONG = Workload("gqa_long_context", PoolShape(80, 4096, 16, 8, 128, "bf16"), 1005,
                    lengths=(32768,), table_blocks=2064,
                    notes="32768 tokens plus up to 256 appended = 2064 blocks")

WORKLOADS = {w.name: w for w in (TINY, LLAMA7B, LLAMA30B_TP4, BATCHED, GQA_LONG)}


def pool_layout(seed: int, purpose: int, num_blocks: int, preoccupied: float):
    """Split a pool's blocks into (occupied by other requests, free in random
    order).  The occupied set is a uniform random subset of
    round(preoccupied * num_blocks) blocks."""
    g = stream(seed, purpose)
    n_occ = int(round(preoccupied * num_blocks))
    perm = g.permutation(num_blocks).astype(np.int32)
    occupied = np.sort(perm[:n_occ])
    free = perm[n_occ:].copy()
    return occupied, free


def request_table(seed: int, num_blocks: int, count: int, preoccupied: float = 0.0, sub: int = 0):
    """A request's source block table: ``count`` distinct blocks drawn at
    random from the blocks not held by other requests, in random order.
    Returns (table, occupied_by_others)."""
    occupied, free = pool_layout(seed, SRC_LAYOUT, num_blocks, preoccupied)
    g = stream(seed, SRC_LAYOUT, 1 + sub)
    if count > len(free):
        raise ValueError("pool too small for the request")
    table = g.choice(free, size=count, replace=False).astype(np.int32)
    return table, occupied


def request_tables(seed: int, num_blocks: int, counts, preoccupied: float = 0.0):
    """Block tables of several requests sharing one pool: request k gets
    counts[k] distinct blocks, no block shared between requests or with the
    blocks other requests hold; every table is in random order.  Returns
    (tables, occupied_by_others)."""
    occupied, free = pool_layout(seed, SRC_LAYOUT, num_blocks, preoccupied)
    need = int(sum(counts))
    if need > len(free):
        raise ValueError("pool too small for the requests")
    g = stream(seed, SRC_LAYOUT, 1)
    pick = g.permutation(free)[:need].astype(np.int32)
    tables, at = [], 0
    for c in counts:
        tables.append(pick[at:at + int(c)].copy())
        at += int(c)
    return tables, occupied


def free_list(seed: int, num_blocks: int, preoccupied: float = 0.0):
    """The destination's free list: its free blocks in random order.
    Returns (free_list, occupied_by_others)."""
    occupied, free = pool_layout(seed, DST_LAYOUT, num_blocks, preoccupied)
    return free, occupied


def append_counts(seed: int, count: int, lo: int, hi: int) -> np.ndarray:
    """Tokens appended by decoding before each incremental stage, uniform in [lo, hi]."""
    return stream(seed, APPENDS).integers(lo, hi + 1, size=count).astype(np.int64)


def lognormal_lengths(seed: int, count: int, median: float, sigma: float, lo: int, hi: int):
    """Request lengths: lognormal with the given median, rounded and clipped."""
    g = stream(seed, LENGTHS)
    x = g.lognormal(mean=np.log(median), sigma=sigma, size=count)
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


def values16(seed: int, purpose: int, count: int, dtype: str, sub: int = 0) -> np.ndarray:
    """``count`` 16-bit values uniform in [-1, 1] rounded to ``dtype``, as
    their raw uint16 bit patterns."""
    g = stream(seed, purpose, sub)
    x = g.uniform(-1.0, 1.0, size=count)
    if dtype == "fp16":
        return x.astype(np.float16).view(np.uint16)
    if dtype == "bf16":
        f = x.astype(np.float32).view(np.uint32)
        # round to nearest even on the upper 16 bits (no NaN/Inf in [-1, 1])
        rounded = f + 0x7FFF + ((f >> 16) & 1)
        return (rounded >> 16).astype(np.uint16)
    raise ValueError(dtype)


def random_bytes(seed: int, purpose: int, count: int, sub: int = 0) -> np.ndarray:
    """Uniform random bytes: every 16-bit pattern, NaN payloads, infinities,
    signed zeros and subnormals included."""
    return stream(seed, purpose, sub).integers(0, 256, size=count, dtype=np.uint8)


def special_patterns16() -> np.ndarray:
    """16-bit patterns a copy must not disturb: fp16/bf16 signalling and
    quiet NaNs with payloads, +-Inf, +-0, smallest and largest subnormals,
    largest finite values."""
    return np.array([0x0000, 0x8000, 0x7C00, 0xFC00, 0x7C01, 0x7DFF, 0x7E00, 0xFE01, 0x0001,
                     0x8001, 0x03FF, 0x83FF, 0x7BFF, 0xFBFF, 0x7F80, 0xFF80, 0x7F81, 0x7FC0,
                     0xFFC1, 0x007F, 0x807F, 0x7F7F, 0xFF7F, 0x3C00, 0xBC00, 0xFFFF],
                    dtype=np.uint16)
