"""Full-size synthetic workloads, set up once for both the benchmark and the
full-size parity tests (so the tests check exactly the configuration the
benchmark times).  Every input comes from the seeded generators in
:mod:`workloads`; large pools are filled on the device."""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

from . import harness
from . import workloads as wl
from .llmig import Pool


@dataclass
class Setup:
    workload: wl.Workload
    shape: wl.PoolShape
    src: Pool
    dst: Pool
    tables: list                   # one source block table per request
    lengths: list                  # initial length of each request
    free: np.ndarray               # destination free list
    src_occupied: np.ndarray       # source blocks held by other requests
    dst_occupied: np.ndarray       # destination blocks held by other requests
    appends: list = field(default_factory=list)   # device tensors [L][2][n][slot] per incremental stage
    counts: list = field(default_factory=list)    # tokens per append batch
    extra: dict = field(default_factory=dict)

    def close(self):
        self.src.close()
        self.dst.close()
        self.appends.clear()
        self.extra.clear()


def _pools(shape: wl.PoolShape, seed: int, dev, num_blocks=None):
    sk, sv = harness.alloc_layers(shape, device=dev, num_blocks=num_blocks)
    dk, dv = harness.alloc_layers(shape, device=dev, num_blocks=num_blocks)
    harness.fill_on_device(sk + sv, seed * 16 + wl.SRC_VALUES)
    harness.fill_on_device(dk + dv, seed * 16 + wl.DST_VALUES)
    return Pool(sk, sv), Pool(dk, dv)


def _append_data(shape, seed, counts, slot_bytes, dev):
    out = []
    for k, c in enumerate(counts):
        bits = wl.values16(seed, wl.APPEND_VALUES, shape.num_layers * 2 * int(c) * slot_bytes // 2,
                           shape.dtype, sub=k)
        out.append(torch.from_numpy(bits.view(np.uint8)).to(dev))
    return out


def llama7b(dev="cuda") -> Setup:
    """LLaMA-7B-shaped multi-stage migration: 8192 tokens, then four seeded
    batches of 16-64 appended tokens, each followed by a stage."""
    w = wl.LLAMA7B
    src, dst = _pools(w.shape, w.seed, dev)
    table, socc = wl.request_table(w.seed, w.shape.num_blocks, w.table_blocks, w.src_preoccupied)
    free, docc = wl.free_list(w.seed, w.shape.num_blocks, w.dst_preoccupied)
    counts = [int(c) for c in wl.append_counts(w.seed, w.appends, w.append_lo, w.append_hi)]
    return Setup(w, w.shape, src, dst, [table], [w.lengths[0]], free, socc, docc,
                 _append_data(w.shape, w.seed, counts, src.slot_bytes, dev), counts)


def llama30b_quarter(dev="cuda", max_append=256) -> Setup:
    """One tensor-parallel rank's quarter of LLaMA-30B (60 layers, 13 heads);
    lengths 1k/4k/16k; decoding simulated by a pool of appendable tokens."""
    w = wl.LLAMA30B_TP4
    src, dst = _pools(w.shape, w.seed, dev)
    table, socc = wl.request_table(w.seed, w.shape.num_blocks, w.table_blocks)
    free, docc = wl.free_list(w.seed, w.shape.num_blocks)
    bits = wl.values16(w.seed, wl.APPEND_VALUES, w.shape.num_layers * 2 * max_append * src.slot_bytes // 2,
                       w.shape.dtype)
    pool = torch.from_numpy(bits.view(np.uint8).reshape(w.shape.num_layers, 2, max_append, src.slot_bytes))
    return Setup(w, w.shape, src, dst, [table], list(w.lengths), free, socc, docc,
                 extra={"append_pool": pool.to(dev)})


BATCH_REQUESTS, BATCH_MEDIAN, BATCH_SIGMA, BATCH_MIN, BATCH_MAX = 64, 512, 1.0, 64, 16384


def batched(dev="cuda") -> Setup:
    """64 requests with lognormal lengths (median 512, sigma 1.0, clipped to
    [64, 16384]) in a source pool whose other half is held by other requests;
    the destination has the same size, half pre-occupied.  Pools hold
    2 x (blocks of all requests), rounded up to 256 blocks."""
    w = wl.BATCHED
    lengths = wl.lognormal_lengths(w.seed, BATCH_REQUESTS, BATCH_MEDIAN, BATCH_SIGMA, BATCH_MIN, BATCH_MAX)
    bs = w.shape.block_size
    counts = [math.ceil(int(n) / bs) for n in lengths]
    nb = math.ceil(2 * sum(counts) / 256) * 256
    shape = wl.PoolShape(w.shape.num_layers, nb, bs, w.shape.kv_heads, w.shape.head_dim, w.shape.dtype)
    if 2 * nb * shape.num_layers * 2 * bs * shape.kv_heads * shape.head_dim * shape.elem_bytes > 200 * 2**30:
        raise RuntimeError("batched pools would exceed 200 GiB")
    src, dst = _pools(shape, w.seed, dev)
    tables, socc = wl.request_tables(w.seed, nb, counts, w.src_preoccupied)
    free, docc = wl.free_list(w.seed, nb, w.dst_preoccupied)
    return Setup(w, shape, src, dst, tables, [int(n) for n in lengths], free, socc, docc)


READER_BYTES = 40 * 10**9


def gqa_long(dev="cuda", max_append=256) -> Setup:
    """GQA long-context migration under load: 80 layers, 8 KV heads, bf16,
    one 32768-token request, and a separate 40 GB region a concurrent
    streaming reader walks over."""
    w = wl.GQA_LONG
    src, dst = _pools(w.shape, w.seed, dev)
    table, socc = wl.request_table(w.seed, w.shape.num_blocks, w.table_blocks)
    free, docc = wl.free_list(w.seed, w.shape.num_blocks)
    bits = wl.values16(w.seed, wl.APPEND_VALUES, w.shape.num_layers * 2 * max_append * src.slot_bytes // 2,
                       w.shape.dtype)
    pool = torch.from_numpy(bits.view(np.uint8).reshape(w.shape.num_layers, 2, max_append, src.slot_bytes))
    region = torch.empty(READER_BYTES // 2, dtype=torch.bfloat16, device=dev)
    harness.fill_on_device([region], w.seed * 16 + wl.EXTRA)
    return Setup(w, w.shape, src, dst, [table], [w.lengths[0]], free, socc, docc,
                 extra={"append_pool": pool.to(dev), "region": region})


def decode_batch(su: Setup, n_seq: int = 16, q_heads: int = 64, seed_purpose: int = wl.EXTRA, dev="cuda"):
    """A decode batch on the source instance of a GQA setup: ``n_seq``
    requests filling the blocks the migrating request does not use (equal
    shares, random order) plus the migrating request itself with its initial
    length.  Returns (tables [B][stride] int32 device tensor, context
    lengths, q [L][B][q_heads][D] device tensor)."""
    shape, table = su.shape, su.tables[0]
    rest = np.setdiff1d(np.arange(shape.num_blocks, dtype=np.int32), table)
    g = wl.stream(su.workload.seed, seed_purpose, 11)
    rest = g.permutation(rest)
    per = len(rest) // n_seq
    stride = max(per, len(table))
    tabs = np.zeros((n_seq + 1, stride), np.int32)
    for k in range(n_seq):
        tabs[k, :per] = rest[k * per:(k + 1) * per]
    tabs[n_seq, :len(table)] = table
    ctx = [per * shape.block_size] * n_seq + [su.lengths[0]]
    bits = wl.values16(su.workload.seed, seed_purpose, shape.num_layers * (n_seq + 1) * q_heads * shape.head_dim,
                       shape.dtype, sub=12)
    q = torch.from_numpy(bits.view(np.int16)).view(harness.TORCH_DTYPE[shape.dtype]).reshape(
        shape.num_layers, n_seq + 1, q_heads, shape.head_dim)
    return torch.from_numpy(tabs).to(dev), ctx, q.to(dev)
