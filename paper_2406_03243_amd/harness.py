"""Device-side plumbing for synthetic migration runs: allocating layer
tensors, filling them from the seeded generators, and copying pools or
single blocks back to host memory for checking.  Holds none of the
migration's arithmetic."""
from __future__ import annotations

import numpy as np
import torch

from . import workloads as wl

TORCH_DTYPE = {"fp16": torch.float16, "bf16": torch.bfloat16}


def alloc_layers(shape: wl.PoolShape, device="cuda", num_blocks=None):
    """Per-layer K and V tensors [num_blocks, block_size, kv_heads, head_dim]."""
    nb = shape.num_blocks if num_blocks is None else num_blocks
    dims = (nb, shape.block_size, shape.kv_heads, shape.head_dim)
    dt = TORCH_DTYPE[shape.dtype]
    k = [torch.empty(dims, dtype=dt, device=device) for _ in range(shape.num_layers)]
    v = [torch.empty(dims, dtype=dt, device=device) for _ in range(shape.num_layers)]
    return k, v


def fill_from_host(tensors, seed: int, purpose: int, dtype: str) -> None:
    """Fill tensors with seeded values drawn on the host (small pools): the
    same seed gives the same bytes on every machine."""
    for idx, t in enumerate(tensors):
        bits = wl.values16(seed, purpose, t.numel(), dtype, sub=idx)
        t.copy_(torch.from_numpy(bits.view(np.int16)).view(t.dtype).reshape(t.shape))


def fill_bytes_from_host(tensors, data: np.ndarray) -> None:
    """Fill tensors, in order, with the given raw bytes."""
    off = 0
    for t in tensors:
        n = t.numel() * t.element_size()
        t.view(torch.uint8).reshape(-1).copy_(torch.from_numpy(data[off:off + n]))
        off += n


def fill_on_device(tensors, seed: int) -> None:
    """Fill large tensors with values uniform in [-1, 1] from a seeded device
    generator (fast; the checks read the result back rather than re-draw it)."""
    g = torch.Generator(device=tensors[0].device)
    g.manual_seed(seed)
    for t in tensors:
        t.uniform_(-1.0, 1.0, generator=g)


def tile_view(t: torch.Tensor) -> torch.Tensor:
    """[num_blocks, tile_bytes] uint8 view of a layer tensor."""
    return t.view(torch.uint8).reshape(t.shape[0], -1)


def snapshot(tensors):
    """Host copies of whole layer tensors as uint8 [num_blocks, tile_bytes]."""
    return [tile_view(t).cpu().numpy() for t in tensors]


def snapshot_blocks(tensors, ids):
    """Host copies of the listed blocks of every tensor, uint8 [len(ids), tile_bytes]."""
    idx = torch.as_tensor(np.asarray(ids, dtype=np.int64), device=tensors[0].device)
    return [tile_view(t).index_select(0, idx).cpu().numpy() for t in tensors]


def concurrent_streams(n: int, candidates: int = 16, probe_bytes: int = 4 * 10**9):
    """``n`` torch streams whose kernels run side by side, and whether they do.

    Streams share the GPU's few hardware queues, and the kernels of two
    streams on one queue run one after the other, so streams meant to
    overlap (a migration beside decoding, double-buffered copies) are chosen
    by measurement: a stream joins the set when a short read launched on it
    completes while a long read on each stream already chosen is still
    running.  When ``candidates`` fresh streams hold no such set (a profiler
    that serialises kernels, say), the set is filled with the remaining
    candidates and the flag is False.  Returns (streams, overlap)."""
    from .llmig import llmig_stream_read

    dev = torch.device("cuda", torch.cuda.current_device())
    long_region = torch.empty(probe_bytes, dtype=torch.uint8, device=dev)
    short_region = torch.empty(16 << 20, dtype=torch.uint8, device=dev)
    long_region.zero_()
    short_region.zero_()
    sink_long = torch.empty(256 * 256, dtype=torch.int64, device=dev)
    sink_short = torch.empty(64 * 256, dtype=torch.int64, device=dev)
    torch.cuda.synchronize()

    def overlaps(a, b) -> bool:
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record(a)
        llmig_stream_read(long_region, 1, 256, sink_long, stream=a)
        e[1].record(a)
        llmig_stream_read(short_region, 1, 64, sink_short, stream=b)
        e[2].record(b)
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[2]) < 0.5 * e[0].elapsed_time(e[1])

    chosen, rest = [], []
    for _ in range(candidates):
        s = torch.cuda.Stream(device=dev)
        if all(overlaps(c, s) and overlaps(s, c) for c in chosen):
            chosen.append(s)
            if len(chosen) == n:
                break
        else:
            rest.append(s)
    del long_region, short_region, sink_long, sink_short
    overlap = len(chosen) == n
    chosen += rest[:n - len(chosen)]
    return chosen, overlap
