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
