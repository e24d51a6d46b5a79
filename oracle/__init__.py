"""CPU oracle for multi-stage KV-cache live migration (Llumnix, arXiv 2406.03243).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The product path (the
HIP library and its Python binding) never imports, loads or calls it, and it
shares no code with them.

The arithmetic lives in ``llmig_oracle.c`` (plain C, memcpy per tile); this
module only marshals numpy arrays into it and adds the multi-stage replay,
which strings the C routines together in the order Llumnix §4.2 describes:
stage 0 copies the blocks already filled while decoding goes on, each later
stage copies the blocks filled during the previous one, and the final stage,
run with the request drained from its batch, copies what is left.

A host pool is a :class:`HostPool`: for each layer a K array and a V array of
``num_blocks`` tiles of ``tile_bytes`` bytes (uint8), the byte image of a
layer tensor of shape [num_blocks, block_size, kv_heads, head_dim].
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "llmig_oracle.c")
LIBRARY = os.path.join(HERE, "libllmig_oracle.so")

OK, EINVAL, ENOSPC, ERANGE = 0, -1, -2, -3
ERROR_NAMES = {OK: "OK", EINVAL: "EINVAL", ENOSPC: "ENOSPC", ERANGE: "ERANGE"}

# Intra-tile layouts of a (layer, K or V, block) tile of bs tokens, H heads,
# D dims (x = 16 / elem_bytes): NHD [bs][H][D], HND [H][bs][D],
# HCNX [H][D/x][bs][x], HDN [H][D][bs].
NHD, HND, HCNX, HDN = 0, 1, 2, 3
LAYOUT_NAMES = {NHD: "NHD", HND: "HND", HCNX: "HCNX", HDN: "HDN"}


def build(source: str = SOURCE, library: str = LIBRARY, quiet: bool = False) -> str:
    """Compile the C oracle with gcc into a shared library; returns its path."""
    tmp = library + ".tmp"
    warn = ["-w"] if quiet else ["-Wall", "-Wextra"]
    subprocess.run(["gcc", "-O2", "-std=c11", *warn, "-shared", "-fPIC", "-o", tmp, source, "-lm"],
                   check=True)
    os.replace(tmp, library)
    return library


_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_pp = ctypes.POINTER(ctypes.c_void_p)


def tile_bytes(block_size: int, kv_heads: int, head_dim: int, elem_bytes: int) -> int:
    """Bytes of one (layer, K or V, block) tile: block_size tokens of
    kv_heads * head_dim elements (Llumnix §5 "Block fusion" gives 128 KB for
    16 tokens of 16-bit LLaMA-7B)."""
    return block_size * kv_heads * head_dim * elem_bytes


@dataclass
class HostPool:
    """Host image of one instance's KV block pool (all layers, K and V)."""
    k: list            # num_layers uint8 arrays of shape [num_blocks, tile_bytes]
    v: list
    block_size: int
    slot_bytes: int    # kv_heads * head_dim * elem_bytes: one token of one layer's K or V

    @property
    def num_layers(self) -> int:
        return len(self.k)

    @property
    def num_blocks(self) -> int:
        return self.k[0].shape[0]

    @property
    def tile_bytes(self) -> int:
        return self.block_size * self.slot_bytes

    @classmethod
    def zeros(cls, num_layers, num_blocks, block_size, slot_bytes):
        t = block_size * slot_bytes
        return cls([np.zeros((num_blocks, t), np.uint8) for _ in range(num_layers)],
                   [np.zeros((num_blocks, t), np.uint8) for _ in range(num_layers)],
                   block_size, slot_bytes)

    def copy(self) -> "HostPool":
        return HostPool([a.copy() for a in self.k], [a.copy() for a in self.v],
                        self.block_size, self.slot_bytes)

    def _ptrs(self):
        for a in self.k + self.v:
            if not (a.flags.c_contiguous and a.dtype == np.uint8
                    and a.shape == (self.num_blocks, self.tile_bytes)):
                raise ValueError("host pool arrays must be contiguous uint8 [num_blocks, tile_bytes]")
        kp = (ctypes.c_void_p * self.num_layers)(*[a.ctypes.data for a in self.k])
        vp = (ctypes.c_void_p * self.num_layers)(*[a.ctypes.data for a in self.v])
        return kp, vp

    def equals(self, other: "HostPool") -> bool:
        return all(np.array_equal(a, b) for a, b in zip(self.k + self.v, other.k + other.v))


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


class Oracle:
    """Handle on one build of the C oracle (the default one, or a variant a
    test compiled itself)."""

    def __init__(self, library: str = LIBRARY):
        if not os.path.exists(library):
            build(SOURCE, library)
        lib = ctypes.CDLL(library)
        lib.oracle_plan.restype = ctypes.c_int
        lib.oracle_plan.argtypes = [_i32p, ctypes.c_int64, _i32p, ctypes.c_int64,
                                    ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                    _i32p, _i32p, ctypes.c_int64, _i64p]
        lib.oracle_copy.restype = None
        lib.oracle_copy.argtypes = [_pp, _pp, _pp, _pp, ctypes.c_int32, ctypes.c_int64,
                                    _i32p, _i32p, ctypes.c_int64]
        for name in ("oracle_pack", "oracle_unpack"):
            fn = getattr(lib, name)
            fn.restype = None
            fn.argtypes = [_pp, _pp, ctypes.c_int32, ctypes.c_int64, _i32p, ctypes.c_int64,
                           ctypes.c_void_p]
        lib.oracle_write_tokens.restype = None
        lib.oracle_write_tokens.argtypes = [_pp, _pp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                            _i32p, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_first_token_mismatch.restype = ctypes.c_int64
        lib.oracle_first_token_mismatch.argtypes = [_pp, _pp, _i32p, _pp, _pp, _i32p,
                                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                                    ctypes.c_int64]
        lib.oracle_half_to_double.restype = ctypes.c_double
        lib.oracle_half_to_double.argtypes = [ctypes.c_uint16]
        lib.oracle_bf16_to_double.restype = ctypes.c_double
        lib.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        lib.oracle_layout_offset.restype = ctypes.c_int64
        lib.oracle_layout_offset.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                             ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
        lib.oracle_copy_layout.restype = None
        lib.oracle_copy_layout.argtypes = [_pp, _pp, _i32p, _pp, _pp, _i32p, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _i32p, _i32p,
                                           ctypes.c_int64]
        lib.oracle_unpack_layout.restype = None
        lib.oracle_unpack_layout.argtypes = [_pp, _pp, _i32p, _i32p, ctypes.c_int32, ctypes.c_int32,
                                             ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _i32p,
                                             ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_write_tokens_layout.restype = None
        lib.oracle_write_tokens_layout.argtypes = [_pp, _pp, _i32p, ctypes.c_int32, ctypes.c_int32,
                                                   ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _i32p,
                                                   ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_first_token_mismatch_layout.restype = ctypes.c_int64
        lib.oracle_first_token_mismatch_layout.argtypes = [_pp, _pp, _i32p, _i32p, _pp, _pp, _i32p, _i32p,
                                                           ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                           ctypes.c_int32, ctypes.c_int32, ctypes.c_int64]
        lib.oracle_decode_attention.restype = None
        lib.oracle_decode_attention.argtypes = [_pp, _pp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                ctypes.c_int32, ctypes.c_int, ctypes.c_void_p, ctypes.c_int32,
                                                ctypes.c_int32, _i32p, ctypes.c_int32, _i32p, ctypes.c_double,
                                                ctypes.c_void_p]
        self.lib = lib

    # ---- one stage's plan (Llumnix §4.2, pre-allocation before each stage) ----
    def plan(self, src_table, dst_free_list, length, from_tok, to_tok, block_size,
             out_cap=None, sentinel=None):
        """Returns (code, map_src, map_dst).  On error both maps are empty.
        ``sentinel`` pre-fills the output arrays so a caller can check that an
        error wrote nothing."""
        st = _i32(src_table)
        fl = _i32(dst_free_list)
        cap = len(fl) if out_cap is None else out_cap
        fill = -7 if sentinel is None else sentinel
        out_s = np.full(max(cap, 1), fill, np.int32)
        out_d = np.full(max(cap, 1), fill, np.int32)
        n = ctypes.c_int64(-1)
        code = self.lib.oracle_plan(st.ctypes.data_as(_i32p), len(st), fl.ctypes.data_as(_i32p),
                                    len(fl), length, from_tok, to_tok, block_size,
                                    out_s.ctypes.data_as(_i32p), out_d.ctypes.data_as(_i32p),
                                    cap, ctypes.byref(n))
        if sentinel is not None:
            return code, out_s, out_d, n.value
        if code != OK:
            return code, np.zeros(0, np.int32), np.zeros(0, np.int32)
        return code, out_s[:n.value].copy(), out_d[:n.value].copy()

    # ---- one stage's copy ----
    def copy(self, src: HostPool, dst: HostPool, map_src, map_dst) -> None:
        ms, md = _i32(map_src), _i32(map_dst)
        assert len(ms) == len(md) and src.tile_bytes == dst.tile_bytes
        assert src.num_layers == dst.num_layers
        if len(ms):
            assert ms.min() >= 0 and ms.max() < src.num_blocks
            assert md.min() >= 0 and md.max() < dst.num_blocks
        sk, sv = src._ptrs()
        dk, dv = dst._ptrs()
        self.lib.oracle_copy(sk, sv, dk, dv, src.num_layers, src.tile_bytes,
                             ms.ctypes.data_as(_i32p), md.ctypes.data_as(_i32p), len(ms))

    # ---- block fusion ----
    def pack(self, pool: HostPool, blocks) -> np.ndarray:
        """Contiguous buffer [layer][K, V][i][tile_bytes] of the listed blocks."""
        b = _i32(blocks)
        if len(b):
            assert b.min() >= 0 and b.max() < pool.num_blocks
        out = np.zeros(pool.num_layers * 2 * len(b) * pool.tile_bytes, np.uint8)
        k, v = pool._ptrs()
        self.lib.oracle_pack(k, v, pool.num_layers, pool.tile_bytes, b.ctypes.data_as(_i32p),
                             len(b), out.ctypes.data)
        return out

    def unpack(self, pool: HostPool, blocks, staging: np.ndarray) -> None:
        b = _i32(blocks)
        if len(b):
            assert b.min() >= 0 and b.max() < pool.num_blocks
        staging = np.ascontiguousarray(staging, dtype=np.uint8)
        assert staging.size >= pool.num_layers * 2 * len(b) * pool.tile_bytes
        k, v = pool._ptrs()
        self.lib.oracle_unpack(k, v, pool.num_layers, pool.tile_bytes, b.ctypes.data_as(_i32p),
                               len(b), staging.ctypes.data)

    # ---- decoding's KV appends ----
    def write_tokens(self, pool: HostPool, table, from_tok: int, data: np.ndarray) -> None:
        """data: uint8 [num_layers][2][n_tok][slot_bytes] written to tokens
        [from_tok, from_tok + n_tok) through ``table``."""
        t = _i32(table)
        data = np.ascontiguousarray(data, dtype=np.uint8)
        n_tok = data.size // (pool.num_layers * 2 * pool.slot_bytes)
        assert data.size == pool.num_layers * 2 * n_tok * pool.slot_bytes
        if n_tok:
            assert (from_tok + n_tok - 1) // pool.block_size < len(t)
        k, v = pool._ptrs()
        self.lib.oracle_write_tokens(k, v, pool.num_layers, pool.block_size, pool.slot_bytes,
                                     t.ctypes.data_as(_i32p), from_tok, n_tok, data.ctypes.data)

    # ---- token identity ----
    def first_token_mismatch(self, a: HostPool, table_a, b: HostPool, table_b, length: int) -> int:
        ta, tb = _i32(table_a), _i32(table_b)
        assert a.slot_bytes == b.slot_bytes and a.block_size == b.block_size
        if length:
            assert (length - 1) // a.block_size < min(len(ta), len(tb))
        ak, av = a._ptrs()
        bk, bv = b._ptrs()
        return self.lib.oracle_first_token_mismatch(ak, av, ta.ctypes.data_as(_i32p), bk, bv,
                                                    tb.ctypes.data_as(_i32p), a.num_layers,
                                                    a.block_size, a.slot_bytes, length)

    # ---- cross-layout migration ----
    def layout_offset(self, layout: int, t: int, h: int, d: int, block_size: int, heads: int, head_dim: int,
                      elem_bytes: int) -> int:
        """Byte offset of element (t, h, d) in a tile of the given layout (-1: no such layout)."""
        return self.lib.oracle_layout_offset(layout, t, h, d, block_size, heads, head_dim, elem_bytes)

    @staticmethod
    def _geometry(pool: HostPool, heads: int, head_dim: int, elem_bytes: int) -> None:
        assert pool.slot_bytes == heads * head_dim * elem_bytes

    def copy_layout(self, src: HostPool, src_layouts, dst: HostPool, dst_layouts, map_src, map_dst,
                    heads: int, head_dim: int, elem_bytes: int) -> None:
        """One stage from a pool whose (K, V) tiles use ``src_layouts`` into
        one whose tiles use ``dst_layouts``: every element moves to the
        position the destination layout gives it."""
        ms, md = _i32(map_src), _i32(map_dst)
        assert len(ms) == len(md) and src.num_layers == dst.num_layers
        assert src.block_size == dst.block_size
        self._geometry(src, heads, head_dim, elem_bytes)
        self._geometry(dst, heads, head_dim, elem_bytes)
        if len(ms):
            assert ms.min() >= 0 and ms.max() < src.num_blocks
            assert md.min() >= 0 and md.max() < dst.num_blocks
        sl, dl = _i32(src_layouts), _i32(dst_layouts)
        assert len(sl) == 2 and len(dl) == 2
        for lay in list(sl) + list(dl):
            assert self.layout_offset(int(lay), 0, 0, 0, src.block_size, heads, head_dim, elem_bytes) >= 0
        sk, sv = src._ptrs()
        dk, dv = dst._ptrs()
        self.lib.oracle_copy_layout(sk, sv, sl.ctypes.data_as(_i32p), dk, dv, dl.ctypes.data_as(_i32p),
                                    src.num_layers, src.block_size, heads, head_dim, elem_bytes,
                                    ms.ctypes.data_as(_i32p), md.ctypes.data_as(_i32p), len(ms))

    def unpack_layout(self, pool: HostPool, pool_layouts, blocks, staging: np.ndarray, staging_layouts,
                      heads: int, head_dim: int, elem_bytes: int) -> None:
        """Scatter a staging buffer whose tiles follow ``staging_layouts``
        into the listed blocks of a pool whose tiles follow ``pool_layouts``."""
        self._geometry(pool, heads, head_dim, elem_bytes)
        b = _i32(blocks)
        if len(b):
            assert b.min() >= 0 and b.max() < pool.num_blocks
        staging = np.ascontiguousarray(staging, dtype=np.uint8)
        assert staging.size >= pool.num_layers * 2 * len(b) * pool.tile_bytes
        pl, sl = _i32(pool_layouts), _i32(staging_layouts)
        assert len(pl) == 2 and len(sl) == 2
        for lay in list(pl) + list(sl):
            assert self.layout_offset(int(lay), 0, 0, 0, pool.block_size, heads, head_dim, elem_bytes) >= 0
        k, v = pool._ptrs()
        self.lib.oracle_unpack_layout(k, v, pl.ctypes.data_as(_i32p), sl.ctypes.data_as(_i32p), pool.num_layers,
                                      pool.block_size, heads, head_dim, elem_bytes, b.ctypes.data_as(_i32p),
                                      len(b), staging.ctypes.data)

    def write_tokens_layout(self, pool: HostPool, layouts, table, from_tok: int, data: np.ndarray,
                            heads: int, head_dim: int, elem_bytes: int) -> None:
        """As :meth:`write_tokens` (data [L][2][n_tok][H*D*e]) into a pool of the given (K, V) layouts."""
        self._geometry(pool, heads, head_dim, elem_bytes)
        t = _i32(table)
        lay = _i32(layouts)
        data = np.ascontiguousarray(data, dtype=np.uint8)
        n_tok = data.size // (pool.num_layers * 2 * pool.slot_bytes)
        assert data.size == pool.num_layers * 2 * n_tok * pool.slot_bytes and len(lay) == 2
        if n_tok:
            assert (from_tok + n_tok - 1) // pool.block_size < len(t)
        k, v = pool._ptrs()
        self.lib.oracle_write_tokens_layout(k, v, lay.ctypes.data_as(_i32p), pool.num_layers, pool.block_size,
                                            heads, head_dim, elem_bytes, t.ctypes.data_as(_i32p), from_tok,
                                            n_tok, data.ctypes.data)

    def first_token_mismatch_layout(self, a: HostPool, a_layouts, table_a, b: HostPool, b_layouts, table_b,
                                    length: int, heads: int, head_dim: int, elem_bytes: int) -> int:
        ta, tb = _i32(table_a), _i32(table_b)
        la, lb = _i32(a_layouts), _i32(b_layouts)
        self._geometry(a, heads, head_dim, elem_bytes)
        self._geometry(b, heads, head_dim, elem_bytes)
        assert a.block_size == b.block_size
        if length:
            assert (length - 1) // a.block_size < min(len(ta), len(tb))
        ak, av = a._ptrs()
        bk, bv = b._ptrs()
        return self.lib.oracle_first_token_mismatch_layout(
            ak, av, la.ctypes.data_as(_i32p), ta.ctypes.data_as(_i32p), bk, bv, lb.ctypes.data_as(_i32p),
            tb.ctypes.data_as(_i32p), a.num_layers, a.block_size, heads, head_dim, elem_bytes, length)

    # ---- decode attention over the paged pool (the work beside a migration) ----
    def half_to_double(self, bits: int) -> float:
        return self.lib.oracle_half_to_double(bits)

    def bf16_to_double(self, bits: int) -> float:
        return self.lib.oracle_bf16_to_double(bits)

    def decode_attention(self, pool: HostPool, kv_heads: int, head_dim: int, dtype: str, q: np.ndarray,
                         tables: np.ndarray, ctx, scale: float) -> np.ndarray:
        """q: uint16 bits [L][B][Hq][D]; tables: int32 [B][stride]; ctx: [B].
        Returns float64 [L][B][Hq][D]."""
        q = np.ascontiguousarray(q, dtype=np.uint16)
        num_layers, batch, q_heads, d = q.shape
        assert num_layers == pool.num_layers and d == head_dim and q_heads % kv_heads == 0
        assert pool.slot_bytes == kv_heads * head_dim * 2
        t = np.ascontiguousarray(tables, dtype=np.int32)
        c = _i32(ctx)
        assert t.shape[0] == batch and len(c) == batch
        for b in range(batch):
            if c[b] > 0:
                need = (c[b] - 1) // pool.block_size + 1
                assert need <= t.shape[1] and t[b, :need].min() >= 0 and t[b, :need].max() < pool.num_blocks
        out = np.zeros((num_layers, batch, q_heads, head_dim), np.float64)
        k, v = pool._ptrs()
        self.lib.oracle_decode_attention(k, v, num_layers, pool.block_size, kv_heads, head_dim,
                                         1 if dtype == "bf16" else 0, q.ctypes.data, batch, q_heads,
                                         t.ctypes.data_as(_i32p), t.shape[1], c.ctypes.data_as(_i32p),
                                         float(scale), out.ctypes.data)
        return out

    # ---- multi-stage migration (Llumnix §4.2) ----
    def migrate(self, src: HostPool, dst: HostPool, src_table, dst_free_list, events, layouts=None):
        """Replay a migration on host pools.

        ``events`` is the ordered list of what happened to the request:
        ``("append", from_tok, data)`` for KV that decoding wrote into the
        source (data laid out as for :meth:`write_tokens`), and
        ``("stage", length, from_tok, to_tok)`` for a stage planned when
        ``length`` tokens were resident.  Each stage takes its destination
        blocks from the head of what is left of the free list.  Returns the
        request's destination block table (one id per logical block, in
        logical order) and the list of per-stage (map_src, map_dst).

        ``layouts`` = (src_layouts, dst_layouts, heads, head_dim, elem_bytes)
        replays a cross-layout migration: appends land in the source's
        layouts and every stage converts into the destination's."""
        free = list(_i32(dst_free_list))
        dst_table = []
        stages = []
        for ev in events:
            if ev[0] == "append":
                if layouts is None:
                    self.write_tokens(src, src_table, ev[1], ev[2])
                else:
                    self.write_tokens_layout(src, layouts[0], src_table, ev[1], ev[2], *layouts[2:])
            elif ev[0] == "stage":
                _, length, lo, hi = ev
                code, ms, md = self.plan(src_table, free, length, lo, hi, src.block_size)
                if code != OK:
                    raise RuntimeError(f"oracle plan failed: {ERROR_NAMES[code]}")
                if layouts is None:
                    self.copy(src, dst, ms, md)
                else:
                    self.copy_layout(src, layouts[0], dst, layouts[1], ms, md, *layouts[2:])
                free = free[len(md):]
                dst_table.extend(int(x) for x in md)
                stages.append((ms, md))
            else:
                raise ValueError(ev[0])
        return np.asarray(dst_table, np.int32), stages


def stage_bounds(initial_len: int, appended: list, block_size: int):
    """Token ranges of a migration's stages (Llumnix §4.2): the first stage
    copies every full block of the initial sequence; after each later batch of
    appended tokens, a non-final stage copies the full blocks completed since
    the previous stage, and the stage after the last batch is final and also
    copies the partial block.  Returns a list of (length, from_tok, to_tok)."""
    out = []
    length = initial_len
    copied = 0
    for k in range(len(appended) + 1):
        if k > 0:
            length += appended[k - 1]
        final = k == len(appended)
        end = length if final else (length // block_size) * block_size
        out.append((length, copied, end))
        copied = end
    return out


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
