"""Python binding of the llmig C ABI (include/llmig.h).

Argument marshalling only: every step of a migration runs in the HIP library
``libllmig.so``.  PyTorch supplies device memory, pinned host memory and
streams; the functions take torch tensors and numpy arrays and pass their
addresses to the library.  Importing this module without the built library
raises ImportError: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(HERE, "libllmig.so")

if not os.path.exists(LIBRARY):
    raise ImportError(f"{LIBRARY} is not built; run __graft_entry__.build() first")

_lib = ctypes.CDLL(LIBRARY)

LLMIG_OK, LLMIG_EINVAL, LLMIG_ENOSPC, LLMIG_ERANGE, LLMIG_EHIP, LLMIG_ESCRATCH = 0, -1, -2, -3, -4, -5
ERROR_NAMES = {0: "OK", -1: "EINVAL", -2: "ENOSPC", -3: "ERANGE", -4: "EHIP", -5: "ESCRATCH"}
# Bytes of the static array behind llmig_decode_attention_noalloc (LLMIG_DECODE_SCRATCH_BYTES).
DECODE_SCRATCH_BYTES = 32 << 20


class LlmigError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        self.name = ERROR_NAMES.get(code, str(code))
        detail = _lib.llmig_strerror(code).decode()
        if code == LLMIG_EHIP:
            detail += f" (hipError_t {_lib.llmig_last_hip_error()})"
        super().__init__(f"{where}: {self.name}: {detail}")


class _PoolDesc(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_blocks", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("elem_bytes", ctypes.c_int32),
                ("k_ptrs", ctypes.POINTER(ctypes.c_uint64)), ("v_ptrs", ctypes.POINTER(ctypes.c_uint64)),
                ("k_layout", ctypes.c_int32), ("v_layout", ctypes.c_int32)]


# Intra-tile layouts (LLMIG_LAYOUT_*): NHD [block_size][heads][head_dim],
# HND [heads][block_size][head_dim], HCNX [heads][head_dim/x][block_size][x]
# with x = 16 / elem_bytes, HDN [heads][head_dim][block_size].
LAYOUT_NHD, LAYOUT_HND, LAYOUT_HCNX, LAYOUT_HDN = 0, 1, 2, 3


_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_vp = ctypes.c_void_p

_lib.llmig_pool_create.argtypes = [ctypes.POINTER(_PoolDesc), ctypes.POINTER(_vp)]
_lib.llmig_pool_create.restype = ctypes.c_int
_lib.llmig_pool_destroy.argtypes = [_vp]
_lib.llmig_pool_destroy.restype = None
_lib.llmig_pool_tile_bytes.argtypes = [_vp]
_lib.llmig_pool_tile_bytes.restype = ctypes.c_int64
_lib.llmig_plan.argtypes = [_vp, ctypes.c_int64, _vp, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                            ctypes.c_int64, ctypes.c_int32, _vp, _vp, ctypes.c_int64, _i64p]
_lib.llmig_plan.restype = ctypes.c_int
_lib.llmig_stage.argtypes = [_vp, _vp, _vp, _vp, ctypes.c_int64, ctypes.c_int, _vp]
_lib.llmig_stage.restype = ctypes.c_int
_lib.llmig_pack.argtypes = [_vp, _vp, ctypes.c_int64, ctypes.c_int, _vp, ctypes.c_int64, _vp]
_lib.llmig_pack.restype = ctypes.c_int
_lib.llmig_unpack.argtypes = [_vp, _vp, ctypes.c_int64, ctypes.c_int, _vp, ctypes.c_int64, _vp]
_lib.llmig_unpack.restype = ctypes.c_int
_lib.llmig_unpack_layout.argtypes = [_vp, _vp, ctypes.c_int64, ctypes.c_int, _vp, ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_int32, _vp]
_lib.llmig_unpack_layout.restype = ctypes.c_int
_lib.llmig_write_tokens.argtypes = [_vp, _vp, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, _vp, _vp]
_lib.llmig_write_tokens.restype = ctypes.c_int
_lib.llmig_stream_read.argtypes = [_vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _vp, ctypes.c_int64, _vp]
_lib.llmig_stream_read.restype = ctypes.c_int
_lib.llmig_migration_create.argtypes = [ctypes.c_int32, ctypes.POINTER(_vp)]
_lib.llmig_migration_create.restype = ctypes.c_int
_lib.llmig_migration_destroy.argtypes = [_vp]
_lib.llmig_migration_destroy.restype = None
_lib.llmig_migration_next.argtypes = [_vp, _vp, ctypes.c_int64, ctypes.c_int64, ctypes.c_int, _vp, ctypes.c_int64,
                                      _vp, _vp, ctypes.c_int64, _i64p]
_lib.llmig_migration_next.restype = ctypes.c_int
_lib.llmig_migration_stage.argtypes = [_vp, _vp, _vp, _vp, ctypes.c_int64, ctypes.c_int64, ctypes.c_int, _vp,
                                       ctypes.c_int64, _vp, _i64p]
_lib.llmig_migration_stage.restype = ctypes.c_int
_lib.llmig_migration_finish.argtypes = [_vp, _vp, _vp, _vp, ctypes.c_int64, ctypes.c_int64, _vp, ctypes.c_int64,
                                        _vp, _i64p]
_lib.llmig_migration_finish.restype = ctypes.c_int
for _name in ("llmig_migration_abort", "llmig_migration_commit"):
    getattr(_lib, _name).argtypes = [_vp, _vp, ctypes.c_int64, _i64p]
    getattr(_lib, _name).restype = ctypes.c_int
_lib.llmig_migration_set_max_workgroups.argtypes = [_vp, ctypes.c_int32]
_lib.llmig_migration_set_max_workgroups.restype = ctypes.c_int
_lib.llmig_migration_set_stage_events.argtypes = [_vp, _vp, _vp]
_lib.llmig_migration_set_stage_events.restype = ctypes.c_int
_lib.llmig_migration_info.argtypes = [_vp, ctypes.POINTER(ctypes.c_int32), _i64p, _i64p, _i64p]
_lib.llmig_migration_info.restype = ctypes.c_int
_lib.llmig_decode_attention_workspace.argtypes = [_vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                  ctypes.c_int32, _i64p]
_lib.llmig_decode_attention_workspace.restype = ctypes.c_int
_lib.llmig_decode_attention.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int32, ctypes.c_int32, _vp,
                                        ctypes.c_int32, _vp, ctypes.c_float, _vp, ctypes.c_int64, _vp, _vp]
_lib.llmig_decode_attention.restype = ctypes.c_int
_lib.llmig_decode_attention_migrate.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int32, ctypes.c_int32, _vp,
                                                ctypes.c_int32, _vp, ctypes.c_float, _vp, ctypes.c_int64, _vp,
                                                _vp, ctypes.c_int32, _vp, ctypes.c_int64, ctypes.c_int64, _vp]
_lib.llmig_decode_attention_migrate.restype = ctypes.c_int
_lib.llmig_decode_attention_noalloc.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int32, ctypes.c_int32, _vp,
                                                ctypes.c_int32, _vp, ctypes.c_float, _vp, _vp]
_lib.llmig_decode_attention_noalloc.restype = ctypes.c_int
_lib.llmig_strerror.argtypes = [ctypes.c_int]
_lib.llmig_strerror.restype = ctypes.c_char_p
_lib.llmig_last_hip_error.argtypes = []
_lib.llmig_last_hip_error.restype = ctypes.c_int


def _check(code: int, where: str) -> None:
    if code != LLMIG_OK:
        raise LlmigError(code, where)


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _used_on(stream, *tensors) -> None:
    """Tells torch's caching allocator that the device tensors are read or
    written by work on ``stream`` (a torch stream): a tensor the caller drops
    right after the call is then not handed out again before that work has
    run.  Raw stream handles carry no such record; their callers keep the
    tensors alive themselves."""
    if isinstance(stream, torch.cuda.Stream):
        for t in tensors:
            if isinstance(t, torch.Tensor) and t.is_cuda:
                t.record_stream(stream)


def _host_i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ids(a):
    """(pointer, length, on_device, keepalive) for an id list: a CUDA int32
    tensor stays on the device, anything else becomes a host int32 array."""
    if isinstance(a, torch.Tensor) and a.is_cuda:
        if a.dtype != torch.int32 or not a.is_contiguous():
            raise ValueError("device id lists must be contiguous int32 tensors")
        return a.data_ptr(), a.numel(), 1, a
    h = _host_i32(a.cpu().numpy() if isinstance(a, torch.Tensor) else a)
    return h.ctypes.data, h.size, 0, h


class Pool:
    """A registered KV block pool: per-layer K and V tensors of shape
    [num_blocks, block_size, num_kv_heads, head_dim] on one GPU.  The tensors
    stay owned by the caller; the handle keeps references to them.
    ``layouts`` gives the (K, V) intra-tile layouts: the bytes of each
    block follow them, whatever the tensors' own shape suggests."""

    def __init__(self, k_layers, v_layers, layouts=(LAYOUT_NHD, LAYOUT_NHD)):
        if len(k_layers) != len(v_layers) or not k_layers:
            raise ValueError("need one K and one V tensor per layer")
        t0 = k_layers[0]
        for t in list(k_layers) + list(v_layers):
            if (not t.is_cuda or not t.is_contiguous() or t.dim() != 4 or t.shape != t0.shape
                    or t.dtype != t0.dtype or t.device != t0.device):
                raise ValueError("layer tensors must be contiguous CUDA tensors of one 4-D shape, dtype and device")
        if t0.device.index != torch.cuda.current_device():
            raise ValueError("register a pool with its device current")
        nb, bs, heads, dim = t0.shape
        kp = (ctypes.c_uint64 * len(k_layers))(*[t.data_ptr() for t in k_layers])
        vp = (ctypes.c_uint64 * len(v_layers))(*[t.data_ptr() for t in v_layers])
        desc = _PoolDesc(len(k_layers), nb, bs, heads, dim, t0.element_size(),
                         ctypes.cast(kp, ctypes.POINTER(ctypes.c_uint64)),
                         ctypes.cast(vp, ctypes.POINTER(ctypes.c_uint64)), int(layouts[0]), int(layouts[1]))
        handle = _vp()
        _check(_lib.llmig_pool_create(ctypes.byref(desc), ctypes.byref(handle)), "llmig_pool_create")
        self._handle = handle
        self.k, self.v = list(k_layers), list(v_layers)
        self.num_layers, self.num_blocks, self.block_size = len(k_layers), nb, bs
        self.num_kv_heads, self.head_dim, self.elem_bytes = heads, dim, t0.element_size()
        self.layouts = (int(layouts[0]), int(layouts[1]))
        self.tile_bytes = _lib.llmig_pool_tile_bytes(handle)
        self.slot_bytes = self.tile_bytes // bs

    @property
    def handle(self):
        if self._handle is None:
            raise ValueError("pool is closed")
        return self._handle

    def close(self) -> None:
        # at interpreter exit the module's globals may already be gone
        if getattr(self, "_handle", None) is not None and _lib is not None:
            _lib.llmig_pool_destroy(self._handle)
            self._handle = None

    def __del__(self):
        self.close()


def llmig_plan(src_table, dst_free_list, length, from_tok, to_tok, block_size, out_cap=None):
    """Plan one stage; returns (map_src, map_dst) as host int32 arrays."""
    st, fl = _host_i32(src_table), _host_i32(dst_free_list)
    cap = len(fl) if out_cap is None else int(out_cap)
    out_s = np.empty(max(cap, 1), np.int32)
    out_d = np.empty(max(cap, 1), np.int32)
    n = ctypes.c_int64(0)
    _check(_lib.llmig_plan(st.ctypes.data, st.size, fl.ctypes.data, fl.size, int(length), int(from_tok),
                           int(to_tok), int(block_size), out_s.ctypes.data, out_d.ctypes.data, cap,
                           ctypes.byref(n)), "llmig_plan")
    return out_s[:n.value], out_d[:n.value]


def llmig_plan_code(src_table, dst_free_list, length, from_tok, to_tok, block_size, out_cap=None,
                    sentinel=None):
    """Raw form of :func:`llmig_plan` for tests: returns (code, out_src,
    out_dst, n) with the full output arrays (pre-filled with ``sentinel``)."""
    st, fl = _host_i32(src_table), _host_i32(dst_free_list)
    cap = len(fl) if out_cap is None else int(out_cap)
    out_s = np.full(max(cap, 1), -7 if sentinel is None else sentinel, np.int32)
    out_d = out_s.copy()
    n = ctypes.c_int64(-1)
    code = _lib.llmig_plan(st.ctypes.data, st.size, fl.ctypes.data, fl.size, int(length), int(from_tok),
                           int(to_tok), int(block_size), out_s.ctypes.data, out_d.ctypes.data, cap,
                           ctypes.byref(n))
    return code, out_s, out_d, n.value


def llmig_stage(src: Pool, dst: Pool, map_src, map_dst, stream=None) -> None:
    """Enqueue one pool-to-pool stage.  Host id arrays travel inside the
    kernel arguments; CUDA int32 tensors are read on the device."""
    ps, ns, ds, ks = _ids(map_src)
    pd, nd, dd, kd = _ids(map_dst)
    if ns != nd or ds != dd:
        raise ValueError("map_src and map_dst must have one length and one location")
    _check(_lib.llmig_stage(src.handle, dst.handle, ps, pd, ns, ds, _stream(stream)), "llmig_stage")
    _used_on(stream, map_src, map_dst)


def _staging(staging: torch.Tensor):
    if not staging.is_contiguous():
        raise ValueError("staging must be contiguous")
    if not staging.is_cuda and not staging.is_pinned():
        raise ValueError("host staging must be pinned memory")
    return staging.data_ptr(), staging.numel() * staging.element_size()


def llmig_pack(src: Pool, blocks, staging: torch.Tensor, stream=None) -> None:
    """Gather the listed blocks into staging laid out [L][K,V][n][tile]."""
    pb, n, on_dev, keep = _ids(blocks)
    ptr, nbytes = _staging(staging)
    _check(_lib.llmig_pack(src.handle, pb, n, on_dev, ptr, nbytes, _stream(stream)), "llmig_pack")
    _used_on(stream, blocks, staging)


def llmig_unpack(dst: Pool, blocks, staging: torch.Tensor, stream=None) -> None:
    """Scatter a buffer laid out as llmig_pack writes it into the listed blocks."""
    pb, n, on_dev, keep = _ids(blocks)
    ptr, nbytes = _staging(staging)
    _check(_lib.llmig_unpack(dst.handle, pb, n, on_dev, ptr, nbytes, _stream(stream)), "llmig_unpack")
    _used_on(stream, blocks, staging)


def llmig_unpack_layout(dst: Pool, blocks, staging: torch.Tensor, staging_layouts, stream=None) -> None:
    """Scatter a buffer packed from a pool whose (K, V) layouts were
    ``staging_layouts`` into the listed blocks, converting to dst's layouts."""
    pb, n, on_dev, keep = _ids(blocks)
    ptr, nbytes = _staging(staging)
    _check(_lib.llmig_unpack_layout(dst.handle, pb, n, on_dev, ptr, nbytes, int(staging_layouts[0]),
                                    int(staging_layouts[1]), _stream(stream)), "llmig_unpack_layout")
    _used_on(stream, blocks, staging)


def llmig_write_tokens(pool: Pool, table, from_tok: int, data: torch.Tensor, stream=None) -> None:
    """Decode stand-in: write tokens [from_tok, from_tok + n_tok) through
    ``table``; data is a CUDA tensor laid out [L][K,V][n_tok][slot_bytes]."""
    if not data.is_cuda or not data.is_contiguous():
        raise ValueError("data must be a contiguous CUDA tensor")
    nbytes = data.numel() * data.element_size()
    per_tok = pool.num_layers * 2 * pool.slot_bytes
    if nbytes % per_tok:
        raise ValueError("data size is not a whole number of tokens")
    t = _host_i32(table)
    _check(_lib.llmig_write_tokens(pool.handle, t.ctypes.data, t.size, int(from_tok), nbytes // per_tok,
                                   data.data_ptr(), _stream(stream)), "llmig_write_tokens")
    _used_on(stream, data)


MIGRATION_STATES = {0: "ACTIVE", 1: "FINISHED", 2: "COMMITTED", 3: "ABORTED"}


class MigrationHandle:
    """The library's migration coordinator (the handshake of Llumnix §4.2):
    reserves destination blocks stage by stage, aborts with their release,
    commits after the final stage."""

    def __init__(self, block_size: int):
        h = _vp()
        _check(_lib.llmig_migration_create(int(block_size), ctypes.byref(h)), "llmig_migration_create")
        self._h = h
        self.block_size = int(block_size)
        self._copied = ctypes.c_int64(0)
        self._n = ctypes.c_int64(0)
        self._n_ref = ctypes.byref(self._n)

    def close(self):
        if getattr(self, "_h", None) is not None and _lib is not None:
            _lib.llmig_migration_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def set_max_workgroups(self, n: int) -> None:
        """Cap the copy grid (0: uncapped) to leave bandwidth to decoding."""
        _check(_lib.llmig_migration_set_max_workgroups(self._h, int(n)), "llmig_migration_set_max_workgroups")

    def set_stage_events(self, start, stop) -> None:
        """Time the next stage's kernels with two torch timing events, which
        the library records right before its first launch and right after its
        last.  An event that torch has not created yet is recorded once here
        so that it exists; a reused one is passed as it is."""
        for e in (start, stop):
            if not e.cuda_event:
                e.record(torch.cuda.current_stream())
        _check(_lib.llmig_migration_set_stage_events(self._h, start.cuda_event, stop.cuda_event),
               "llmig_migration_set_stage_events")

    def copied_tokens(self) -> int:
        """Tokens the stages so far have copied (the coordinator's own count)."""
        _check(_lib.llmig_migration_info(self._h, None, ctypes.byref(self._copied), None, None),
               "llmig_migration_info")
        return self._copied.value

    def info(self):
        st, cp, rs, ns = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(_lib.llmig_migration_info(self._h, ctypes.byref(st), ctypes.byref(cp), ctypes.byref(rs),
                                         ctypes.byref(ns)), "llmig_migration_info")
        return {"state": MIGRATION_STATES[st.value], "copied_tokens": cp.value, "reserved_blocks": rs.value,
                "stages": ns.value}

    def next(self, src_table, length: int, final: bool, dst_free_list):
        """Plan and reserve the next stage without copying; returns (map_src, map_dst)."""
        st, fl = _host_i32(src_table), _host_i32(dst_free_list)
        cap = max(fl.size, 1)
        out_s, out_d = np.empty(cap, np.int32), np.empty(cap, np.int32)
        n = ctypes.c_int64(0)
        _check(_lib.llmig_migration_next(self._h, st.ctypes.data, st.size, int(length), int(bool(final)),
                                         fl.ctypes.data, fl.size, out_s.ctypes.data, out_d.ctypes.data, cap,
                                         ctypes.byref(n)), "llmig_migration_next")
        return out_s[:n.value].copy(), out_d[:n.value].copy()

    def stage_ptrs(self, src_handle, dst_handle, table_ptr: int, table_len: int, length: int, final: bool,
                   free_ptr: int, free_len: int, stream_ptr: int) -> int:
        """stage() with every argument already an address or an int (the
        caller keeps the arrays alive): marshalling without conversions, for
        drivers that call it on the downtime path."""
        code = _lib.llmig_migration_stage(self._h, src_handle, dst_handle, table_ptr, table_len, length,
                                          1 if final else 0, free_ptr, free_len, stream_ptr, self._n_ref)
        if code != LLMIG_OK:
            err = LlmigError(code, "llmig_migration_stage")
            err.consumed = self._n.value
            raise err
        return self._n.value

    def finish_ptrs(self, src_handle, dst_handle, table_ptr: int, table_len: int, length: int, free_ptr: int,
                    free_len: int, stream_ptr: int) -> int:
        """The final stage and the wait for it (llmig_migration_finish),
        arguments as for stage_ptrs; returns the free-list entries consumed."""
        code = _lib.llmig_migration_finish(self._h, src_handle, dst_handle, table_ptr, table_len, length, free_ptr,
                                           free_len, stream_ptr, self._n_ref)
        if code != LLMIG_OK:
            err = LlmigError(code, "llmig_migration_finish")
            err.consumed = self._n.value
            raise err
        return self._n.value

    def stage(self, src: "Pool", dst: "Pool", src_table: np.ndarray, length: int, final: bool,
              dst_free_list: np.ndarray, stream=None) -> int:
        """Plan, reserve and launch the next stage; returns the number of
        free-list entries consumed.  A HIP error after the reservation
        raises with ``consumed`` set to the entries reserved all the same
        (an abort returns them); other errors consume nothing."""
        st, fl = _host_i32(src_table), _host_i32(dst_free_list)
        n = ctypes.c_int64(0)
        code = _lib.llmig_migration_stage(self._h, src.handle, dst.handle, st.ctypes.data, st.size,
                                          int(length), int(bool(final)), fl.ctypes.data,
                                          fl.size, _stream(stream), ctypes.byref(n))
        if code != LLMIG_OK:
            err = LlmigError(code, "llmig_migration_stage")
            err.consumed = n.value
            raise err
        return n.value

    def _take(self, fn, where):
        cap = max(self.info()["reserved_blocks"], 1)
        out = np.empty(cap, np.int32)
        n = ctypes.c_int64(0)
        _check(fn(self._h, out.ctypes.data, cap, ctypes.byref(n)), where)
        return out[:n.value].copy()

    def abort(self) -> np.ndarray:
        """Abort; returns the reserved destination blocks to release."""
        return self._take(_lib.llmig_migration_abort, "llmig_migration_abort")

    def commit(self) -> np.ndarray:
        """Commit after the final stage; returns the destination block table."""
        return self._take(_lib.llmig_migration_commit, "llmig_migration_commit")


def decode_workspace_bytes(ctx_lens, num_layers: int, q_heads: int, head_dim: int) -> int:
    c = _host_i32(ctx_lens)
    n = ctypes.c_int64(0)
    _check(_lib.llmig_decode_attention_workspace(c.ctypes.data, c.size, int(num_layers), int(q_heads),
                                                 int(head_dim), ctypes.byref(n)), "llmig_decode_attention_workspace")
    return n.value


def _attention_args(pool: Pool, q: torch.Tensor, tables: torch.Tensor, ctx_lens, out: torch.Tensor) -> np.ndarray:
    if q.dtype not in (torch.float16, torch.bfloat16) or not q.is_cuda or not q.is_contiguous():
        raise ValueError("q must be a contiguous CUDA fp16/bf16 tensor")
    if q.dim() != 4 or q.shape[0] != pool.num_layers or q.shape[3] != pool.head_dim or q.dtype != pool.k[0].dtype:
        raise ValueError("q must be [num_layers][batch][q_heads][head_dim] of the pool's layers and type")
    if tables.dtype != torch.int32 or not tables.is_cuda or not tables.is_contiguous() or tables.dim() != 2:
        raise ValueError("tables must be a contiguous CUDA int32 [batch][stride] tensor")
    if out.dtype != torch.float32 or not out.is_cuda or not out.is_contiguous() or out.shape != q.shape:
        raise ValueError("out must be a contiguous CUDA float32 tensor shaped like q")
    c = _host_i32(ctx_lens)
    if c.size != q.shape[1] or tables.shape[0] < q.shape[1]:
        raise ValueError("ctx_lens must hold one length per sequence of q, tables one row each")
    return c


def llmig_decode_attention(pool: Pool, q: torch.Tensor, tables: torch.Tensor, ctx_lens, scale: float,
                           workspace: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    """Decode attention over ``pool`` (the work beside a migration).  q: CUDA
    [L][B][Hq][D] fp16/bf16; tables: CUDA int32 [B][stride]; ctx_lens: host
    lengths; out: CUDA float32 [L][B][Hq][D]."""
    c = _attention_args(pool, q, tables, ctx_lens, out)
    if not workspace.is_cuda or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous CUDA tensor")
    _check(_lib.llmig_decode_attention(pool.handle, 1 if q.dtype == torch.bfloat16 else 0, q.data_ptr(),
                                       q.shape[1], q.shape[2], tables.data_ptr(), tables.shape[1],
                                       c.ctypes.data, float(scale), workspace.data_ptr(),
                                       workspace.numel() * workspace.element_size(), out.data_ptr(),
                                       _stream(stream)), "llmig_decode_attention")
    _used_on(stream, q, tables, workspace, out)


def llmig_decode_attention_migrate(pool: Pool, q: torch.Tensor, tables: torch.Tensor, ctx_lens, scale: float,
                                   workspace: torch.Tensor, out: torch.Tensor, dst: Pool, seq: int,
                                   dst_ids: torch.Tensor, from_block: int, stream=None) -> None:
    """llmig_decode_attention that also carries a migration stage: logical
    blocks [from_block, from_block + len(dst_ids)) of sequence ``seq`` are
    written into ``dst`` blocks ``dst_ids`` (a CUDA int32 tensor) as the
    attention reads them."""
    c = _attention_args(pool, q, tables, ctx_lens, out)
    if not workspace.is_cuda or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous CUDA tensor")
    if dst_ids.dtype != torch.int32 or not dst_ids.is_cuda or not dst_ids.is_contiguous() or dst_ids.dim() != 1:
        raise ValueError("dst_ids must be a contiguous CUDA int32 vector")
    _check(_lib.llmig_decode_attention_migrate(pool.handle, 1 if q.dtype == torch.bfloat16 else 0, q.data_ptr(),
                                               q.shape[1], q.shape[2], tables.data_ptr(), tables.shape[1],
                                               c.ctypes.data, float(scale), workspace.data_ptr(),
                                               workspace.numel() * workspace.element_size(), out.data_ptr(),
                                               dst.handle, int(seq), dst_ids.data_ptr(), int(from_block),
                                               int(from_block) + dst_ids.numel(), _stream(stream)),
           "llmig_decode_attention_migrate")
    _used_on(stream, q, tables, workspace, out, dst_ids)


def llmig_stream_read(region: torch.Tensor, passes: int, workgroups: int, out: torch.Tensor, stream=None) -> None:
    """Harness: read ``region`` ``passes`` times on ``workgroups`` workgroups
    (decode stand-in); ``out`` is a CUDA int64 tensor of workgroups * 256."""
    if (not region.is_cuda or not out.is_cuda or out.dtype != torch.int64 or not region.is_contiguous()
            or not out.is_contiguous()):
        raise ValueError("region and out must be contiguous CUDA tensors, out int64")
    _check(_lib.llmig_stream_read(region.data_ptr(), region.numel() * region.element_size(), int(passes),
                                  int(workgroups), out.data_ptr(), out.numel(), _stream(stream)),
           "llmig_stream_read")
    _used_on(stream, region, out)


def llmig_decode_attention_noalloc(pool: Pool, q: torch.Tensor, tables: torch.Tensor, ctx_lens, scale: float,
                                   out: torch.Tensor, stream=None) -> None:
    """llmig_decode_attention with its partial results in the library's
    static device array (for callers that cannot allocate); raises
    LlmigError ESCRATCH when they need more than DECODE_SCRATCH_BYTES."""
    c = _attention_args(pool, q, tables, ctx_lens, out)
    _check(_lib.llmig_decode_attention_noalloc(pool.handle, 1 if q.dtype == torch.bfloat16 else 0, q.data_ptr(),
                                               q.shape[1], q.shape[2], tables.data_ptr(), tables.shape[1],
                                               c.ctypes.data, float(scale), out.data_ptr(), _stream(stream)),
           "llmig_decode_attention_noalloc")
    _used_on(stream, q, tables, out)
