"""Host-side checks that need no GPU: the C-ABI library loads and exports
everything include/llmig.h declares, its planner agrees with the oracle's on
every small case and every error class, and the argument checks of the
enqueueing calls fail before touching the GPU."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest
import torch

import oracle
from paper_2406_03243_amd import workloads as wl
from paper_2406_03243_amd import llmig

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
           if f.endswith(".h")]


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names.update(re.findall(r"\b(llmig_\w+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert {"llmig_plan", "llmig_stage", "llmig_pack", "llmig_unpack"} <= set(names)
    lib = ctypes.CDLL(llmig.LIBRARY)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_error_codes_match_header():
    text = open(os.path.join(ROOT, "include", "llmig.h")).read()
    codes = {m[0]: int(m[1]) for m in re.findall(r"#define (LLMIG_\w+) \((-?\d+)\)", text)}
    codes.update({m[0]: int(m[1]) for m in re.findall(r"#define (LLMIG_OK) (\d+)", text)})
    assert codes == {"LLMIG_OK": 0, "LLMIG_EINVAL": -1, "LLMIG_ENOSPC": -2, "LLMIG_ERANGE": -3,
                     "LLMIG_EHIP": -4, "LLMIG_ESCRATCH": -5}
    for name, code in codes.items():
        assert llmig.ERROR_NAMES[code] == name[len("LLMIG_"):]
        assert llmig._lib.llmig_strerror(code)
    assert llmig._lib.llmig_strerror(12345) == b"unknown error"


def _both(table, free, length, lo, hi, bs, out_cap=None):
    got = llmig.llmig_plan_code(table, free, length, lo, hi, bs, out_cap=out_cap, sentinel=-9)
    want = oracle.default().plan(table, free, length, lo, hi, bs, out_cap=out_cap, sentinel=-9)
    return got, want


def test_plan_matches_oracle_exhaustive():
    rng = np.random.default_rng(101)
    for bs in (1, 2, 3, 4, 16):
        for length in range(0, 49):
            nb = -(-length // bs)
            ids = rng.permutation(300).astype(np.int32)
            table, free = ids[:nb], ids[nb:nb + nb + 1]
            for lo in range(0, length + 1):
                for hi in range(0, length + 1):
                    got, want = _both(table, free, length, lo, hi, bs)
                    assert got[0] == want[0], (bs, length, lo, hi)
                    assert got[3] == want[3]
                    assert np.array_equal(got[1], want[1]) and np.array_equal(got[2], want[2])


def test_plan_matches_oracle_random_and_errors():
    rng = np.random.default_rng(202)
    codes = set()
    for trial in range(4000):
        bs = int(rng.choice([1, 2, 4, 8, 16, 32]))
        length = int(rng.integers(0, 3000))
        nb = -(-length // bs)
        ids = rng.permutation(4 * nb + 64).astype(np.int32)
        table = ids[:max(0, nb + int(rng.integers(-2, 3)))]
        free = ids[len(table):len(table) + int(rng.integers(0, nb + 4))]
        lo = int(rng.integers(0, length + 2)) // bs * bs if rng.random() < 0.8 else int(rng.integers(0, length + 2))
        hi = length if rng.random() < 0.4 else int(rng.integers(lo if lo <= length else 0, length + 2))
        if rng.random() < 0.7 and hi != length:
            hi = hi // bs * bs
        table, free = table.copy(), free.copy()
        if rng.random() < 0.05 and len(table) > 1:
            table[rng.integers(len(table))] = -int(rng.integers(1, 5))
        if rng.random() < 0.05 and len(free) > 1:
            free[rng.integers(len(free))] = free[0]
        if rng.random() < 0.05 and len(table) > 1:
            table[rng.integers(len(table))] = table[0]
        cap = None if rng.random() < 0.9 else int(rng.integers(0, nb + 2))
        got, want = _both(table, free, length, lo, hi, bs, out_cap=cap)
        assert got[0] == want[0], (trial, bs, length, lo, hi)
        assert got[3] == want[3]
        assert np.array_equal(got[1], want[1]) and np.array_equal(got[2], want[2])
        codes.add(got[0])
    assert codes == {0, -1, -2, -3}


def test_plan_null_arguments():
    lib = llmig._lib
    n = ctypes.c_int64(5)
    assert lib.llmig_plan(None, 0, None, 0, 0, 0, 0, 16, None, None, 0, None) == llmig.LLMIG_EINVAL
    assert lib.llmig_plan(None, 0, None, 0, 0, 0, 0, 16, None, None, 0, ctypes.byref(n)) == 0
    assert n.value == 0
    assert lib.llmig_plan(None, 0, None, 0, 20, 0, 16, 16, None, None, 0, ctypes.byref(n)) == llmig.LLMIG_EINVAL


def test_plan_large_ids_no_huge_scratch():
    table = np.array([2**31 - 1 - k for k in range(100)], np.int32)
    free = np.array([2**31 - 1000 - k for k in range(100)], np.int32)
    ms, md = llmig.llmig_plan(table, free, 1600, 0, 1600, 16)
    assert np.array_equal(ms, table) and np.array_equal(md, free)


def test_enqueue_calls_reject_bad_arguments_without_gpu():
    lib = llmig._lib
    assert lib.llmig_stage(None, None, None, None, 0, 0, None) == llmig.LLMIG_EINVAL
    assert lib.llmig_pack(None, None, 0, 0, None, 0, None) == llmig.LLMIG_EINVAL
    assert lib.llmig_unpack(None, None, 0, 0, None, 0, None) == llmig.LLMIG_EINVAL
    assert lib.llmig_unpack_layout(None, None, 0, 0, None, 0, 0, 0, None) == llmig.LLMIG_EINVAL
    assert lib.llmig_unpack_layout(None, None, 0, 0, None, 0, 1, 3, None) == llmig.LLMIG_EINVAL
    assert lib.llmig_unpack_layout(None, None, 0, 0, None, 0, 4, 0, None) == llmig.LLMIG_EINVAL
    assert lib.llmig_write_tokens(None, None, 0, 0, 0, None, None) == llmig.LLMIG_EINVAL
    assert lib.llmig_decode_attention_noalloc(None, 0, None, 1, 1, None, 1, None, 1.0, None,
                                              None) == llmig.LLMIG_EINVAL
    assert lib.llmig_pool_create(None, None) == llmig.LLMIG_EINVAL
    out = ctypes.c_void_p(1)
    assert lib.llmig_pool_create(None, ctypes.byref(out)) == llmig.LLMIG_EINVAL and not out.value
    lib.llmig_pool_destroy(None)
    assert lib.llmig_pool_tile_bytes(None) == -1


def test_pool_desc_validation_without_gpu():
    lib = llmig._lib
    ptrs = (ctypes.c_uint64 * 2)(0x1000, 0x2000)
    bad_align = (ctypes.c_uint64 * 2)(0x1008, 0x2000)
    overlap = (ctypes.c_uint64 * 2)(0x1000, 0x1000)
    out = ctypes.c_void_p()
    cases = [
        (2, 4, 16, 1, 1, 2, ptrs, ptrs),     # tile of 32 B fine, but K and V share memory
        (2, 4, 1, 1, 1, 2, ptrs, ptrs),      # 2-byte tile: not a multiple of 16
        (0, 4, 16, 1, 8, 2, ptrs, ptrs),     # no layers
        (2, 0, 16, 1, 8, 2, ptrs, ptrs),     # no blocks
        (2, 4, 16, 1, 8, 2, bad_align, ptrs),
        (2, 4, 16, 1, 8, 2, ptrs, overlap),
    ]
    other = (ctypes.c_uint64 * 2)(0x100000, 0x200000)
    layout_cases = [
        (2, 4, 16, 1, 8, 2, ptrs, other, 4, 0),                       # no such layout
        (2, 4, 16, 1, 8, 2, ptrs, other, 0, -1),
        (2, 4, 16, 1, 4, 2, ptrs, other, llmig.LAYOUT_HCNX, 0),       # head_dim * 2 not a multiple of 16
        (2, 4, 16, 3, 16, 1, ptrs, ptrs, llmig.LAYOUT_HDN, 0),        # a valid layout; K and V share memory
    ]
    for L, nb, bs, h, d, e, kp, vp, *lay in cases + layout_cases:
        lk, lv = lay if lay else (0, 0)
        desc = llmig._PoolDesc(L, nb, bs, h, d, e, ctypes.cast(kp, ctypes.POINTER(ctypes.c_uint64)),
                               ctypes.cast(vp, ctypes.POINTER(ctypes.c_uint64)), lk, lv)
        assert lib.llmig_pool_create(ctypes.byref(desc), ctypes.byref(out)) == llmig.LLMIG_EINVAL
        assert not out.value


def test_workload_generators_are_seeded_and_shaped():
    a, occ = wl.request_table(1002, 4096, 528, 0.4)
    b, _ = wl.request_table(1002, 4096, 528, 0.4)
    assert np.array_equal(a, b) and len(set(a.tolist())) == 528
    assert len(occ) == round(0.4 * 4096) and not set(a.tolist()) & set(occ.tolist())
    f, focc = wl.free_list(1002, 4096, 0.4)
    assert len(f) + len(focc) == 4096 and not set(f.tolist()) & set(focc.tolist())
    c = wl.append_counts(1002, 4, 16, 64)
    assert len(c) == 4 and c.min() >= 16 and c.max() <= 64
    lens = wl.lognormal_lengths(1004, 64, 512, 1.0, 64, 16384)
    assert lens.min() >= 64 and lens.max() <= 16384 and 200 < np.median(lens) < 1300
    for dt in ("fp16", "bf16"):
        bits = wl.values16(5, wl.SRC_VALUES, 10000, dt)
        t = torch.from_numpy(bits.view(np.int16)).view(torch.float16 if dt == "fp16" else torch.bfloat16)
        x = t.float()
        assert x.min() >= -1 and x.max() <= 1 and x.std() > 0.5
    # bf16 rounding agrees with torch's round-to-nearest-even conversion
    g = wl.stream(5, wl.SRC_VALUES)
    ref = torch.from_numpy(g.uniform(-1.0, 1.0, size=10000).astype(np.float32)).to(torch.bfloat16)
    assert torch.equal(ref.view(torch.int16),
                       torch.from_numpy(wl.values16(5, wl.SRC_VALUES, 10000, "bf16").view(np.int16)))


C_CLIENT = r"""
#include <stdio.h>
#include "llmig.h"

int main(void)
{
    /* a request of 40 tokens in blocks of 16: three logical blocks */
    const int32_t table[3] = {7, 2, 9};
    const int32_t free_list[4] = {11, 12, 13, 14};
    int32_t out_src[4], out_dst[4];
    int64_t n = -1;
    llmig_pool_desc desc = {0};
    llmig_pool *pool = NULL;
    int rc = llmig_plan(table, 3, free_list, 4, 40, 16, 40, 16, out_src, out_dst, 4, &n);
    if (rc != LLMIG_OK || n != 2 || out_src[0] != 2 || out_src[1] != 9 || out_dst[0] != 11 || out_dst[1] != 12)
        return 1;
    if (llmig_plan(table, 3, free_list, 1, 40, 0, 40, 16, out_src, out_dst, 4, &n) != LLMIG_ENOSPC || n != 0)
        return 2;
    if (llmig_pool_create(&desc, &pool) != LLMIG_EINVAL || pool != NULL)
        return 3;
    printf("%s\n", llmig_strerror(LLMIG_ERANGE));
    return 0;
}
"""


def test_header_is_plain_c(tmp_path):
    """llmig.h compiles as C99 with every warning an error, and a C program
    linked against the library plans a stage through it (no GPU needed)."""
    src = tmp_path / "client.c"
    src.write_text(C_CLIENT)
    exe = tmp_path / "client"
    lib_dir = os.path.dirname(llmig.LIBRARY)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(ROOT, "include"),
                    str(src), "-o", str(exe), "-L", lib_dir, "-lllmig", "-Wl,-rpath," + lib_dir], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert res.returncode == 0, (res.returncode, res.stderr)
    assert res.stdout.strip() == "block id out of range"
