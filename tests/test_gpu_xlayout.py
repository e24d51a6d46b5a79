"""GPU parity of cross-layout migration: stages between pools whose K and V
tiles keep their elements in different intra-tile layouts, against the CPU
oracle, byte for byte (tolerance 0: the conversion moves 16-bit elements
unchanged).  Every case runs through the C ABI and prints its name first."""
import itertools
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle import HostPool
from paper_2406_03243_amd import harness
from paper_2406_03243_amd import workloads as wl

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2406_03243_amd import llmig, migrate
    from paper_2406_03243_amd.llmig import LlmigError, Pool

NHD, HND, HCNX, HDN = oracle.NHD, oracle.HND, oracle.HCNX, oracle.HDN
LAYOUTS = (NHD, HND, HCNX, HDN)
NAMES = oracle.LAYOUT_NAMES

# Eight (source K, source V) -> (destination K, destination V) choices whose
# K and V sides together cover all 16 (source, destination) layout pairs.
_PAIRS = list(itertools.product(LAYOUTS, LAYOUTS))
LAYOUT_CALLS = [((_PAIRS[2 * j][0], _PAIRS[2 * j + 1][0]), (_PAIRS[2 * j][1], _PAIRS[2 * j + 1][1]))
                for j in range(8)]


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def host_image(pool) -> HostPool:
    return HostPool(harness.snapshot(pool.k), harness.snapshot(pool.v), pool.block_size, pool.slot_bytes)


def make_pool(shape, seed, purpose, layouts, num_blocks=None):
    k, v = harness.alloc_layers(shape, num_blocks=num_blocks)
    total = sum(t.numel() * t.element_size() for t in k + v)
    harness.fill_bytes_from_host(k + v, wl.random_bytes(seed, purpose, total))
    return Pool(k, v, layouts=layouts)


def assert_same(gpu: HostPool, want: HostPool, what: str):
    for l in range(want.num_layers):
        for kv, (a, b) in enumerate(((gpu.k[l], want.k[l]), (gpu.v[l], want.v[l]))):
            if not np.array_equal(a, b):
                bad = np.nonzero((a != b).any(axis=1))[0]
                raise AssertionError(f"{what}: layer {l} {'KV'[kv]} differs in blocks {bad[:10].tolist()}"
                                     f" ({len(bad)} blocks)")


def lay_name(sl, dl):
    return f"K{NAMES[sl[0]]}-{NAMES[dl[0]]}_V{NAMES[sl[1]]}-{NAMES[dl[1]]}"


def run_stage(shape, sl, dl, n, seed, ids_on_device=False, nbd=None):
    src = make_pool(shape, seed, wl.SRC_VALUES, sl)
    dst = make_pool(shape, seed, wl.DST_VALUES, dl, num_blocks=nbd)
    g = wl.stream(seed, wl.EXTRA)
    ms = g.choice(shape.num_blocks, n, replace=False).astype(np.int32)
    md = g.choice(dst.num_blocks, n, replace=False).astype(np.int32)
    hs, hd = host_image(src), host_image(dst)
    if ids_on_device:
        llmig.llmig_stage(src, dst, torch.from_numpy(ms).cuda(), torch.from_numpy(md).cuda())
    else:
        llmig.llmig_stage(src, dst, ms, md)
    torch.cuda.synchronize()
    oracle.default().copy_layout(hs, sl, hd, dl, ms, md, shape.kv_heads, shape.head_dim, 2)
    assert_same(host_image(dst), hd, "destination")
    assert_same(host_image(src), hs, "source")


# (layers, blocks, block_size, heads, head_dim, dtype, pairs): head slabs of
# 1, 2, 4 and 8 chunks per lane, a ragged slab, and block sizes that are not
# powers of two.
GEOMETRIES = [
    (2, 40, 16, 4, 128, "fp16", 23),    # 4 KiB slabs (LLaMA heads)
    (2, 60, 8, 3, 64, "bf16", 31),      # 1 KiB slabs: one chunk per lane
    (1, 50, 16, 2, 64, "fp16", 17),     # 2 KiB
    (1, 30, 32, 2, 128, "bf16", 9),     # 8 KiB: eight chunks per lane
    (1, 20, 32, 2, 256, "fp16", 7),     # 16 KiB: sixteen chunks per lane (block 32, head_dim 256)
    (2, 40, 16, 3, 40, "fp16", 13),     # 80 chunks: a partial second round
    (1, 40, 24, 2, 64, "bf16", 11),     # three 8-token groups per dim
]


@pytest.mark.parametrize("geom", GEOMETRIES, ids=lambda g: f"bs{g[2]}_H{g[3]}_D{g[4]}")
def test_convert_every_layout_pair(geom):
    L, nb, bs, h, d, dt, n = geom
    shape = wl.PoolShape(L, nb, bs, h, d, dt)
    for j, (sl, dl) in enumerate(LAYOUT_CALLS):
        say("convert", geom, lay_name(sl, dl))
        run_stage(shape, sl, dl, n, seed=8100 + 7 * j + bs)


def test_convert_without_hdn_any_block_size():
    # 12-token blocks: every layout pair that does not involve HDN
    shape = wl.PoolShape(2, 40, 12, 2, 64, "fp16")
    for sl, dl in [((NHD, HND), (HCNX, NHD)), ((HCNX, HCNX), (HND, NHD)), ((HND, NHD), (NHD, HCNX))]:
        say("convert bs12", lay_name(sl, dl))
        run_stage(shape, sl, dl, 15, seed=8300)


@pytest.mark.parametrize("dev", [False, True], ids=["host_ids", "device_ids"])
def test_convert_many_pairs(dev):
    # 600 pairs: three launches of inline ids, or one of device ids
    shape = wl.PoolShape(2, 700, 16, 2, 64, "bf16")
    sl, dl = (NHD, NHD), (HCNX, HDN)
    say("convert 600 pairs", "device" if dev else "host", lay_name(sl, dl))
    run_stage(shape, sl, dl, 600, seed=8400, ids_on_device=dev, nbd=650)


def test_convert_only_v_differs():
    # K layouts agree (moved chunk for chunk), V converts
    shape = wl.PoolShape(2, 50, 16, 4, 128, "fp16")
    for sl, dl in [((NHD, NHD), (NHD, HDN)), ((HCNX, HDN), (HCNX, NHD))]:
        say("convert one side", lay_name(sl, dl))
        run_stage(shape, sl, dl, 21, seed=8500)


def test_write_tokens_every_layout():
    shape = wl.PoolShape(2, 30, 16, 3, 64, "fp16")
    seed = 8600
    for lay in [(HND, HCNX), (HDN, NHD), (HCNX, HDN)]:
        say("write tokens", NAMES[lay[0]], NAMES[lay[1]])
        pool = make_pool(shape, seed, wl.SRC_VALUES, lay)
        table = wl.stream(seed, wl.EXTRA).choice(30, 8, replace=False).astype(np.int32)
        lo, n_tok = 5, 70
        data = wl.random_bytes(seed, wl.APPEND_VALUES, 2 * 2 * n_tok * pool.slot_bytes)
        host = host_image(pool)
        llmig.llmig_write_tokens(pool, table, lo, torch.from_numpy(data).cuda())
        torch.cuda.synchronize()
        oracle.default().write_tokens_layout(host, lay, table, lo, data, 3, 64, 2)
        assert_same(host_image(pool), host, "written pool")


@pytest.mark.parametrize("layouts", [((NHD, NHD), (HCNX, HDN)), ((HCNX, HDN), (NHD, NHD))],
                         ids=["flash_to_paged", "paged_to_flash"])
def test_multistage_cross_layout(layouts):
    """A whole multi-stage migration between engines of different layouts:
    decoding appends into the source's layout between stages, every stage
    converts, and the destination ends holding every token."""
    sl, dl = layouts
    say("multistage cross-layout", lay_name(sl, dl))
    shape = wl.PoolShape(3, 300, 16, 4, 128, "bf16")
    seed = 8700 + sl[0]
    src = make_pool(shape, seed, wl.SRC_VALUES, sl)
    dst = make_pool(shape, seed, wl.DST_VALUES, dl)
    initial, counts = 1000, [37, 16, 5, 29]
    final_len = initial + sum(counts)
    nb = -(-final_len // 16)
    g = wl.stream(seed, wl.EXTRA)
    table = g.choice(300, nb, replace=False).astype(np.int32)
    free = g.permutation(300).astype(np.int32)
    appends_host = [wl.random_bytes(seed, wl.APPEND_VALUES, 3 * 2 * c * src.slot_bytes, sub=k)
                    for k, c in enumerate(counts)]
    appends = [torch.from_numpy(a).cuda() for a in appends_host]
    hs, hd = host_image(src), host_image(dst)
    mig_stream, dec_stream = harness.concurrent_streams(2)[0]
    m, _ = migrate.run_scheduled(src, dst, table, free, initial, appends, mig_stream, dec_stream)
    torch.cuda.synchronize()
    dst_table = m.commit()
    events, cur = [], initial
    for k, (length, lo, hi) in enumerate(oracle.stage_bounds(initial, counts, 16)):
        if k > 0:
            events.append(("append", cur, appends_host[k - 1]))
            cur += counts[k - 1]
        events.append(("stage", length, lo, hi))
    want_table, _ = oracle.default().migrate(hs, hd, table, free, events, layouts=(sl, dl, 4, 128, 2))
    assert np.array_equal(dst_table, want_table)
    assert_same(host_image(dst), hd, "destination")
    assert oracle.default().first_token_mismatch_layout(host_image(src), sl, table, host_image(dst), dl,
                                                         dst_table, final_len, 4, 128, 2) == -1


def test_capped_grid_converts_the_same():
    shape = wl.PoolShape(2, 200, 16, 4, 128, "fp16")
    sl, dl = (NHD, NHD), (HCNX, HDN)
    for cap in (1, 7, 64):
        say("capped conversion", cap)
        seed = 8800 + cap
        src = make_pool(shape, seed, wl.SRC_VALUES, sl)
        dst = make_pool(shape, seed, wl.DST_VALUES, dl)
        g = wl.stream(seed, wl.EXTRA)
        table = g.choice(200, 40, replace=False).astype(np.int32)
        free = g.permutation(200).astype(np.int32)
        hs, hd = host_image(src), host_image(dst)
        h = llmig.MigrationHandle(16)
        h.set_max_workgroups(cap)
        n = h.stage(src, dst, table, 640, False, free)
        torch.cuda.synchronize()
        oracle.default().copy_layout(hs, sl, hd, dl, table[:n], free[:n], 4, 128, 2)
        assert_same(host_image(dst), hd, f"cap {cap}")


def test_unsupported_conversions_are_rejected():
    say("conversion errors")

    def pools(shape, sl, dl, dtype=None):
        k, v = harness.alloc_layers(shape)
        k2, v2 = harness.alloc_layers(shape)
        if dtype is not None:
            k, v, k2, v2 = ([t.view(dtype) for t in x] for x in (k, v, k2, v2))
        return Pool(k, v, layouts=sl), Pool(k2, v2, layouts=dl)

    ids = np.array([0, 1], np.int32)
    # HDN needs block_size % 8 == 0
    a, b = pools(wl.PoolShape(1, 4, 12, 1, 64, "fp16"), (NHD, NHD), (NHD, HDN))
    with pytest.raises(LlmigError):
        llmig.llmig_stage(a, b, ids, ids)
    # slabs over 16 KiB
    a, b = pools(wl.PoolShape(1, 4, 64, 1, 256, "fp16"), (NHD, NHD), (HND, NHD))
    with pytest.raises(LlmigError):
        llmig.llmig_stage(a, b, ids, ids)
    # 1-byte elements convert nowhere (same layouts still copy)
    a, b = pools(wl.PoolShape(1, 4, 16, 1, 64, "fp16"), (NHD, NHD), (HND, NHD), dtype=torch.uint8)
    with pytest.raises(LlmigError):
        llmig.llmig_stage(a, b, ids, ids)
    a, b = pools(wl.PoolShape(1, 4, 16, 1, 64, "fp16"), (HND, NHD), (HND, NHD), dtype=torch.uint8)
    llmig.llmig_stage(a, b, ids, ids)
    # the coordinator checks before it reserves anything
    a, b = pools(wl.PoolShape(1, 4, 12, 1, 64, "fp16"), (NHD, NHD), (HDN, NHD))
    h = llmig.MigrationHandle(12)
    with pytest.raises(LlmigError):
        h.stage(a, b, np.array([0], np.int32), 12, False, np.array([1, 2], np.int32))
    assert h.info()["reserved_blocks"] == 0
    # decode attention reads NHD pools only
    a, _ = pools(wl.PoolShape(1, 4, 16, 2, 64, "fp16"), (HCNX, HDN), (NHD, NHD))
    q = torch.zeros((1, 1, 2, 64), dtype=torch.float16, device="cuda")
    out = torch.zeros(q.shape, dtype=torch.float32, device="cuda")
    ws = torch.zeros(1 << 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(LlmigError):
        llmig.llmig_decode_attention(a, q, torch.zeros((1, 1), dtype=torch.int32, device="cuda"), [10], 1.0,
                                     ws, out)
    torch.cuda.synchronize()


@pytest.mark.parametrize("where", ["device", "pinned"])
def test_unpack_converts_between_layouts(where):
    """Block fusion across engines: pack from a pool of one layout, unpack
    into a pool of another, converting on the way in."""
    shape = wl.PoolShape(2, 60, 16, 4, 128, "bf16")
    for j, (sl, dl) in enumerate([((NHD, NHD), (HCNX, HDN)), ((HCNX, HDN), (NHD, HND)), ((HND, NHD), (HND, HDN))]):
        say("unpack convert", where, lay_name(sl, dl))
        seed = 8900 + j
        src = make_pool(shape, seed, wl.SRC_VALUES, sl)
        dst = make_pool(shape, seed, wl.DST_VALUES, dl)
        g = wl.stream(seed, wl.EXTRA)
        n = 37
        ms = g.choice(60, n, replace=False).astype(np.int32)
        md = g.choice(60, n, replace=False).astype(np.int32)
        nbytes = n * 2 * 2 * src.tile_bytes
        if where == "device":
            staging = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        else:
            staging = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
        hs, hd = host_image(src), host_image(dst)
        llmig.llmig_pack(src, ms, staging)
        llmig.llmig_unpack_layout(dst, torch.from_numpy(md).cuda() if j == 1 else md, staging, sl)
        torch.cuda.synchronize()
        want = oracle.default().pack(hs, ms)
        oracle.default().unpack_layout(hd, dl, md, want, sl, 4, 128, 2)
        assert_same(host_image(dst), hd, "destination")


def test_unpack_layout_errors_and_plain_case():
    say("unpack convert errors")
    shape = wl.PoolShape(1, 8, 12, 1, 64, "fp16")
    k, v = harness.alloc_layers(shape)
    pool = Pool(k, v, layouts=(NHD, NHD))
    staging = torch.zeros(2 * 2 * pool.tile_bytes, dtype=torch.uint8, device="cuda")
    ids = np.array([0, 1], np.int32)
    with pytest.raises(LlmigError):                     # HDN with 12-token blocks
        llmig.llmig_unpack_layout(pool, ids, staging, (HDN, NHD))
    with pytest.raises(LlmigError):                     # no such layout
        llmig.llmig_unpack_layout(pool, ids, staging, (NHD, 7))
    with pytest.raises(LlmigError):                     # staging too small
        llmig.llmig_unpack_layout(pool, ids, staging[:100], (HND, NHD))
    with pytest.raises(LlmigError):                     # repeated destination
        llmig.llmig_unpack_layout(pool, np.array([1, 1], np.int32), staging, (HND, NHD))
    # equal layouts: the plain unpack, bytes as they are
    data = wl.random_bytes(9000, wl.EXTRA, staging.numel())
    staging.copy_(torch.from_numpy(data))
    llmig.llmig_unpack_layout(pool, ids, staging, (NHD, NHD))
    torch.cuda.synchronize()
    got = host_image(pool)
    t = pool.tile_bytes
    assert np.array_equal(got.k[0][0], data[:t]) and np.array_equal(got.k[0][1], data[t:2 * t])
    assert np.array_equal(got.v[0][0], data[2 * t:3 * t]) and np.array_equal(got.v[0][1], data[3 * t:])


def test_convert_pools_past_16_bit_ids():
    # 70000-block pools: ids past 65535 travel as 32-bit words, 256 pairs a launch
    shape = wl.PoolShape(2, 70000, 8, 2, 8, "fp16")
    sl, dl = (NHD, HCNX), (HDN, NHD)
    say("convert, 70000-block pools", lay_name(sl, dl))
    run_stage(shape, sl, dl, 300, seed=9300, nbd=66000)
