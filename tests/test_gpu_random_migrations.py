"""Randomised whole migrations on the GPU against the oracle's replay: for
120 seeded cases, a random pool geometry (layers, block size, heads, head
dim, 16-bit type), random K/V layouts on each side where a conversion is
supported, a random initial length, up to five batches of appended tokens
written by the decode stand-in between stages, and sometimes a capped copy
grid.  Source and destination must equal the replay byte for byte, and every
token must be found at its destination slot."""
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
    from paper_2406_03243_amd.llmig import Pool

NHD, HND, HCNX, HDN = 0, 1, 2, 3


def host_image(pool) -> HostPool:
    return HostPool(harness.snapshot(pool.k), harness.snapshot(pool.v), pool.block_size, pool.slot_bytes)


def draw_case(seed):
    g = wl.stream(seed, wl.EXTRA)
    layers = int(g.integers(1, 5))
    bs = int(g.choice([1, 2, 4, 8, 16, 32]))
    heads = int(g.integers(1, 9))
    dim = int(g.choice([8, 16, 64, 72, 128]))
    dtype = str(g.choice(["fp16", "bf16"]))
    layouts = [(NHD, NHD), (NHD, NHD)]
    if g.random() < 0.5:                       # a cross-layout migration, where supported
        allowed = [NHD, HND, HCNX] + ([HDN] if bs % 8 == 0 else [])
        if bs * dim * 2 <= 16384:
            layouts = [tuple(int(x) for x in g.choice(allowed, 2)) for _ in range(2)]
    initial = int(g.integers(0, 40 * bs + 1))
    counts = [int(x) for x in g.integers(0, 3 * bs + 2, int(g.integers(0, 6)))]
    cap = int(g.choice([0, 0, 1, 3, 50]))
    return layers, bs, heads, dim, dtype, layouts, initial, counts, cap


@pytest.mark.parametrize("seed", range(120))
def test_random_migration(seed):
    layers, bs, heads, dim, dtype, (sl, dl), initial, counts, cap = draw_case(10_000 + seed)
    print("[case] random migration", seed, dict(layers=layers, bs=bs, heads=heads, dim=dim, dtype=dtype,
                                                  src=sl, dst=dl, initial=initial, counts=counts, cap=cap),
          flush=True)
    sys.stdout.flush()
    final_len = initial + sum(counts)
    nb = -(-final_len // bs)
    nbs, nbd = nb + 20, nb + 30
    shape_s = wl.PoolShape(layers, nbs, bs, heads, dim, dtype)
    shape_d = wl.PoolShape(layers, nbd, bs, heads, dim, dtype)
    sk, sv = harness.alloc_layers(shape_s)
    dk, dv = harness.alloc_layers(shape_d)
    harness.fill_bytes_from_host(sk + sv, wl.random_bytes(seed, wl.SRC_VALUES,
                                                          sum(t.numel() * 2 for t in sk + sv)))
    harness.fill_bytes_from_host(dk + dv, wl.random_bytes(seed, wl.DST_VALUES,
                                                          sum(t.numel() * 2 for t in dk + dv)))
    src, dst = Pool(sk, sv, layouts=sl), Pool(dk, dv, layouts=dl)
    g = wl.stream(seed, wl.SRC_LAYOUT)
    table = g.choice(nbs, nb, replace=False).astype(np.int32)
    free = g.permutation(nbd).astype(np.int32)
    appends_host = [wl.random_bytes(seed, wl.APPEND_VALUES, layers * 2 * c * src.slot_bytes, sub=k)
                    for k, c in enumerate(counts)]
    hs, hd = host_image(src), host_image(dst)
    before = [t.clone() for t in dk + dv] if cap else None
    mig, dec = torch.cuda.Stream(), torch.cuda.Stream()
    m, _ = migrate.run_scheduled(src, dst, table, free, initial,
                                 [torch.from_numpy(a).cuda() for a in appends_host], mig, dec)
    torch.cuda.synchronize()
    events, cur = [], initial
    for k, (length, lo, hi) in enumerate(oracle.stage_bounds(initial, counts, bs)):
        if k > 0:
            events.append(("append", cur, appends_host[k - 1]))
            cur += counts[k - 1]
        events.append(("stage", length, lo, hi))
    same = sl == (NHD, NHD) and dl == (NHD, NHD)
    lay = None if same else (sl, dl, heads, dim, 2)
    want_table, _ = oracle.default().migrate(hs, hd, table, free, events, layouts=lay)
    assert np.array_equal(np.asarray(m.dst_table, np.int32), want_table)
    gs, gd = host_image(src), host_image(dst)
    assert gs.equals(hs), "source differs from the replay"
    assert gd.equals(hd), "destination differs from the replay"
    assert oracle.default().first_token_mismatch_layout(gs, sl, table, gd, dl, want_table, final_len,
                                                        heads, dim, 2) == -1
    if cap:
        # The request again, from the final source into the untouched
        # destination, with the copy grid capped: the same blocks in the same
        # places (non-final stages never see a block that is written later,
        # and the final stage copies the partial block after every append).
        dst2 = Pool(before[:layers], before[layers:], layouts=dl)
        m2 = migrate.Migration(src, dst2, table, free, mig, max_workgroups=cap)
        m2.stage(final_len, final=False)
        m2.stage(final_len, final=True)
        torch.cuda.synchronize()
        assert np.array_equal(np.asarray(m2.dst_table, np.int32), want_table)
        assert host_image(dst2).equals(gd), "capped grid differs"


@pytest.mark.parametrize("seed", range(60))
def test_random_block_fusion(seed):
    """Block fusion (§5) on random cases: pack a random list of source blocks
    (repeats allowed) into device or pinned staging, unpack it into distinct
    destination blocks, converting between layouts where they differ; ids
    from the host or the device."""
    g = wl.stream(20_000 + seed, wl.EXTRA)
    layers, bs, heads, dim, dtype, (sl, dl), _, _, _ = draw_case(20_000 + seed)
    n = int(g.integers(1, 80))
    nbs, nbd = int(g.integers(1, 100)), n + int(g.integers(0, 40))
    where = str(g.choice(["device", "pinned"]))
    dev_ids = bool(g.random() < 0.5)
    print("[case] random fusion", seed, dict(layers=layers, bs=bs, heads=heads, dim=dim, src=sl, dst=dl, n=n,
                                               staging=where, device_ids=dev_ids), flush=True)
    sk, sv = harness.alloc_layers(wl.PoolShape(layers, nbs, bs, heads, dim, dtype))
    dk, dv = harness.alloc_layers(wl.PoolShape(layers, nbd, bs, heads, dim, dtype))
    harness.fill_bytes_from_host(sk + sv, wl.random_bytes(seed, wl.SRC_VALUES, sum(t.numel() * 2 for t in sk + sv)))
    harness.fill_bytes_from_host(dk + dv, wl.random_bytes(seed, wl.DST_VALUES, sum(t.numel() * 2 for t in dk + dv)))
    src, dst = Pool(sk, sv, layouts=sl), Pool(dk, dv, layouts=dl)
    blocks = g.integers(0, nbs, n).astype(np.int32)            # repeats allowed when packing
    into = g.permutation(nbd)[:n].astype(np.int32)
    nbytes = n * layers * 2 * src.tile_bytes
    if where == "device":
        staging = torch.empty(nbytes + 48, dtype=torch.uint8, device="cuda")
    else:
        staging = torch.empty(nbytes + 48, dtype=torch.uint8, pin_memory=True)
    staging.fill_(0x5C)
    torch.cuda.synchronize()
    hs, hd = host_image(src), host_image(dst)
    ids_b = torch.from_numpy(blocks).cuda() if dev_ids else blocks
    ids_i = torch.from_numpy(into).cuda() if dev_ids else into
    llmig.llmig_pack(src, ids_b, staging)
    torch.cuda.synchronize()
    got = staging.cpu().numpy()
    want = oracle.default().pack(hs, blocks)
    assert np.array_equal(got[:nbytes], want)
    assert (got[nbytes:] == 0x5C).all()
    if sl == dl:
        llmig.llmig_unpack(dst, ids_i, staging)
        oracle.default().unpack(hd, into, want)
    else:
        llmig.llmig_unpack_layout(dst, ids_i, staging, sl)
        oracle.default().unpack_layout(hd, dl, into, want, sl, heads, dim, 2)
    torch.cuda.synchronize()
    assert host_image(dst).equals(hd), "destination differs from the oracle"
    assert host_image(src).equals(hs), "source changed"
