"""GPU parity of llmig_decode_attention_migrate: a decode-attention pass
that also carries a migration stage of one of its sequences (Llumnix §4.2
stage copy, as a side effect of decode's reads of the same KV).

Every case checks, through the C ABI, against the oracle:
  * the attention output, to the error bound of tests/attn_cases.py, and
    that it is the output of the plain llmig_decode_attention call;
  * the destination pool, byte for byte over every block: the stage's
    blocks hold what the oracle's tile copy of the same pairs writes and
    every other block keeps its bytes (a stage ending in the sequence's
    partly filled last block writes that block's token rows only: its
    slots past the length keep the destination's bytes);
  * the source pool, unchanged.
Cases cover head dims 64 and 128, block sizes 1-32, grouped and ungrouped
heads, stages that start inside a partition and end inside another,
sequences of several 2048-token partitions, a call split over two launches
with the migrating sequence in both, and seeded random shapes."""
import sys

import numpy as np
import pytest
import torch

import attn_cases as ac
from oracle import HostPool
from paper_2406_03243_amd import harness
from paper_2406_03243_amd import workloads as wl

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2406_03243_amd.llmig import (LlmigError, Pool, decode_workspace_bytes, llmig_decode_attention,
                                            llmig_decode_attention_migrate)


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def to_device(shape: wl.PoolShape, host: HostPool):
    k, v = harness.alloc_layers(shape)
    for t, a in zip(k + v, host.k + host.v):
        harness.tile_view(t).copy_(torch.from_numpy(a))
    return Pool(k, v)


def host_image(pool) -> HostPool:
    return HostPool(harness.snapshot(pool.k), harness.snapshot(pool.v), pool.block_size, pool.slot_bytes)


def dst_host(shape: wl.PoolShape, seed: int) -> HostPool:
    tile = shape.block_size * shape.kv_heads * shape.head_dim * 2
    draw = [wl.values16(seed, wl.DST_VALUES, shape.num_blocks * tile // 2, shape.dtype, sub=i).view(np.uint8)
            .reshape(shape.num_blocks, tile) for i in range(2 * shape.num_layers)]
    return HostPool(draw[:shape.num_layers], draw[shape.num_layers:], shape.block_size,
                    shape.kv_heads * shape.head_dim * 2)


def same_pool(got: HostPool, want: HostPool, what: str):
    for l in range(want.num_layers):
        for kv, (g, w) in enumerate(((got.k[l], want.k[l]), (got.v[l], want.v[l]))):
            if not np.array_equal(g, w):
                bad = np.argwhere((g != w).any(axis=1))[:, 0]
                raise AssertionError(f"{what}: layer {l} {'KV'[kv]} blocks {bad[:8].tolist()} differ")


def keep_tail(want: HostPool, before: HostPool, ids, to_block: int, length: int, bs: int):
    """In the expected destination, give back the pre-stage bytes of the
    slots past `length` in the stage's last block when that block is the
    sequence's partly filled last one (no token lives there)."""
    filled = length - (to_block - 1) * bs
    if len(ids) == 0 or filled >= bs:
        return
    d, lo = int(ids[-1]), filled * want.slot_bytes
    for a, b in zip(want.k + want.v, before.k + before.v):
        a[d, lo:] = b[d, lo:]


def run_case(case, seq, from_block, to_block, seed, extra_dst_blocks=7):
    num_layers, num_blocks, bs, kv_heads, head_dim, group, ctx, dtype, _ = case
    host, qbits, tables, ctx, scale = ac.case_inputs(case, seed)
    shape = wl.PoolShape(num_layers, num_blocks, bs, kv_heads, head_dim, dtype)
    dshape = wl.PoolShape(num_layers, num_blocks + extra_dst_blocks, bs, kv_heads, head_dim, dtype)
    hd = dst_host(dshape, seed)
    src, dst = to_device(shape, host), to_device(dshape, hd)
    g = wl.stream(seed, wl.EXTRA, 7)
    ids = g.permutation(dshape.num_blocks)[:to_block - from_block].astype(np.int32)
    dst_ids = torch.from_numpy(ids).cuda()
    tdt = harness.TORCH_DTYPE[dtype]
    q = torch.from_numpy(qbits.view(np.int16)).view(tdt).cuda()
    tab = torch.from_numpy(tables).cuda()
    out = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    plain = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(16, decode_workspace_bytes(ctx, num_layers, q.shape[2], head_dim)), dtype=torch.uint8,
                     device="cuda")
    llmig_decode_attention_migrate(src, q, tab, ctx, scale, ws, out, dst, seq, dst_ids, from_block)
    torch.cuda.synchronize()
    llmig_decode_attention(src, q, tab, ctx, scale, ws, plain)
    torch.cuda.synchronize()
    orc = ac.default_oracle()
    want = orc.decode_attention(host, kv_heads, head_dim, dtype, qbits, tables, ctx, scale)
    tol = ac.tolerance(orc, host, kv_heads, head_dim, dtype, qbits, tables, ctx, scale)
    got = out.cpu().numpy().astype(np.float64)
    ratio = ac.excess(got, want, tol)
    identical = torch.equal(out, plain)
    say(f"max error / bound {ratio.max():.3g}; output identical to the plain call: {identical}")
    assert not (~(ratio <= 1.0)).any(), f"bound ratio {np.nanmax(ratio):.3g}"
    assert identical, "the carried stage changed the attention output"
    before = hd.copy()
    orc.copy(host, hd, tables[seq, from_block:to_block], ids)
    keep_tail(hd, before, ids, to_block, ctx[seq], bs)
    same_pool(host_image(dst), hd, "destination")
    same_pool(host_image(src), host, "source")


# (attention case, migrating sequence, first block, end block)
CASES = [
    (ac.CASES[0], 2, 0, 37),          # 600 tokens: all 37 full blocks, D 128, 8 heads a group
    (ac.CASES[1], 0, 5, 32),          # starts inside the partition, D 64
    (ac.CASES[2], 0, 0, 256),         # two partitions of 2048
    (ac.CASES[2], 0, 100, 200),       # a range across the partition boundary
    (ac.CASES[3], 1, 3, 11),          # 8-token blocks, 4 sequences
    (ac.CASES[5], 1, 100, 7500),      # 133 items, two launches: sequence 1 spans both
    (ac.CASES[7], 2, 0, 15),          # 4-token blocks
    (ac.CASES[9], 1, 0, 625),         # 32-token blocks, ten partitions
    (ac.CASES[6], 0, 42, 43),         # the last whole block of 700 tokens, 16 query heads on one KV head
    (ac.CASES[0], 2, 30, 38),         # ends in the partly filled last block (600 tokens: 8 in block 37)
    (ac.CASES[3], 1, 0, 12),          # 95 tokens in 8-token blocks: the whole request, last block 7/8 full
    (ac.CASES[7], 2, 10, 16),         # 62 tokens in 4-token blocks: the last block half full
    (ac.CASES[5], 2, 1000, 1250),     # 20000 tokens, a sequence spanning both launches, last block full
    ((1, 2100, 1, 2, 64, 4, [2050, 7], "fp16", False), 0, 1000, 2050),   # 1-token blocks across a partition edge
    ((2, 200, 32, 2, 128, 8, [1000, 70], "bf16", False), 0, 20, 32),     # 32-token blocks, last one 8/32 full
]


def case_id(c):
    return f"{ac.case_id(c[0])}_seq{c[1]}_blocks{c[2]}-{c[3]}"


@pytest.mark.parametrize("c", CASES, ids=case_id)
def test_attention_carries_stage(c):
    case, seq, lo, hi = c
    say("attention + stage", case_id(c))
    run_case(case, seq, lo, hi, ac.case_seed(case))


@pytest.mark.parametrize("seed", range(12))
def test_attention_carries_stage_random(seed):
    """Seeded random shapes (block sizes 1-32, head dims 64/128, groups,
    batches, lengths) with a random sequence and block range."""
    case = ac.random_case(40_000 + seed)
    ctx = case[6]
    g = wl.stream(40_000 + seed, wl.LENGTHS, 1)
    full = [-(-n // case[2]) for n in ctx]       # blocks holding tokens, the last one perhaps partly
    seq = int(np.argmax(full)) if g.random() < 0.5 else int(g.integers(0, len(ctx)))
    lo = int(g.integers(0, full[seq] + 1))
    hi = int(g.integers(lo, full[seq] + 1))
    say("attention + stage random", seed, case, seq, lo, hi)
    run_case(case, seq, lo, hi, 40_000 + seed)


def test_attention_stage_skips_ids_outside_the_pool():
    """Device destination ids are the caller's guarantee and are not read on
    the host; an id past the destination pool or a negative one must still
    not be written anywhere: the other blocks of the stage are copied and
    every other destination block keeps its bytes."""
    case = ac.CASES[1]
    num_layers, num_blocks, bs, kv_heads, head_dim, group, _, dtype, _ = case
    host, qbits, tables, ctx, scale = ac.case_inputs(case, ac.case_seed(case))
    shape = wl.PoolShape(num_layers, num_blocks, bs, kv_heads, head_dim, dtype)
    say("attention + stage, ids outside the pool", shape)
    hd = dst_host(shape, 77)
    src, dst = to_device(shape, host), to_device(shape, hd)
    lo, hi = 2, 30
    ids = wl.stream(77, wl.EXTRA, 7).permutation(num_blocks)[:hi - lo].astype(np.int32)
    ids[1], ids[3] = num_blocks + 5, -3
    q = torch.from_numpy(qbits.view(np.int16)).view(harness.TORCH_DTYPE[dtype]).cuda()
    tab = torch.from_numpy(tables).cuda()
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    ws = torch.empty(decode_workspace_bytes(ctx, num_layers, q.shape[2], head_dim), dtype=torch.uint8, device="cuda")
    llmig_decode_attention_migrate(src, q, tab, ctx, scale, ws, out, dst, 0, torch.from_numpy(ids).cuda(), lo)
    torch.cuda.synchronize()
    keep = np.array([k for k in range(hi - lo) if k not in (1, 3)])
    ac.default_oracle().copy(host, hd, tables[0, lo:hi][keep], ids[keep])
    same_pool(host_image(dst), hd, "destination")


def test_attention_stage_rejects_bad_arguments():
    """Argument errors are refused before anything is enqueued: the
    destination pool keeps every byte."""
    say("attention + stage errors")
    shape = wl.PoolShape(1, 40, 16, 2, 64, "fp16")
    host = dst_host(shape, 5)
    src = to_device(shape, host)
    hd = dst_host(wl.PoolShape(1, 40, 16, 2, 64, "fp16"), 6)
    dst = to_device(shape, hd)
    q = torch.zeros((1, 1, 4, 64), dtype=torch.float16, device="cuda")
    tab = torch.arange(4, dtype=torch.int32, device="cuda").view(1, 4)
    out = torch.zeros(q.shape, dtype=torch.float32, device="cuda")
    ws = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    ids = torch.arange(10, 15, dtype=torch.int32, device="cuda")
    bad = [
        dict(seq=1, from_block=0, dst_ids=ids[:2]),             # no sequence 1
        dict(seq=-1, from_block=0, dst_ids=ids[:2]),
        dict(seq=0, from_block=0, dst_ids=ids[:5]),             # 5 blocks: a 50-token sequence holds 4
        dict(seq=0, from_block=-1, dst_ids=ids[:2]),
    ]
    for kw in bad:
        with pytest.raises(LlmigError):
            llmig_decode_attention_migrate(src, q, tab, [50], 1.0, ws, out, dst, **kw)
    # destination ids that are not 4-byte aligned, through the C ABI itself
    from paper_2406_03243_amd import llmig as L
    c = L._host_i32([50])
    rc = L._lib.llmig_decode_attention_migrate(src.handle, 0, q.data_ptr(), 1, 4, tab.data_ptr(), 4, c.ctypes.data,
                                               1.0, ws.data_ptr(), ws.numel(), out.data_ptr(), dst.handle, 0,
                                               ids.data_ptr() + 2, 0, 2, None)
    assert rc == -1, rc
    with pytest.raises(LlmigError):                             # the source pool itself
        llmig_decode_attention_migrate(src, q, tab, [50], 1.0, ws, out, src, 0, ids[:2], 0)
    hk, hv = harness.alloc_layers(wl.PoolShape(1, 40, 16, 2, 128, "fp16"))
    with pytest.raises(LlmigError):                             # other geometry
        llmig_decode_attention_migrate(src, q, tab, [50], 1.0, ws, out, Pool(hk, hv), 0, ids[:2], 0)
    big_k, big_v = harness.alloc_layers(wl.PoolShape(1, 1 << 19, 16, 2, 64, "fp16"))   # 2^31-byte layer tensors
    with pytest.raises(LlmigError):                             # beyond the stores' 32-bit offsets
        llmig_decode_attention_migrate(src, q, tab, [50], 1.0, ws, out, Pool(big_k, big_v), 0, ids[:2], 0)
    del big_k, big_v
    torch.cuda.synchronize()
    same_pool(host_image(dst), hd, "destination after refused calls")
    # an empty stage is the plain call
    llmig_decode_attention_migrate(src, q, tab, [50], 1.0, ws, out, dst, 0, ids[:0], 2)
    plain = torch.zeros_like(out)
    llmig_decode_attention(src, q, tab, [50], 1.0, ws, plain)
    torch.cuda.synchronize()
    assert torch.equal(out, plain)
    same_pool(host_image(dst), hd, "destination after an empty stage")



@pytest.mark.parametrize("split,carry_final", [(1, False), (3, False), (1, True), (2, True)])
def test_migration_carried_by_decode_steps(split, carry_final):
    """A whole migration whose first stage rides on `split` decode steps of a
    batch the request belongs to (migrate.run_carried): each step writes its
    share of the request's whole blocks into the destination and produces
    one token of the request; the final stage then copies the rest, as a
    stage of its own after the drain or, with carry_final, carried by the
    request's last decode step.  The recorded schedule, replayed by the
    oracle, gives the destination byte for byte (a carried final stage
    leaves the slots past the length in the last block as they were), and
    every token of the request reads the same in both pools."""
    import oracle
    from paper_2406_03243_amd import migrate
    shape = wl.PoolShape(2, 600, 16, 4, 128, "bf16")
    seed = 8080 + split
    say("migration carried by decode steps", split, carry_final, shape)
    host = dst_host(shape, seed + 1)
    src = to_device(shape, host)
    hd = dst_host(shape, seed)
    dst = to_device(shape, hd)
    g = wl.stream(seed, wl.EXTRA, 3)
    perm = g.permutation(shape.num_blocks).astype(np.int32)
    table, others = perm[:80], perm[80:]
    initial = 79 * 16 + 5                       # 79 whole blocks and 5 tokens of the 80th
    n_other, per = 3, 120
    stride = max(per, len(table))
    tabs = np.zeros((n_other + 1, stride), np.int32)
    for k in range(n_other):
        tabs[k, :per] = others[k * per:(k + 1) * per]
    tabs[n_other, :len(table)] = table
    ctx = [per * 16 - 7 * k for k in range(n_other)] + [initial]
    q_heads = 16
    qbits = wl.values16(seed, wl.APPEND_VALUES, shape.num_layers * len(ctx) * q_heads * shape.head_dim, "bf16", sub=9)
    q = torch.from_numpy(qbits.view(np.int16)).view(torch.bfloat16).reshape(shape.num_layers, len(ctx), q_heads,
                                                                             shape.head_dim).cuda()
    tab = torch.from_numpy(tabs).cuda()
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    ws = torch.empty(decode_workspace_bytes([c + split for c in ctx], shape.num_layers, q_heads, shape.head_dim),
                     dtype=torch.uint8, device="cuda")
    append = wl.values16(seed, wl.APPEND_VALUES, shape.num_layers * 2 * split * src.slot_bytes // 2, "bf16", sub=4)
    append = append.view(np.uint8).reshape(shape.num_layers, 2, split, src.slot_bytes)
    (attn, mig, dec), _ = harness.concurrent_streams(3)
    lengths = list(ctx)

    def step(carry):
        pool, ids, first = carry
        llmig_decode_attention_migrate(src, q, tab, lengths, 0.125, ws, out, pool, n_other, ids, first, stream=attn)
        lengths[n_other] += 1                   # the request's context grows by the step's token

    free = np.ascontiguousarray(g.permutation(shape.num_blocks).astype(np.int32))
    m, downtime, _ = migrate.run_carried(src, dst, table, initial, free, step, torch.from_numpy(append).cuda(),
                                         attn, mig, dec, split=split, carry_final=carry_final)
    torch.cuda.synchronize()
    assert [r.from_tok for r in m.stages] == [0, 79 * 16] and m.stages[0].to_tok == 79 * 16
    assert m.stages[-1].final and m.stages[-1].to_tok == initial + split
    assert downtime == 0.0 if carry_final else downtime > 0
    events = [("stage", initial, 0, 79 * 16), ("append", initial, np.ascontiguousarray(append)),
              ("stage", initial + split, 79 * 16, initial + split)]
    hs, before = host.copy(), hd.copy()
    dst_table, _ = oracle.default().migrate(hs, hd, table, free, events)
    assert np.array_equal(dst_table, m.commit())
    if carry_final:
        keep_tail(hd, before, dst_table, len(dst_table), initial + split, 16)
    gs, gd = host_image(src), host_image(dst)
    same_pool(gs, hs, "source (with the appended tokens)")
    same_pool(gd, hd, "destination")
    assert oracle.default().first_token_mismatch(gs, table, gd, dst_table, initial + split) == -1
