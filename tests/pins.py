"""Pins: checks that tie the CPU oracle to what the paper and plain
mathematics fix, independent of the oracle's own formulation.

Each ``pin_*`` takes an :class:`oracle.Oracle` and raises AssertionError when
the oracle breaks what it pins.  ``tests/test_oracle_pins.py`` runs them on
the oracle; ``tests/test_oracle_mutants.py`` runs them on copies of the
oracle with one plausible mistake planted each, and requires every copy to
fail at least one pin.

What pins what:
  * planner  - closed form n = ceil(to/bs) - from/bs with the table slice and
               the free-list prefix; partition of a sequence of stages; the
               paper's worked example (1k tokens -> 4k tiles over 32 layers,
               Llumnix §5 "Block fusion"); error classes and no partial
               output on error;
  * geometry - 128 KB tiles for 16-bit LLaMA-7B (Llumnix §5) and 3.2 GB for
               a 4k-token LLaMA-2-13B request (Llumnix §2), loosely;
  * copy     - torch advanced indexing on a [layer, K/V, block, byte] tensor;
               contiguous id ranges reduce to one contiguous byte copy; blocks
               outside the mapping and the source stay untouched;
  * pack     - torch.index_select + stack; unpack(pack(x)) round trip;
  * appends  - numpy indexing of the [num_blocks, block_size, slot] view;
  * identity - planted single-byte differences are found at their token;
  * stages   - a whole multi-stage replay ends with every token identical,
               ceil(len/bs) blocks, stages partitioning the block set;
  * 16-bit   - fp16 and bf16 decoding against numpy/torch for all 65536
               bit patterns;
  * decode attention - dense torch float64 softmax attention over the
               gathered sequence; one token gives its V row; zero scale
               gives the mean of V; grouped heads read their own KV head;
               moving the tokens between blocks leaves the output unchanged.
  * layouts  - every layout's placement equals numpy's reshape/transpose of
               the [block_size, heads, head_dim] tile, for 1-, 2- and 4-byte
               elements; offsets are a bijection onto the tile; conversions
               round-trip and compose; same-layout conversion is the byte
               copy; appends and token identity read through numpy's view;
               a cross-layout multi-stage replay keeps every token; a
               converting unpack equals the plain unpack for equal layouts,
               the converting stage copy after a pack, and numpy's view.
"""
from __future__ import annotations

import json
import os

import numpy as np
import torch

from oracle import EINVAL, ENOSPC, ERANGE, HCNX, HDN, HND, NHD, OK, HostPool, stage_bounds

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "paper_worked_examples.json")


def _ceil_div(a, b):
    return -(-a // b)


def _random_pool(rng, num_layers, num_blocks, block_size, slot_bytes):
    t = block_size * slot_bytes
    return HostPool([rng.integers(0, 256, (num_blocks, t), dtype=np.uint8) for _ in range(num_layers)],
                    [rng.integers(0, 256, (num_blocks, t), dtype=np.uint8) for _ in range(num_layers)],
                    block_size, slot_bytes)


def _as_tensor(pool: HostPool) -> torch.Tensor:
    """[layer, K/V, block, byte] uint8 tensor of a host pool."""
    return torch.stack([torch.stack([torch.from_numpy(k), torch.from_numpy(v)])
                        for k, v in zip(pool.k, pool.v)])


# --------------------------------------------------------------------------- planner
def pin_plan_closed_form(orc):
    rng = np.random.default_rng(7)
    for bs, max_len in ((1, 24), (2, 30), (3, 33), (4, 40), (16, 70)):
        for length in range(0, max_len + 1):
            nb = _ceil_div(length, bs)
            ids = rng.permutation(500).astype(np.int32)
            table = ids[:nb + 2]
            free = ids[nb + 2:nb + 2 + nb + 3]
            for lo in range(0, length + 1, bs):
                for hi in range(lo, length + 1):
                    if hi % bs and hi != length:
                        continue
                    code, ms, md = orc.plan(table, free, length, lo, hi, bs)
                    n = _ceil_div(hi, bs) - lo // bs
                    assert code == OK, (bs, length, lo, hi, code)
                    assert np.array_equal(ms, table[lo // bs:lo // bs + n]), (bs, length, lo, hi)
                    assert np.array_equal(md, free[:n]), (bs, length, lo, hi)


def pin_plan_partition(orc):
    """Stages with whole-block interior boundaries partition the request's
    blocks: concatenated in order they give the table prefix, and the
    destinations the free-list prefix."""
    rng = np.random.default_rng(11)
    for _ in range(300):
        bs = int(rng.choice([1, 2, 4, 16]))
        length = int(rng.integers(1, 400))
        nb = _ceil_div(length, bs)
        ids = rng.permutation(4000).astype(np.int32)
        table, free = ids[:nb], ids[nb:2 * nb + 5]
        inner = sorted(set(int(x) * bs for x in rng.integers(0, length // bs + 1, rng.integers(0, 6))))
        bounds = [0] + [b for b in inner if 0 < b < length] + [length]
        got_s, got_d, left = [], [], free
        for lo, hi in zip(bounds[:-1], bounds[1:]):
            code, ms, md = orc.plan(table, left, length, lo, hi, bs)
            assert code == OK
            got_s.append(ms)
            got_d.append(md)
            left = left[len(md):]
        s, d = np.concatenate(got_s), np.concatenate(got_d)
        assert len(s) == nb and np.array_equal(s, table)
        assert np.array_equal(d, free[:nb])
        assert len(set(s.tolist())) == nb


def pin_plan_errors(orc):
    table = np.arange(100, 120, dtype=np.int32)      # 20 blocks
    free = np.arange(500, 520, dtype=np.int32)
    cases = [
        ((table, free, 200, 8, 32, 16), EINVAL),        # from not on a block boundary
        ((table, free, 200, 16, 40, 16), EINVAL),       # to not on a boundary and not len
        ((table, free, 200, 0, 201, 16), EINVAL),       # to beyond len
        ((table, free, 200, 48, 32, 16), EINVAL),       # from > to
        ((table, free, -1, 0, 0, 16), EINVAL),          # negative length
        ((table, free, 200, 0, 200, 0), EINVAL),        # block size 0
        ((table[:12], free, 200, 0, 192, 16), EINVAL),  # table misses block 12 of len 200
        ((table, free[:12], 200, 0, 200, 16), ENOSPC),  # 13 blocks needed, 12 free
        ((table, free[:0], 200, 0, 16, 16), ENOSPC),
    ]
    for args, want in cases:
        code, out_s, out_d, n = orc.plan(*args, sentinel=-9)
        assert code == want, (args[2:], code, want)
        assert n == 0 and (out_s == -9).all() and (out_d == -9).all(), args[2:]
    # exact fit is not ENOSPC
    code, ms, md = orc.plan(table, free[:13], 200, 0, 200, 16)
    assert code == OK and len(md) == 13
    # output capacity one short of the stage
    code, _, _, n = orc.plan(table, free, 200, 0, 200, 16, out_cap=12, sentinel=-9)
    assert code == EINVAL and n == 0
    code, ms, _ = orc.plan(table, free, 200, 0, 200, 16, out_cap=13)
    assert code == OK and len(ms) == 13
    # negative ids inside the stage: ERANGE; outside the stage: fine
    bad = table.copy()
    bad[3] = -1
    assert orc.plan(bad, free, 200, 0, 64, 16)[0] == ERANGE
    assert orc.plan(bad, free, 200, 64, 200, 16)[0] == OK
    badf = free.copy()
    badf[2] = -5
    assert orc.plan(table, badf, 200, 0, 48, 16)[0] == ERANGE
    assert orc.plan(table, badf, 200, 0, 32, 16)[0] == OK
    # duplicate ids inside the stage: EINVAL; outside the stage: fine
    dup = table.copy()
    dup[5] = dup[2]
    assert orc.plan(dup, free, 200, 0, 96, 16)[0] == EINVAL
    assert orc.plan(dup, free, 200, 48, 96, 16)[0] == OK
    dupf = free.copy()
    dupf[4] = dupf[0]
    assert orc.plan(table, dupf, 200, 0, 80, 16)[0] == EINVAL
    assert orc.plan(table, dupf, 200, 0, 64, 16)[0] == OK
    # empty stages
    for lo, hi in ((0, 0), (192, 192), (64, 64)):
        code, ms, md = orc.plan(table, free, 200, lo, hi, 16)
        assert code == OK and len(ms) == 0 and len(md) == 0
    code, ms, md = orc.plan(table[:0], free, 0, 0, 0, 16)
    assert code == OK and len(ms) == 0


# --------------------------------------------------------------------------- geometry
def pin_paper_examples(orc):
    g = json.load(open(GOLDEN))
    one_k = g["one_k_tokens"]["value"]
    m = g["llama7b_tile"]["model"]
    from oracle import tile_bytes
    t7 = tile_bytes(m["block_size"], m["kv_heads"], m["head_dim"], m["elem_bytes"])
    assert t7 == g["llama7b_tile"]["tile_bytes"] == 128 * 1024
    ex = g["llama7b_1k_tokens_tiles"]
    assert ex["tokens"] == one_k
    n_blocks = 200
    code, ms, _ = orc.plan(np.arange(n_blocks, dtype=np.int32), np.arange(n_blocks, dtype=np.int32),
                           ex["tokens"], 0, ex["tokens"], m["block_size"])
    assert code == OK
    assert len(ms) * m["num_layers"] * 2 == ex["tiles"]
    e13 = g["llama2_13b_4k_tokens_kv"]
    m13 = e13["model"]
    code, ms, _ = orc.plan(np.arange(400, dtype=np.int32), np.arange(400, dtype=np.int32),
                           e13["tokens"], 0, e13["tokens"], m13["block_size"])
    assert code == OK
    kv = len(ms) * m13["num_layers"] * 2 * tile_bytes(m13["block_size"], m13["kv_heads"],
                                                         m13["head_dim"], m13["elem_bytes"])
    assert abs(kv - e13["kv_bytes_printed"]) <= e13["rel_tolerance"] * e13["kv_bytes_printed"]


# --------------------------------------------------------------------------- copy
def pin_copy_matches_indexing(orc):
    rng = np.random.default_rng(3)
    for num_layers, nb_src, nb_dst, bs, slot, n in ((3, 37, 41, 4, 48, 11), (1, 5, 5, 1, 16, 5),
                                                   (2, 64, 30, 16, 32, 30)):
        src = _random_pool(rng, num_layers, nb_src, bs, slot)
        dst = _random_pool(rng, num_layers, nb_dst, bs, slot)
        ms = rng.choice(nb_src, n, replace=False).astype(np.int32)
        md = rng.choice(nb_dst, n, replace=False).astype(np.int32)
        want = _as_tensor(dst).clone()
        want[:, :, torch.from_numpy(md).long()] = _as_tensor(src)[:, :, torch.from_numpy(ms).long()]
        src0 = src.copy()
        orc.copy(src, dst, ms, md)
        assert torch.equal(_as_tensor(dst), want)
        assert src.equals(src0)


def pin_copy_contiguous_is_one_memcpy(orc):
    rng = np.random.default_rng(5)
    src = _random_pool(rng, 2, 50, 8, 24)
    dst = _random_pool(rng, 2, 60, 8, 24)
    a, b, n = 7, 31, 19
    want = [x.copy() for x in dst.k + dst.v]
    t = src.tile_bytes
    for w, s in zip(want, src.k + src.v):
        w.reshape(-1)[b * t:(b + n) * t] = s.reshape(-1)[a * t:(a + n) * t]
    orc.copy(src, dst, np.arange(a, a + n), np.arange(b, b + n))
    assert all(np.array_equal(w, x) for w, x in zip(want, dst.k + dst.v))


def pin_copy_leaves_rest_untouched(orc):
    rng = np.random.default_rng(9)
    src = _random_pool(rng, 4, 30, 2, 16)
    dst = _random_pool(rng, 4, 30, 2, 16)
    before = dst.copy()
    ms = np.array([3, 9, 27], np.int32)
    md = np.array([0, 29, 14], np.int32)
    orc.copy(src, dst, ms, md)
    keep = np.setdiff1d(np.arange(30), md)
    for x, y in zip(dst.k + dst.v, before.k + before.v):
        assert np.array_equal(x[keep], y[keep])
    for x, y in zip(dst.k + dst.v, src.k + src.v):
        assert np.array_equal(x[md], y[ms])


# --------------------------------------------------------------------------- pack / unpack
def pin_pack_matches_index_select(orc):
    rng = np.random.default_rng(13)
    pool = _random_pool(rng, 3, 40, 4, 32)
    blocks = rng.choice(40, 17, replace=False).astype(np.int32)
    got = orc.pack(pool, blocks)
    idx = torch.from_numpy(blocks).long()
    want = torch.stack([torch.stack([torch.index_select(torch.from_numpy(k), 0, idx),
                                     torch.index_select(torch.from_numpy(v), 0, idx)])
                        for k, v in zip(pool.k, pool.v)]).reshape(-1)
    assert torch.equal(torch.from_numpy(got), want)


def pin_pack_unpack_round_trip(orc):
    rng = np.random.default_rng(17)
    src = _random_pool(rng, 2, 33, 4, 16)
    blocks_src = rng.choice(33, 12, replace=False).astype(np.int32)
    blocks_dst = rng.choice(20, 12, replace=False).astype(np.int32)
    dst = HostPool.zeros(2, 20, 4, 16)
    orc.unpack(dst, blocks_dst, orc.pack(src, blocks_src))
    rest = np.setdiff1d(np.arange(20), blocks_dst)
    for x, y in zip(dst.k + dst.v, src.k + src.v):
        assert np.array_equal(x[blocks_dst], y[blocks_src])
        assert not x[rest].any()
    # and back through the same blocks of the same pool: unpack(pack(x)) == x
    again = dst.copy()
    orc.unpack(again, blocks_dst, orc.pack(dst, blocks_dst))
    assert again.equals(dst)


# --------------------------------------------------------------------------- appends
def pin_write_tokens_layout(orc):
    rng = np.random.default_rng(19)
    num_layers, nb, bs, heads, dim, e = 2, 12, 4, 3, 8, 2
    slot = heads * dim * e
    pool = _random_pool(rng, num_layers, nb, bs, slot)
    before = pool.copy()
    table = rng.choice(nb, 6, replace=False).astype(np.int32)
    lo, n_tok = 5, 13
    data = rng.integers(0, 256, (num_layers, 2, n_tok, slot), dtype=np.uint8)
    orc.write_tokens(pool, table, lo, data)
    touched = set()
    for l in range(num_layers):
        for kv, arr in enumerate((pool.k[l], pool.v[l])):
            view = arr.reshape(nb, bs, heads, dim * e)
            for j in range(n_tok):
                t = lo + j
                assert np.array_equal(view[table[t // bs], t % bs].reshape(-1), data[l, kv, j])
                touched.add((int(table[t // bs]), t % bs))
    for l in range(num_layers):
        for a, b in ((pool.k[l], before.k[l]), (pool.v[l], before.v[l])):
            va, vb = a.reshape(nb, bs, slot), b.reshape(nb, bs, slot)
            for blk in range(nb):
                for s in range(bs):
                    if (blk, s) not in touched:
                        assert np.array_equal(va[blk, s], vb[blk, s])


# --------------------------------------------------------------------------- token identity
def pin_token_identity_finds_differences(orc):
    rng = np.random.default_rng(23)
    num_layers, bs, slot, length = 3, 4, 16, 22
    a = _random_pool(rng, num_layers, 10, bs, slot)
    b = _random_pool(rng, num_layers, 12, bs, slot)
    ta = rng.choice(10, 6, replace=False).astype(np.int32)
    tb = rng.choice(12, 6, replace=False).astype(np.int32)
    orc.copy(a, b, ta, tb)
    assert orc.first_token_mismatch(a, ta, b, tb, length) == -1
    for t, layer, use_v, byte in ((0, 0, False, 0), (21, 2, True, slot - 1), (13, 1, True, 5),
                                  (7, 2, False, 9)):
        c = b.copy()
        arr = (c.v if use_v else c.k)[layer]
        arr[tb[t // bs], (t % bs) * slot + byte] ^= 0x40
        assert orc.first_token_mismatch(a, ta, c, tb, length) == t, (t, layer, use_v)
    # a slot beyond the length is not part of the sequence
    c = b.copy()
    c.k[0][tb[5], 3 * slot] ^= 1        # token 23 > length - 1
    assert orc.first_token_mismatch(a, ta, c, tb, length) == -1


# --------------------------------------------------------------------------- multi-stage
def pin_multistage_replay(orc):
    rng = np.random.default_rng(29)
    num_layers, bs, slot = 2, 4, 24
    nb_src, nb_dst = 40, 45
    for initial, appended in ((37, [3, 9, 1, 6]), (16, [4, 4]), (5, []), (0, [7]), (12, [0, 0, 2])):
        final_len = initial + sum(appended)
        nb = _ceil_div(final_len, bs)
        src = _random_pool(rng, num_layers, nb_src, bs, slot)
        dst = _random_pool(rng, num_layers, nb_dst, bs, slot)
        dst0 = dst.copy()
        table = rng.choice(nb_src, nb + 1, replace=False).astype(np.int32)
        free = rng.permutation(nb_dst).astype(np.int32)
        bounds = stage_bounds(initial, appended, bs)
        assert len(bounds) == len(appended) + 1
        events, cur = [], initial
        for k, (length, lo, hi) in enumerate(bounds):
            if k > 0:
                data = rng.integers(0, 256, (num_layers, 2, appended[k - 1], slot), dtype=np.uint8)
                events.append(("append", cur, data))
                cur += appended[k - 1]
            assert length == cur
            events.append(("stage", length, lo, hi))
        dst_table, stages = orc.migrate(src, dst, table, free, events)
        # every appended token's K and V bytes sit in its source slot
        for ev in events:
            if ev[0] == "append":
                for j in range(ev[2].shape[2]):
                    t = ev[1] + j
                    cols = slice((t % bs) * slot, (t % bs + 1) * slot)
                    for l in range(num_layers):
                        assert np.array_equal(src.k[l][table[t // bs], cols], ev[2][l, 0, j])
                        assert np.array_equal(src.v[l][table[t // bs], cols], ev[2][l, 1, j])
        assert len(dst_table) == nb
        assert np.array_equal(dst_table, free[:nb])
        assert np.array_equal(np.concatenate([s for s, _ in stages] + [np.zeros(0, np.int32)]),
                              table[:nb])
        assert orc.first_token_mismatch(src, table, dst, dst_table, final_len) == -1
        rest = np.setdiff1d(np.arange(nb_dst), dst_table)
        for x, y in zip(dst.k + dst.v, dst0.k + dst0.v):
            assert np.array_equal(x[rest], y[rest])
        # non-final stages hold whole blocks only
        for length, lo, hi in bounds[:-1]:
            assert lo % bs == 0 and hi % bs == 0


# --------------------------------------------------------------------------- decode attention
def pin_16bit_conversions_exhaustive(orc):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    want_h = bits.view(np.float16).astype(np.float64)
    want_b = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    got_h = np.array([orc.half_to_double(int(b)) for b in bits])
    got_b = np.array([orc.bf16_to_double(int(b)) for b in bits])
    for got, want in ((got_h, want_h), (got_b, want_b)):
        nan = np.isnan(want)
        assert np.array_equal(np.isnan(got), nan)
        assert np.array_equal(got[~nan], want[~nan])


def _attn_case(rng, num_layers, nb, bs, kv_heads, head_dim, group, ctx, dtype):
    """A random pool, queries and block tables for decode attention."""
    slot = kv_heads * head_dim * 2
    t = bs * slot
    vals = rng.uniform(-1, 1, size=(2, num_layers, nb, t // 2))
    if dtype == "fp16":
        bits = vals.astype(np.float16).view(np.uint16)
    else:
        bits = torch.from_numpy(vals.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    pool = HostPool([np.ascontiguousarray(bits[0, l]).view(np.uint8) for l in range(num_layers)],
                    [np.ascontiguousarray(bits[1, l]).view(np.uint8) for l in range(num_layers)], bs, slot)
    batch = len(ctx)
    stride = max(1, max(-(-c // bs) for c in ctx))
    tables = np.stack([rng.choice(nb, stride, replace=False) for _ in range(batch)]).astype(np.int32)
    qv = rng.uniform(-1, 1, size=(num_layers, batch, kv_heads * group, head_dim))
    if dtype == "fp16":
        q = qv.astype(np.float16).view(np.uint16)
    else:
        q = torch.from_numpy(qv.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    return pool, q, tables


def _dense(pool, layer, table, ctx, kv_heads, head_dim, dtype, which):
    """[ctx, kv_heads, head_dim] float64 of a sequence's K or V, by torch indexing."""
    arr = (pool.k if which == "k" else pool.v)[layer].view(np.uint16).reshape(pool.num_blocks, pool.block_size,
                                                                             kv_heads, head_dim)
    t = torch.from_numpy(arr.view(np.int16)).view(torch.float16 if dtype == "fp16" else torch.bfloat16).double()
    tok = torch.arange(ctx)
    return t[torch.from_numpy(table.astype(np.int64))[tok // pool.block_size], tok % pool.block_size]


def _as_f64(bits, dtype):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.float16 if dtype == "fp16" else torch.bfloat16).double()


def pin_attention_matches_torch(orc):
    rng = np.random.default_rng(31)
    for dtype, group, ctx in (("fp16", 1, [5, 16, 33, 1]), ("bf16", 4, [40, 7]), ("fp16", 2, [64, 0, 3])):
        L, nb, bs, hkv, d = 2, 40, 8, 2, 16
        pool, q, tables = _attn_case(rng, L, nb, bs, hkv, d, group, ctx, dtype)
        scale = 1 / np.sqrt(d)
        got = orc.decode_attention(pool, hkv, d, dtype, q, tables, ctx, scale)
        qf = _as_f64(q, dtype)
        for l in range(L):
            for b, c in enumerate(ctx):
                if c == 0:
                    assert not got[l, b].any()
                    continue
                K = _dense(pool, l, tables[b], c, hkv, d, dtype, "k").repeat_interleave(group, dim=1)
                V = _dense(pool, l, tables[b], c, hkv, d, dtype, "v").repeat_interleave(group, dim=1)
                s = torch.einsum("hd,thd->ht", qf[l, b], K) * scale
                want = torch.einsum("ht,thd->hd", torch.softmax(s, dim=1), V).numpy()
                assert np.allclose(got[l, b], want, rtol=1e-12, atol=1e-12), (dtype, l, b)


def pin_attention_special_cases(orc):
    rng = np.random.default_rng(37)
    L, nb, bs, hkv, d, group = 1, 12, 4, 2, 8, 3
    # one token: the output is that token's V row
    pool, q, tables = _attn_case(rng, L, nb, bs, hkv, d, group, [1], "fp16")
    got = orc.decode_attention(pool, hkv, d, "fp16", q, tables, [1], 0.7)
    V = _dense(pool, 0, tables[0], 1, hkv, d, "fp16", "v")[0].repeat_interleave(group, dim=0).numpy()
    assert np.array_equal(got[0, 0], V)
    # zero scale: uniform weights, the output is the mean of V
    pool, q, tables = _attn_case(rng, L, nb, bs, hkv, d, group, [11], "bf16")
    got = orc.decode_attention(pool, hkv, d, "bf16", q, tables, [11], 0.0)
    V = _dense(pool, 0, tables[0], 11, hkv, d, "bf16", "v").repeat_interleave(group, dim=1).mean(0).numpy()
    assert np.allclose(got[0, 0], V, rtol=1e-13, atol=1e-13)
    # grouped heads: V non-zero in KV head 1 only -> query heads of group 1 alone see it
    for a in pool.v:
        a.view(np.uint16).reshape(nb, bs, hkv, d)[:, :, 0, :] = 0
    got = orc.decode_attention(pool, hkv, d, "bf16", q, tables, [11], 0.5)
    assert not got[0, 0, :group].any() and np.abs(got[0, 0, group:]).max() > 0


def pin_attention_token_order_invariant(orc):
    """Attention is a sum over tokens: permuting where tokens live (blocks
    and slots) together with the table leaves the output unchanged."""
    rng = np.random.default_rng(41)
    L, nb, bs, hkv, d, group, ctx = 1, 16, 4, 1, 8, 2, 16
    pool, q, tables = _attn_case(rng, L, nb, bs, hkv, d, group, [ctx], "fp16")
    base = orc.decode_attention(pool, hkv, d, "fp16", q, tables, [ctx], 0.3)
    # shuffle the four blocks of the table, moving their contents along
    perm = rng.permutation(4)
    moved = pool.copy()
    new_table = tables.copy()
    spare = [x for x in range(nb) if x not in set(tables[0].tolist())][:4]
    for j in range(4):
        src_blk, dst_blk = tables[0, perm[j]], spare[j]
        for arr_new, arr_old in zip(moved.k + moved.v, pool.k + pool.v):
            arr_new[dst_blk] = arr_old[src_blk]
        new_table[0, j] = dst_blk
    # new logical block j holds old block perm[j]: token order changes, the set does not
    got = orc.decode_attention(moved, hkv, d, "fp16", q, new_table, [ctx], 0.3)
    assert np.allclose(got, base, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------- cross-layout
LAYOUTS = (NHD, HND, HCNX, HDN)
_UINT = {1: np.uint8, 2: np.uint16, 4: np.uint32}


def _arrange(logical, layout, e):
    """Byte image of a [bs, H, D] tile in ``layout``, by numpy reshape/transpose."""
    bs, heads, dim = logical.shape
    if layout == NHD:
        a = logical
    elif layout == HND:
        a = logical.transpose(1, 0, 2)
    elif layout == HCNX:
        x = 16 // e
        a = logical.reshape(bs, heads, dim // x, x).transpose(1, 2, 0, 3)
    else:
        a = logical.transpose(1, 2, 0)
    return np.ascontiguousarray(a).view(np.uint8).reshape(-1)


def _logical(tile, layout, bs, heads, dim, e):
    """[bs, H, D] view of a tile's bytes in ``layout``: the inverse of _arrange."""
    a = np.ascontiguousarray(tile).view(_UINT[e])
    if layout == NHD:
        return a.reshape(bs, heads, dim)
    if layout == HND:
        return a.reshape(heads, bs, dim).transpose(1, 0, 2)
    if layout == HCNX:
        x = 16 // e
        return a.reshape(heads, dim // x, bs, x).transpose(2, 0, 1, 3).reshape(bs, heads, dim)
    return a.reshape(heads, dim, bs).transpose(2, 0, 1)


XGEOMS = [(8, 3, 16, 2), (3, 2, 32, 1), (4, 2, 8, 4), (16, 1, 24, 2)]   # bs, heads, head_dim, elem_bytes


def pin_xlayout_offsets_bijective(orc):
    for bs, heads, dim, e in XGEOMS:
        tile = bs * heads * dim * e
        for lay in LAYOUTS:
            offs = sorted(orc.layout_offset(lay, t, h, d, bs, heads, dim, e)
                          for t in range(bs) for h in range(heads) for d in range(dim))
            assert offs == list(range(0, tile, e)), (lay, bs, heads, dim, e)
    assert orc.layout_offset(4, 0, 0, 0, 8, 1, 16, 2) == -1
    assert orc.layout_offset(HCNX, 0, 0, 0, 8, 1, 16, 3) == -1


def pin_xlayout_matches_numpy_transposes(orc):
    for bs, heads, dim, e in XGEOMS:
        n_el = bs * heads * dim
        assert n_el < 256 ** e
        a_k = (np.arange(n_el) % 256 ** e).astype(_UINT[e]).reshape(bs, heads, dim)
        a_v = a_k[::-1].copy()
        slot = heads * dim * e
        rng = np.random.default_rng(bs * 1000 + dim)
        for lk in LAYOUTS:
            for lv in LAYOUTS:
                src = _random_pool(rng, 2, 3, bs, slot)
                src.k[1][0] = a_k.view(np.uint8).reshape(-1)
                src.v[1][0] = a_v.view(np.uint8).reshape(-1)
                dst = _random_pool(rng, 2, 4, bs, slot)
                orc.copy_layout(src, (NHD, NHD), dst, (lk, lv), [0], [3], heads, dim, e)
                assert np.array_equal(dst.k[1][3], _arrange(a_k, lk, e)), (bs, dim, e, lk)
                assert np.array_equal(dst.v[1][3], _arrange(a_v, lv, e)), (bs, dim, e, lv)
                back = _random_pool(rng, 2, 2, bs, slot)
                orc.copy_layout(dst, (lk, lv), back, (NHD, NHD), [3], [1], heads, dim, e)
                assert np.array_equal(back.k[1][1], src.k[1][0]) and np.array_equal(back.v[1][1], src.v[1][0])


def pin_xlayout_round_trip_and_composition(orc):
    rng = np.random.default_rng(37)
    bs, heads, dim, e, num_layers = 8, 2, 16, 2, 2
    slot = heads * dim * e
    src = _random_pool(rng, num_layers, 6, bs, slot)
    ms = np.array([4, 0, 5], np.int32)
    md = np.array([1, 6, 3], np.int32)
    pairs = [(a, b) for a in LAYOUTS for b in LAYOUTS]
    for x in pairs:
        # same layouts on both sides: exactly the byte copy
        d1, d2 = _random_pool(rng, num_layers, 7, bs, slot), None
        d2 = d1.copy()
        orc.copy_layout(src, x, d1, x, ms, md, heads, dim, e)
        orc.copy(src, d2, ms, md)
        assert d1.equals(d2), x
        for y in pairs[(x[0] * 5 + x[1]) % 4::3]:
            mid = _random_pool(rng, num_layers, 7, bs, slot)
            orc.copy_layout(src, x, mid, y, ms, md, heads, dim, e)
            back = src.copy()
            orc.copy_layout(mid, y, back, x, md, ms, heads, dim, e)
            assert back.equals(src), (x, y)
            for z in (pairs[(y[1] * 3 + x[0]) % len(pairs)],):
                via = _random_pool(rng, num_layers, 8, bs, slot)
                direct = via.copy()
                orc.copy_layout(mid, y, via, z, md, [7, 2, 0], heads, dim, e)
                orc.copy_layout(src, x, direct, z, ms, [7, 2, 0], heads, dim, e)
                assert via.equals(direct), (x, y, z)


def pin_xlayout_appends_and_identity(orc):
    rng = np.random.default_rng(41)
    bs, heads, dim, e, num_layers, nb = 8, 3, 16, 2, 2, 9
    slot = heads * dim * e
    table = rng.choice(nb, 4, replace=False).astype(np.int32)
    lo, n_tok = 3, 21
    data = rng.integers(0, 256, (num_layers, 2, n_tok, slot), dtype=np.uint8)
    base = _random_pool(rng, num_layers, nb, bs, slot)
    a, b = base.copy(), base.copy()
    orc.write_tokens_layout(a, (NHD, NHD), table, lo, data, heads, dim, e)
    orc.write_tokens(b, table, lo, data)
    assert a.equals(b)
    for lay in ((HDN, HCNX), (HND, HDN), (HCNX, NHD)):
        p = base.copy()
        orc.write_tokens_layout(p, lay, table, lo, data, heads, dim, e)
        for l in range(num_layers):
            for kv, arr in enumerate((p.k[l], p.v[l])):
                for j in range(n_tok):
                    t = lo + j
                    view = _logical(arr[table[t // bs]], lay[kv], bs, heads, dim, e)
                    want = data[l, kv, j].view(np.uint16).reshape(heads, dim)
                    assert np.array_equal(view[t % bs], want), (lay, l, kv, t)
        # slots outside [lo, lo + n_tok) are untouched
        for l in range(num_layers):
            for kv, (x, y) in enumerate(((p.k[l], base.k[l]), (p.v[l], base.v[l]))):
                for blk in range(nb):
                    vx = _logical(x[blk], lay[kv], bs, heads, dim, e)
                    vy = _logical(y[blk], lay[kv], bs, heads, dim, e)
                    for s in range(bs):
                        hit = blk in table and lo <= list(table).index(blk) * bs + s < lo + n_tok
                        if not hit:
                            assert np.array_equal(vx[s], vy[s])
    # token identity across layouts finds a planted element at its token
    length = 29
    src = _random_pool(rng, num_layers, nb, bs, slot)
    dst = _random_pool(rng, num_layers, nb + 2, bs, slot)
    tb = rng.choice(nb + 2, 4, replace=False).astype(np.int32)
    sl, dl = (HND, HDN), (HCNX, NHD)
    orc.copy_layout(src, sl, dst, dl, table, tb, heads, dim, e)
    assert orc.first_token_mismatch_layout(src, sl, table, dst, dl, tb, length, heads, dim, e) == -1
    for t, l, kv, h, d in ((0, 0, 0, 0, 0), (28, 1, 1, 2, 15), (17, 1, 0, 1, 9), (9, 0, 1, 2, 3)):
        c = dst.copy()
        arr = (c.k if kv == 0 else c.v)[l][tb[t // bs]]
        logical = _logical(arr, dl[kv], bs, heads, dim, e).copy()
        logical[t % bs, h, d] ^= 0x0100
        arr[:] = _arrange(logical, dl[kv], e)
        assert orc.first_token_mismatch_layout(src, sl, table, c, dl, tb, length, heads, dim, e) == t
    c = dst.copy()
    arr = c.k[0][tb[3]]
    logical = _logical(arr, dl[0], bs, heads, dim, e).copy()
    logical[5, 0, 0] ^= 1                                   # token 29: beyond the length
    arr[:] = _arrange(logical, dl[0], e)
    assert orc.first_token_mismatch_layout(src, sl, table, c, dl, tb, length, heads, dim, e) == -1


def pin_xlayout_unpack(orc):
    rng = np.random.default_rng(47)
    bs, heads, dim, e, num_layers = 8, 2, 16, 2, 2
    slot = heads * dim * e
    src = _random_pool(rng, num_layers, 9, bs, slot)
    blocks_src = np.array([7, 2, 5, 0], np.int32)
    blocks_dst = np.array([1, 6, 3, 8], np.int32)
    for sl, dl in (((HCNX, HDN), (NHD, NHD)), ((NHD, HND), (HDN, HCNX)), ((HND, HND), (HND, HND))):
        staging = orc.pack(src, blocks_src)
        # staging layouts equal to the pool's: exactly the plain unpack
        a = _random_pool(rng, num_layers, 10, bs, slot)
        b = a.copy()
        orc.unpack_layout(a, dl, blocks_dst, staging, dl, heads, dim, e)
        orc.unpack(b, blocks_dst, staging)
        assert a.equals(b)
        # pack in one layout, unpack into another == the converting stage copy
        c = _random_pool(rng, num_layers, 10, bs, slot)
        d = c.copy()
        orc.unpack_layout(c, dl, blocks_dst, staging, sl, heads, dim, e)
        orc.copy_layout(src, sl, d, dl, blocks_src, blocks_dst, heads, dim, e)
        assert c.equals(d), (sl, dl)
    # a staging tile arranged by numpy in HDN lands as the NHD (logical) image
    logical = (np.arange(bs * heads * dim) * 7 % 65521).astype(np.uint16).reshape(bs, heads, dim)
    one = HostPool.zeros(1, 2, bs, slot)
    staging = np.concatenate([_arrange(logical, HDN, e), _arrange(logical[::-1].copy(), HCNX, e)])
    orc.unpack_layout(one, (NHD, NHD), [1], staging, (HDN, HCNX), heads, dim, e)
    assert np.array_equal(one.k[0][1], logical.view(np.uint8).reshape(-1))
    assert np.array_equal(one.v[0][1], logical[::-1].copy().view(np.uint8).reshape(-1))
    assert not one.k[0][0].any()


def pin_xlayout_multistage_replay(orc):
    rng = np.random.default_rng(43)
    bs, heads, dim, e, num_layers = 8, 2, 16, 2, 2
    slot = heads * dim * e
    initial, appended = 19, [5, 11, 2]
    final_len = initial + sum(appended)
    nb = _ceil_div(final_len, bs)
    for sl, dl in (((NHD, NHD), (HCNX, HDN)), ((HCNX, HDN), (NHD, NHD)), ((HND, HDN), (HDN, HND))):
        src = _random_pool(rng, num_layers, 20, bs, slot)
        dst = _random_pool(rng, num_layers, 22, bs, slot)
        dst0 = dst.copy()
        table = rng.choice(20, nb, replace=False).astype(np.int32)
        free = rng.permutation(22).astype(np.int32)
        events, cur = [], initial
        for k, (length, lo, hi) in enumerate(stage_bounds(initial, appended, bs)):
            if k > 0:
                data = rng.integers(0, 256, (num_layers, 2, appended[k - 1], slot), dtype=np.uint8)
                events.append(("append", cur, data))
                cur += appended[k - 1]
            events.append(("stage", length, lo, hi))
        dst_table, _ = orc.migrate(src, dst, table, free, events, layouts=(sl, dl, heads, dim, e))
        # every appended token sits in its source slot, in the source's layouts
        for ev in events:
            if ev[0] == "append":
                for j in range(ev[2].shape[2]):
                    t = ev[1] + j
                    for l in range(num_layers):
                        for kv, arr in ((0, src.k[l]), (1, src.v[l])):
                            got = _logical(arr[table[t // bs]], sl[kv], bs, heads, dim, e)[t % bs]
                            want = np.ascontiguousarray(ev[2][l, kv, j]).view(_UINT[e]).reshape(heads, dim)
                            assert np.array_equal(got, want), (sl, l, kv, t)
        assert np.array_equal(dst_table, free[:nb])
        for l in range(num_layers):
            for kv in range(2):
                sarr = (src.k if kv == 0 else src.v)[l]
                darr = (dst.k if kv == 0 else dst.v)[l]
                for j in range(nb):
                    a = _logical(sarr[table[j]], sl[kv], bs, heads, dim, e)
                    b = _logical(darr[dst_table[j]], dl[kv], bs, heads, dim, e)
                    assert np.array_equal(a, b), (sl, dl, l, kv, j)
        rest = np.setdiff1d(np.arange(22), dst_table)
        for x, y in zip(dst.k + dst.v, dst0.k + dst0.v):
            assert np.array_equal(x[rest], y[rest])


# In file order: cheap checks of a part run before the pins that would write
# through a broken part of it.
ALL_PINS = [v for k, v in globals().items() if k.startswith("pin_")]
