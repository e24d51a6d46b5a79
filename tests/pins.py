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
               ceil(len/bs) blocks, stages partitioning the block set.
"""
from __future__ import annotations

import json
import os

import numpy as np
import torch

from oracle import EINVAL, ENOSPC, ERANGE, OK, HostPool, stage_bounds

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


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
