"""The migration coordinator (handshake of Llumnix §4.2) on the host: stage
by stage reservation, refusal when the destination cannot reserve, abort
with release of every reserved block, commit after the final stage.  No GPU:
the planning half of the coordinator (llmig_migration_next) is pure host
code; its stages are checked against the oracle's planner and the oracle's
stage boundaries."""
import numpy as np
import pytest

import oracle
from paper_2406_03243_amd.llmig import LlmigError, MigrationHandle


def code_of(fn, *a):
    try:
        fn(*a)
    except LlmigError as e:
        return e.name
    return "OK"


def test_stages_match_the_oracle():
    rng = np.random.default_rng(404)
    orc = oracle.default()
    for trial in range(300):
        bs = int(rng.choice([1, 2, 4, 16]))
        initial = int(rng.integers(0, 300))
        appended = [int(x) for x in rng.integers(0, 40, rng.integers(0, 5))]
        total = initial + sum(appended)
        nb = -(-total // bs)
        ids = rng.permutation(4 * nb + 50).astype(np.int32)
        table, free = ids[:nb + 1], ids[nb + 1:2 * nb + 20]
        m = MigrationHandle(bs)
        left = free
        for length, lo, hi in oracle.stage_bounds(initial, appended, bs):
            final = hi == length and (length, lo, hi) == oracle.stage_bounds(initial, appended, bs)[-1]
            ms, md = m.next(table, length, final, left)
            code, oms, omd = orc.plan(table, left, length, lo, hi, bs)
            assert code == oracle.OK
            assert np.array_equal(ms, oms) and np.array_equal(md, omd), (trial, length, lo, hi)
            left = left[len(md):]
            info = m.info()
            assert info["copied_tokens"] == hi
        assert m.info()["state"] == "FINISHED"
        dst_table = m.commit()
        assert np.array_equal(dst_table, free[:nb])
        assert m.info()["state"] == "COMMITTED"


def test_refused_preallocation_changes_nothing_and_abort_releases():
    bs = 16
    table = np.arange(100, 140, dtype=np.int32)
    free = np.arange(500, 540, dtype=np.int32)
    m = MigrationHandle(bs)
    ms, md = m.next(table, 300, False, free)           # 18 whole blocks
    assert len(md) == 18
    before = m.info()
    # the destination has only 2 free blocks left: the next stage (3 blocks) is refused
    assert code_of(m.next, table, 340, False, free[18:20]) == "ENOSPC"
    assert m.info() == before
    released = m.abort()
    assert np.array_equal(released, free[:18])
    assert m.info()["state"] == "ABORTED" and m.info()["reserved_blocks"] == 0
    assert code_of(m.next, table, 340, True, free[18:]) == "EINVAL"
    assert code_of(m.commit) == "EINVAL"
    assert code_of(m.abort) == "EINVAL"


@pytest.mark.parametrize("abort_after", [0, 1, 2, 3])
def test_abort_after_any_stage_returns_exactly_the_reserved_blocks(abort_after):
    """The request finished or was preempted (or the peer failed) after a stage."""
    bs = 4
    table = np.arange(0, 60, dtype=np.int32)
    free = np.arange(1000, 1060, dtype=np.int32)
    m = MigrationHandle(bs)
    length, left, consumed = 50, free, 0
    for k in range(abort_after):
        _, md = m.next(table, length, False, left)
        left = left[len(md):]
        consumed += len(md)
        length += 7
    released = m.abort()
    assert np.array_equal(released, free[:consumed])
    assert m.info()["state"] == "ABORTED"


def test_commit_needs_the_final_stage():
    m = MigrationHandle(16)
    table = np.arange(10, dtype=np.int32)
    free = np.arange(50, 60, dtype=np.int32)
    assert code_of(m.commit) == "EINVAL"
    m.next(table, 40, False, free)                      # blocks 0, 1
    assert code_of(m.commit) == "EINVAL"
    assert m.info()["state"] == "ACTIVE"
    ms, md = m.next(table, 41, True, free[2:])          # block 2 (partial)
    assert list(ms) == [2] and list(md) == [52]
    assert code_of(m.next, table, 45, True, free[3:]) == "EINVAL"   # nothing may follow the final stage
    assert list(m.commit()) == [50, 51, 52]
    assert code_of(m.abort) == "EINVAL"


def test_final_stage_with_nothing_left():
    m = MigrationHandle(8)
    table = np.arange(4, dtype=np.int32)
    free = np.arange(10, 14, dtype=np.int32)
    m.next(table, 32, False, free)
    ms, md = m.next(table, 32, True, free[4:])
    assert len(ms) == 0 and m.info()["state"] == "FINISHED"
    assert list(m.commit()) == [10, 11, 12, 13]


def test_length_cannot_shrink_and_bad_arguments_change_nothing():
    m = MigrationHandle(16)
    table = np.arange(20, dtype=np.int32)
    free = np.arange(100, 120, dtype=np.int32)
    m.next(table, 100, False, free)                      # copied 96
    before = m.info()
    assert code_of(m.next, table, 90, False, free[6:]) == "EINVAL"
    assert code_of(m.next, table[:3], 200, False, free[6:]) == "EINVAL"     # table misses blocks
    bad = table.copy()
    bad[7] = -3
    assert code_of(m.next, bad, 130, False, free[6:]) == "ERANGE"
    dup = free[6:].copy()
    dup[1] = dup[0]
    assert code_of(m.next, table, 140, False, dup) == "EINVAL"
    assert m.info() == before
    with pytest.raises(LlmigError):
        MigrationHandle(0)


def test_handshake_with_injected_faults():
    """Random runs of the handshake: decoding appends, stages are
    pre-allocated against a destination that sometimes runs short, the
    request sometimes finishes early, the peer sometimes fails.  The
    reservation always equals the consumed head of the free list, an abort
    returns it whole, and a commit returns one block per logical block."""
    rng = np.random.default_rng(77)
    outcomes = {"commit": 0, "enospc": 0, "finished": 0, "peer": 0}
    for trial in range(400):
        bs = int(rng.choice([1, 4, 16]))
        length = int(rng.integers(1, 200))
        table = rng.permutation(2000).astype(np.int32)[:(length + 400) // bs + 2]
        free = rng.permutation(np.arange(5000, 5000 + 600)).astype(np.int32)
        avail = int(rng.integers(0, 600))             # what the destination can still reserve
        m = MigrationHandle(bs)
        consumed = 0
        while True:
            remaining = -(-length // bs) - m.info()["copied_tokens"] // bs
            final = remaining <= 1 or m.info()["stages"] >= 6
            r = rng.random()
            if r < 0.05:                                # peer failure
                outcome = "peer"
                break
            try:
                _, md = m.next(table, length, final, free[consumed:avail])
            except LlmigError as e:
                assert e.name == "ENOSPC"
                outcome = "enospc"
                break
            assert np.array_equal(md, free[consumed:consumed + len(md)])
            consumed += len(md)
            assert m.info()["reserved_blocks"] == consumed
            if final:
                outcome = "commit"
                break
            if rng.random() < 0.1:                      # the request completed mid-migration
                outcome = "finished"
                break
            length += int(rng.integers(1, 40))
        if outcome == "commit":
            got = m.commit()
            assert len(got) == -(-length // bs) and np.array_equal(got, free[:consumed])
        else:
            got = m.abort()
            assert np.array_equal(got, free[:consumed])
        outcomes[outcome] += 1
    assert all(v > 0 for v in outcomes.values()), outcomes
