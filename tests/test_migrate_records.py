"""The Python driver's stage records follow the library's coordinator (host
only, no GPU): over hypothesis-drawn schedules, the records that
migrate.Migration keeps (token range, blocks, consumed free-list entries)
equal the oracle's stage bounds for the schedule (Llumnix §4.2) and the
coordinator's own state, and the committed destination table equals the
consumed head of the free list."""
import math

import numpy as np
from hypothesis import given, settings, strategies as st

import oracle
from paper_2406_03243_amd import migrate


def _drive_scheduled(bs, initial, appended, table, free):
    m = migrate.Migration(None, None, table, free, None, block_size=bs)
    length = initial
    m.plan(length, final=not appended)
    for k, c in enumerate(appended):
        length += c
        m.plan(length, final=k == len(appended) - 1)
    return m, length


@settings(max_examples=300, deadline=None)
@given(bs=st.sampled_from([1, 2, 3, 4, 16]), initial=st.integers(0, 300),
       appended=st.lists(st.integers(0, 70), max_size=6), seed=st.integers(0, 2**32 - 1))
def test_scheduled_records_follow_the_coordinator(bs, initial, appended, seed):
    total = initial + sum(appended)
    rng = np.random.default_rng(seed)
    ids = rng.permutation(2 * math.ceil(total / bs) + 8).astype(np.int32)
    nb = math.ceil(total / bs)
    table, free = ids[:nb], ids[nb:]
    m, length = _drive_scheduled(bs, initial, appended, table, free)
    assert [(r.length, r.from_tok, r.to_tok) for r in m.stages] == oracle.stage_bounds(initial, appended, bs)
    info = m.coord.info()
    assert info["state"] == "FINISHED" and info["copied_tokens"] == length == m.copied_tok
    assert info["stages"] == len(m.stages) and info["reserved_blocks"] == sum(r.blocks for r in m.stages)
    assert sum(r.blocks for r in m.stages) == math.ceil(length / bs)
    assert np.array_equal(m.commit(), m.dst_table)
    assert np.array_equal(m.dst_table, free[:math.ceil(length / bs)])


@settings(max_examples=200, deadline=None)
@given(bs=st.sampled_from([1, 4, 16]), initial=st.integers(1, 400),
       per_stage=st.lists(st.integers(1, 40), min_size=1, max_size=10), last=st.integers(0, 3),
       max_stages=st.integers(2, 8))
def test_timed_rule_records_follow_the_coordinator(bs, initial, per_stage, last, max_stages):
    """The time-driven driver's decision (final when at most ``last`` blocks
    remain, or at the stage cap), with the tokens each stage produced drawn
    instead of timed."""
    total = initial + sum(per_stage)
    nb = math.ceil(total / bs)
    ids = np.arange(2 * nb + 8, dtype=np.int32)[::-1].copy()
    table, free = ids[:nb], ids[nb:]
    m = migrate.Migration(None, None, table, free, None, block_size=bs)
    length = initial
    m.plan(length, final=False)
    appended = []
    for k, c in enumerate(per_stage):
        length += c
        appended.append(c)
        if m.remaining_blocks(length) <= last or len(m.stages) + 1 >= max_stages or k == len(per_stage) - 1:
            m.plan(length, final=True)
            break
        m.plan(length, final=False)
    assert m.stages[-1].final and m.copied_tok == length
    assert [(r.length, r.from_tok, r.to_tok) for r in m.stages] == oracle.stage_bounds(initial, appended, bs)
    assert len(m.stages) <= max(max_stages, 2)
    assert m.coord.info()["copied_tokens"] == length
    assert np.array_equal(m.commit(), free[:math.ceil(length / bs)])
