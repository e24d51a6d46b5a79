"""Property tests on the host (no GPU): the library's planner against the
oracle's on hypothesis-drawn tables, free lists and token ranges, and the
append-only race freedom of a multi-stage migration driven through the
library's coordinator (no block a stage copied is written again by decoding,
the condition under which a stage may run while decoding goes on, Llumnix
§4.2)."""
import numpy as np
from hypothesis import given, settings, strategies as st

import oracle
from paper_2406_03243_amd import llmig
from paper_2406_03243_amd.llmig import MigrationHandle


@st.composite
def plan_cases(draw):
    bs = draw(st.sampled_from([1, 2, 3, 4, 7, 16]))
    length = draw(st.integers(0, 200))
    nb = -(-length // bs)
    # ranges: mostly valid stage bounds, sometimes not
    lo = draw(st.integers(0, length)) // bs * bs if draw(st.booleans()) else draw(st.integers(-3, length + 3))
    hi = draw(st.sampled_from([length, max(lo, 0) + draw(st.integers(0, 3)) * bs,
                               draw(st.integers(-2, length + 5))]))
    pool = draw(st.integers(max(nb, 1), 4 * max(nb, 1) + 8))
    ids = draw(st.permutations(list(range(pool))))
    table = list(ids[:nb + draw(st.integers(-1, 2))]) if nb else []
    free = list(draw(st.permutations(list(range(pool))))[:draw(st.integers(0, pool))])
    # plant a repeat or a negative id now and then
    if table and draw(st.integers(0, 9)) == 0:
        table[draw(st.integers(0, len(table) - 1))] = table[0] if draw(st.booleans()) else -1
    if free and draw(st.integers(0, 9)) == 0:
        free[draw(st.integers(0, len(free) - 1))] = free[0] if draw(st.booleans()) else -5
    return bs, length, lo, hi, np.array(table, np.int32), np.array(free, np.int32)


@settings(max_examples=600, deadline=None)
@given(plan_cases())
def test_plan_matches_oracle_on_drawn_cases(case):
    bs, length, lo, hi, table, free = case
    code, oms, omd = oracle.default().plan(table, free, length, lo, hi, bs)
    try:
        ms, md = llmig.llmig_plan(table, free, length, lo, hi, bs)
        got = oracle.OK
    except llmig.LlmigError as e:
        got, ms, md = e.code, np.zeros(0, np.int32), np.zeros(0, np.int32)
    assert got == code, (case, got, code)
    assert np.array_equal(ms, oms) and np.array_equal(md, omd)


@st.composite
def schedules(draw):
    bs = draw(st.sampled_from([1, 4, 16]))
    initial = draw(st.integers(0, 120))
    appends = draw(st.lists(st.integers(0, 40), max_size=6))
    return bs, initial, appends


@settings(max_examples=300, deadline=None)
@given(schedules())
def test_no_copied_block_is_written_again(sched):
    """Replay appends and stages in order through the coordinator, tracking
    which logical blocks each stage copied; every append must land in blocks
    no earlier stage has copied, and the stages must cover the sequence."""
    bs, initial, appends = sched
    total = initial + sum(appends)
    nb = -(-total // bs)
    table = np.arange(1000, 1000 + nb + 1, dtype=np.int32)
    free = np.arange(nb + 5, dtype=np.int32)
    m = MigrationHandle(bs)
    copied = set()
    length = initial
    left = free
    for k in range(len(appends) + 1):
        if k > 0:
            written = {t // bs for t in range(length, length + appends[k - 1])}
            assert not written & copied, (sched, k, sorted(written & copied))
            length += appends[k - 1]
        final = k == len(appends)
        ms, md = m.next(table, length, final, left)
        stage_blocks = {int(np.where(table == s)[0][0]) for s in ms}
        assert not stage_blocks & copied                 # no block is copied twice
        copied |= stage_blocks
        left = left[len(md):]
    assert copied == set(range(nb))                       # the stages partition the sequence
    assert np.array_equal(m.commit(), free[:nb])
