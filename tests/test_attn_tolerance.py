"""The decode-attention error bound can fail (CPU only).

The GPU parity test accepts the kernel's output when it lies within the
bound of tests/attn_cases.py of the fp64 oracle.  A bound that grows with
the sequence length alone would also accept an output that lost a whole
2048-token partition of a long sequence, or the partitions of the second
launch of a call, which is exactly the kind of mistake a flash-decoding
merge can make.  Here, for every fixed case, the oracle's own result with
such a piece dropped must violate the bound, while the exact result passes
it with room to spare."""
import numpy as np
import pytest

import attn_cases as ac


def _oracle_and_bound(case):
    host, q, tables, ctx, scale = ac.case_inputs(case, ac.case_seed(case))
    _, _, bs, kv_heads, head_dim, _, _, dtype, _ = case
    orc = ac.default_oracle()
    want = orc.decode_attention(host, kv_heads, head_dim, dtype, q, tables, ctx, scale)
    tol = ac.tolerance(orc, host, kv_heads, head_dim, dtype, q, tables, ctx, scale)
    return orc, host, q, tables, ctx, scale, want, tol


def _dropped(orc, case, host, q, tables, ctx, scale, pieces):
    """Oracle output with the token ranges pieces[b] = [(lo, hi), ...] removed."""
    _, _, bs, kv_heads, head_dim, _, _, dtype, _ = case
    t, n = tables, list(ctx)
    for b, ranges in pieces.items():
        for lo, hi in sorted(ranges, reverse=True):        # later ranges first: earlier offsets stay valid
            t, n = ac.drop_tokens(t, n, bs, b, lo, hi)
    return orc.decode_attention(host, kv_heads, head_dim, dtype, q, t, n, scale)


# cases with a sequence of several partitions (the two-launch case, whose
# oracle calls take seconds each, is the second test's)
MULTI = [c for c in ac.CASES if ac.PART_TOKENS < max(c[6]) <= 50000]


@pytest.mark.parametrize("case", MULTI, ids=ac.case_id)
def test_dropping_one_partition_violates_the_bound(case):
    orc, host, q, tables, ctx, scale, want, tol = _oracle_and_bound(case)
    assert ac.excess(want, want, tol).max() == 0.0
    checked = 0
    for b, n in enumerate(ctx):
        parts = [(lo, hi) for (bb, lo, hi) in ac.items(ctx) if bb == b]
        if len(parts) < 2:
            continue
        for j in sorted({0, len(parts) // 2, len(parts) - 1}):
            got = _dropped(orc, case, host, q, tables, ctx, scale, {b: [parts[j]]})
            ratio = ac.excess(got[:, b], want[:, b], tol[:, b]).max()
            print(f"sequence {b} ({n} tokens), partition {j} of {len(parts)} dropped: "
                  f"max error / bound {ratio:.3g}")
            assert ratio > 1.0, f"sequence {b}: dropping partition {j} stays within the bound"
            checked += 1
    assert checked > 0


@pytest.mark.parametrize("case", [c for c in ac.CASES if len(ac.items(c[6])) > ac.ITEMS_PER_LAUNCH],
                         ids=ac.case_id)
def test_dropping_the_second_launch_violates_the_bound(case):
    orc, host, q, tables, ctx, scale, want, tol = _oracle_and_bound(case)
    late = ac.items(ctx)[ac.ITEMS_PER_LAUNCH:]
    pieces = {}
    for b, lo, hi in late:
        pieces.setdefault(b, []).append((lo, hi))
    # the items of one sequence in the second launch are a run at its end: drop it as one range
    pieces = {b: [(min(r[0] for r in rs), max(r[1] for r in rs))] for b, rs in pieces.items()}
    got = _dropped(orc, case, host, q, tables, ctx, scale, pieces)
    for b in pieces:
        ratio = ac.excess(got[:, b], want[:, b], tol[:, b]).max()
        print(f"second launch dropped: sequence {b} keeps {ctx[b] - (pieces[b][0][1] - pieces[b][0][0])} of "
              f"{ctx[b]} tokens, max error / bound {ratio:.3g}")
        assert ratio > 1.0


def test_bound_is_small_against_the_output():
    """Where the weighted mean of |V| is not tiny (a one-token row can make
    it so, and then the absolute terms dominate), the bound is a small
    fraction of it: under 5e-4, about 1.5e-4 at 50,000 tokens."""
    for case in ac.CASES:
        orc, host, q, tables, ctx, scale, want, tol = _oracle_and_bound(case)
        A = orc.decode_attention(ac.abs_v_pool(host), case[3], case[4], case[7], q, tables, ctx, scale)
        live = A > 0.05
        rel = (tol[live] / A[live]).max()
        print(f"{ac.case_id(case)}: largest bound / weighted |V| = {rel:.3g}")
        assert rel < 5e-4


def test_drop_tokens_is_attention_over_the_rest():
    """drop_tokens keeps every other token: on a small case, dropping a
    range equals attention over a table and length built by hand."""
    case = (1, 64, 4, 1, 64, 2, [40], "fp16", False)
    host, q, tables, ctx, scale = ac.case_inputs(case, 7)
    orc = ac.default_oracle()
    t, n = ac.drop_tokens(tables, ctx, 4, 0, 8, 20)
    assert n == [28]
    by_hand = np.zeros_like(tables)
    row = list(tables[0, :2]) + list(tables[0, 5:10])
    by_hand[0, :len(row)] = row
    a = orc.decode_attention(host, 1, 64, "fp16", q, t, n, scale)
    b = orc.decode_attention(host, 1, 64, "fp16", q, by_hand, [28], scale)
    assert np.array_equal(a, b)
    full = orc.decode_attention(host, 1, 64, "fp16", q, tables, ctx, scale)
    assert not np.array_equal(a, full)
