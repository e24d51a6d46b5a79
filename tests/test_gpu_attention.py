"""GPU parity of paged decode attention (the decode work measured beside a
migration) against the fp64 oracle, through the C ABI.

Inputs and the error bound come from tests/attn_cases.py: the bound is
derived from the kernel's arithmetic (fp32 accumulation, the 16-bit hi/lo
split of the softmax weights) and scales with the softmax-weighted mean of
|V| rather than with the sequence length alone, so a lost 2048-token
partition, or a lost launch of partitions, fails it (checked on the CPU by
tests/test_attn_tolerance.py).  Each case prints its largest absolute error
and its largest error-to-bound ratio."""
import sys

import numpy as np
import pytest
import torch

import attn_cases as ac
from paper_2406_03243_amd import harness
from paper_2406_03243_amd import workloads as wl

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2406_03243_amd.llmig import LlmigError, Pool, decode_workspace_bytes, llmig_decode_attention


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def device_pool(case, host):
    num_layers, num_blocks, bs, kv_heads, head_dim, _, _, dtype, _ = case
    shape = wl.PoolShape(num_layers, num_blocks, bs, kv_heads, head_dim, dtype)
    k, v = harness.alloc_layers(shape)
    for t, a in zip(k + v, host.k + host.v):
        harness.tile_view(t).copy_(torch.from_numpy(a))
    return k, v


def run_case(case, seed):
    num_layers, num_blocks, bs, kv_heads, head_dim, group, ctx, dtype, _ = case
    host, qbits, tables, ctx, scale = ac.case_inputs(case, seed)
    k, v = device_pool(case, host)
    pool = Pool(k, v)
    q_heads = kv_heads * group
    tdt = harness.TORCH_DTYPE[dtype]
    q = torch.from_numpy(qbits.view(np.int16)).view(tdt).cuda()
    tab = torch.from_numpy(tables).cuda()
    out = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(1, decode_workspace_bytes(ctx, num_layers, q_heads, head_dim)), dtype=torch.uint8,
                     device="cuda")
    llmig_decode_attention(pool, q, tab, ctx, scale, ws, out)
    torch.cuda.synchronize()
    orc = ac.default_oracle()
    want = orc.decode_attention(host, kv_heads, head_dim, dtype, qbits, tables, ctx, scale)
    tol = ac.tolerance(orc, host, kv_heads, head_dim, dtype, qbits, tables, ctx, scale)
    got = out.cpu().numpy().astype(np.float64)
    err = np.abs(got - want)
    ratio = ac.excess(got, want, tol)
    say(f"max |error| {err.max():.3g}, max error / bound {ratio.max():.3g}, max |out| {np.abs(want).max():.3g}")
    bad = ~(ratio <= 1.0)           # NaN counts as bad
    assert not bad.any(), f"max error {err.max():.3g} (bound ratio {np.nanmax(ratio):.3g}) at {np.argwhere(bad)[:5].tolist()}"
    return pool, err.max()


@pytest.mark.parametrize("case", ac.CASES, ids=ac.case_id)
def test_decode_attention_matches_oracle(case):
    say("decode attention", case)
    run_case(case, seed=ac.case_seed(case))


@pytest.mark.parametrize("seed", range(30))
def test_decode_attention_random(seed):
    """30 seeded random shapes: layers, block size 1-32, KV heads, head dim,
    group size, batch, context lengths (zero included) and type."""
    case = ac.random_case(30_000 + seed)
    say("decode attention random", seed, case)
    run_case(case, seed=30_000 + seed)


def test_decode_attention_rejects_unsupported():
    say("decode attention errors")
    shape = wl.PoolShape(1, 20, 16, 2, 96, "fp16")
    k, v = harness.alloc_layers(shape)
    pool = Pool(k, v)
    q = torch.zeros((1, 1, 2, 96), dtype=torch.float16, device="cuda")
    tab = torch.zeros((1, 2), dtype=torch.int32, device="cuda")
    out = torch.zeros(q.shape, dtype=torch.float32, device="cuda")
    ws = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    with pytest.raises(LlmigError):                      # head_dim 96
        llmig_decode_attention(pool, q, tab, [10], 1.0, ws, out)
    shape = wl.PoolShape(1, 20, 16, 2, 64, "fp16")
    k, v = harness.alloc_layers(shape)
    pool = Pool(k, v)
    q = torch.zeros((1, 1, 6, 64), dtype=torch.float16, device="cuda")     # group 3
    out = torch.zeros(q.shape, dtype=torch.float32, device="cuda")
    with pytest.raises(LlmigError):
        llmig_decode_attention(pool, q, tab, [10], 1.0, ws, out)
    q = torch.zeros((1, 1, 4, 64), dtype=torch.float16, device="cuda")
    out = torch.zeros(q.shape, dtype=torch.float32, device="cuda")
    with pytest.raises(LlmigError):                      # 40 tokens need 3 blocks, the table holds 2
        llmig_decode_attention(pool, q, tab, [40], 1.0, ws, out)
    with pytest.raises(LlmigError):                      # workspace too small
        llmig_decode_attention(pool, q, tab, [10], 1.0, ws[:16], out)
    with pytest.raises(LlmigError):                      # workspace not 16-byte aligned
        llmig_decode_attention(pool, q, tab, [10], 1.0, ws[4:], out)
    out_off = torch.zeros(out.numel() + 1, dtype=torch.float32, device="cuda")[1:].view(out.shape)
    with pytest.raises(LlmigError):                      # out not 16-byte aligned
        llmig_decode_attention(pool, q, tab, [10], 1.0, ws, out_off)
    bad_q = [torch.zeros((2, 1, 4, 64), dtype=torch.float16, device="cuda"),   # layers
             torch.zeros((1, 1, 4, 128), dtype=torch.float16, device="cuda"),  # head_dim
             torch.zeros((1, 1, 4, 64), dtype=torch.bfloat16, device="cuda")]  # type
    for bq in bad_q:
        with pytest.raises(ValueError):
            llmig_decode_attention(pool, bq, tab, [10], 1.0, ws, torch.zeros(bq.shape, dtype=torch.float32,
                                                                             device="cuda"))
    with pytest.raises(ValueError):                      # one length per sequence
        llmig_decode_attention(pool, q, tab, [10, 10], 1.0, ws, out)
    with pytest.raises(ValueError):                      # a table row per sequence
        q2 = torch.zeros((1, 2, 4, 64), dtype=torch.float16, device="cuda")
        llmig_decode_attention(pool, q2, tab, [10, 10], 1.0, ws, torch.zeros(q2.shape, dtype=torch.float32,
                                                                              device="cuda"))
    llmig_decode_attention(pool, q, tab, [10], 1.0, ws, out)
    torch.cuda.synchronize()
