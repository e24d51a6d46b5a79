"""GPU parity of paged decode attention (the decode work measured beside a
migration) against the fp64 oracle, through the C ABI.

Tolerance: inputs are exact fp16/bf16 values in [-1, 1]; the kernel
multiplies them on the matrix cores with fp32 accumulation, exponentiates in
fp32, and carries the softmax weights into the P.V product as a 16-bit high
part plus the 16-bit rounding of the rest (about 2^-16 relative for bf16,
2^-22 for fp16).  A softmax-
weighted mean of values in [-1, 1] accumulated over n tokens in fp32 is off
by at most about n * eps32 = n * 6e-8, so a case whose longest sequence has
n tokens allows an absolute error of max(1e-4, n * 6e-8) plus 1e-4
relative."""
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
    from paper_2406_03243_amd.llmig import LlmigError, Pool, decode_workspace_bytes, llmig_decode_attention

EPS32, RTOL = 6e-8, 1e-4


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def run_case(num_layers, num_blocks, bs, kv_heads, head_dim, group, ctx, dtype, seed):
    shape = wl.PoolShape(num_layers, num_blocks, bs, kv_heads, head_dim, dtype)
    k, v = harness.alloc_layers(shape)
    harness.fill_from_host(k + v, seed, wl.SRC_VALUES, dtype)
    pool = Pool(k, v)
    q_heads = kv_heads * group
    batch = len(ctx)
    stride = max(1, max(-(-c // bs) for c in ctx))
    g = wl.stream(seed, wl.EXTRA)
    tables = np.stack([g.choice(num_blocks, stride, replace=False) for _ in range(batch)]).astype(np.int32)
    qbits = wl.values16(seed, wl.APPEND_VALUES, num_layers * batch * q_heads * head_dim, dtype).reshape(
        num_layers, batch, q_heads, head_dim)
    tdt = harness.TORCH_DTYPE[dtype]
    q = torch.from_numpy(qbits.view(np.int16)).view(tdt).cuda()
    tab = torch.from_numpy(tables).cuda()
    out = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(1, decode_workspace_bytes(ctx, num_layers, q_heads, head_dim)), dtype=torch.uint8,
                     device="cuda")
    scale = 1.0 / np.sqrt(head_dim)
    llmig_decode_attention(pool, q, tab, ctx, scale, ws, out)
    torch.cuda.synchronize()
    host = HostPool(harness.snapshot(k), harness.snapshot(v), bs, pool.slot_bytes)
    want = oracle.default().decode_attention(host, kv_heads, head_dim, dtype, qbits, tables, ctx, scale)
    got = out.cpu().numpy().astype(np.float64)
    err = np.abs(got - want)
    atol = max(1e-4, max(ctx) * EPS32)
    bad = err > atol + RTOL * np.abs(want)
    assert not bad.any(), f"max error {err.max():.3g} at {np.argwhere(bad)[:5].tolist()}"
    return pool, err.max()


CASES = [
    # layers, blocks, block_size, kv_heads, head_dim, group, context lengths, dtype
    (2, 300, 16, 2, 128, 8, [1, 17, 600, 0, 1024], "fp16"),
    (2, 200, 16, 4, 64, 1, [513, 31, 7], "bf16"),
    (1, 400, 16, 2, 128, 4, [4096, 5, 2000], "bf16"),
    (3, 100, 8, 1, 64, 2, [96, 95, 97, 1], "fp16"),
    (1, 3200, 16, 1, 128, 2, [50000, 49999, 40000], "fp16"),  # 138 partitions of 1024: two launches of items
    (2, 120, 16, 1, 128, 16, [700, 33], "bf16"),               # 16 query heads on one KV head
    (1, 300, 4, 2, 64, 4, [1000, 3, 62], "bf16"),             # 4-token blocks: a 16-token group spans blocks
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[7]}_D{c[4]}_G{c[5]}_ctx{max(c[6])}")
def test_decode_attention_matches_oracle(case):
    say("decode attention", case)
    run_case(*case, seed=500 + sum(case[6]) % 97)


def random_case(seed):
    g = wl.stream(seed, wl.LENGTHS)
    bs = int(g.choice([1, 2, 4, 8, 16, 32]))
    batch = int(g.integers(1, 9))
    ctx = [int(x) for x in g.integers(0, 1500, batch)]
    if g.random() < 0.2:
        ctx[int(g.integers(0, batch))] = 0
    blocks = max(1, max(-(-c // bs) for c in ctx)) + int(g.integers(0, 20))
    return (int(g.integers(1, 4)), blocks, bs, int(g.integers(1, 5)), int(g.choice([64, 128])),
            int(g.choice([1, 2, 4, 8, 16])), ctx, str(g.choice(["fp16", "bf16"])))


@pytest.mark.parametrize("seed", range(30))
def test_decode_attention_random(seed):
    """30 seeded random shapes: layers, block size 1-32, KV heads, head dim,
    group size, batch, context lengths (zero included) and type."""
    case = random_case(30_000 + seed)
    say("decode attention random", seed, case)
    run_case(*case, seed=30_000 + seed)


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
