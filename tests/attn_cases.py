"""Decode-attention test cases and the error bound the GPU kernel is held to.

Shared by the GPU parity test (tests/test_gpu_attention.py) and the CPU test
that shows the bound is tight enough to catch a lost partition
(tests/test_attn_tolerance.py): both build a case's inputs here, from the
seeded generators, so they see the same bytes.

The bound, per output element (layer l, sequence b, query head h, dim d),
with n = ctx[b] tokens, u = 2^-24 (fp32 unit roundoff) and lambda = 8:

    tol = A * (eps_p + lambda * u * (2 * sqrt(depth(n)) + 4 * (sqrt(D) + 2) * S + 2))
          + lambda * sqrt(n) * u_lo / W + u

  A     = sum_t p_t |v_td| / sum_t p_t, the softmax-weighted mean of |V|,
          computed by the fp64 oracle on the pool with V's sign bits
          cleared (the weights p_t are the same).  Every error below is
          relative to a weight p_t or to a sum of weighted terms, so it
          reaches the output scaled by (at most twice) this mean, not by
          |out|, which cancellation can make arbitrarily small.
  eps_p the kernel feeds each weight to the P.V product as its 16-bit
          rounding plus the 16-bit rounding of the remainder: relative
          error 2^-16 for bf16 (8-bit significands), 2^-22 for fp16.
  depth the longest chain of fp32 additions behind one output: the 16
          terms of one matrix-core product, then a wavefront's token groups
          of its partition (two products each, the weight's high and low
          parts; a wavefront takes every fourth group of 16 tokens of a
          partition of 2048), the merge of four wavefronts and the merge of
          ceil(n / 2048) partitions:
              depth(n) = 16 + 2 * ceil(min(n, 2048) / 64) + 4 + ceil(n / 2048).
          In the probabilistic rounding-error model (Higham and Mary, 2019)
          a chain of k additions is off by lambda * sqrt(k) * u of the sum
          of the magnitudes of its terms with probability at least
          1 - 2 exp(-lambda^2 / 2); the weighted sum and the weight sum
          each contribute one such term.  Rescaling a running sum by
          exp(m_old - m_new) multiplies the weighted sum and the weight sum
          by the same number, so its rounding cancels in their ratio.
  S     = scale * sum_d |q_d|, a bound on |score| since |k| <= 1.  A score
          is a D-term fp32 dot product (error lambda * sqrt(D) * u * S) and
          enters as exp(score - max), so a weight's relative error is twice
          that, plus the rounding of the scaled scores and the exponential's
          own few ulps (the "+ 2" terms); exp(x)'s relative error equals
          x's absolute error.
  u_lo  fp16 only: the remainder of a small weight falls below fp16's
          normal range and is rounded to a multiple of 2^-24, an absolute
          error of at most 2^-25 per token (|v| <= 1); n of them, of random
          sign, over the weight sum W = sum_t exp(score_t - max score) >= 1,
          computed here in float64 from the gathered keys.
  u     absolute floor, for rows whose A is 0 (a sequence of no tokens,
          whose output the kernel sets to exactly 0).

Dropping one 2048-token partition of a 50,000-token sequence moves the
output by ~2e-3; this bound is ~1e-4 there, and tests/test_attn_tolerance.py
checks on the CPU that every such drop is rejected.
"""
from __future__ import annotations

import math

import numpy as np

import oracle
from oracle import HostPool
from paper_2406_03243_amd import workloads as wl

LAMBDA = 8.0
U32 = 2.0 ** -24
EPS_P = {"bf16": 2.0 ** -16, "fp16": 2.0 ** -22}

# The library splits a call into (sequence, partition) items of 2048 tokens
# and launches the partial kernel on 128 items at a time; the tests use the
# split to drop exactly what one item, or one launch, covers.
PART_TOKENS = 2048
ITEMS_PER_LAUNCH = 128

# layers, blocks, block_size, kv_heads, head_dim, group, context lengths, dtype, V positive
CASES = [
    (2, 300, 16, 2, 128, 8, [1, 17, 600, 0, 1024], "fp16", False),
    (2, 200, 16, 4, 64, 1, [513, 31, 7], "bf16", False),
    (1, 400, 16, 2, 128, 4, [4096, 5, 2000], "bf16", False),
    (3, 100, 8, 1, 64, 2, [96, 95, 97, 1], "fp16", False),
    (1, 3200, 16, 1, 128, 2, [50000, 49999, 40000], "fp16", False),  # 70 partitions of 2048
    (1, 8400, 16, 1, 128, 2, [131072, 120000, 20000], "fp16", False), # 133 items: two launches,
                                                                      # the third sequence spans both
    (2, 120, 16, 1, 128, 16, [700, 33], "bf16", False),               # 16 query heads on one KV head
    (1, 300, 4, 2, 64, 4, [1000, 3, 62], "bf16", False),              # 4-token blocks
    (1, 3200, 16, 1, 128, 2, [50000, 49999, 40000], "bf16", True),    # V in [0, 1]: output far from 0
    (1, 1200, 32, 2, 64, 4, [9000, 20000, 1025], "fp16", True),       # 32-token blocks, partial last items
]


def case_id(c) -> str:
    return f"{c[7]}_D{c[4]}_G{c[5]}_bs{c[2]}_ctx{max(c[6])}" + ("_vpos" if c[8] else "")


def case_seed(c) -> int:
    return 500 + sum(c[6]) % 97 + (1000 if c[8] else 0)


def random_case(seed: int):
    g = wl.stream(seed, wl.LENGTHS)
    bs = int(g.choice([1, 2, 4, 8, 16, 32]))
    batch = int(g.integers(1, 9))
    ctx = [int(x) for x in g.integers(0, 1500, batch)]
    if g.random() < 0.2:
        ctx[int(g.integers(0, batch))] = 0
    blocks = max(1, max(-(-c // bs) for c in ctx)) + int(g.integers(0, 20))
    return (int(g.integers(1, 4)), blocks, bs, int(g.integers(1, 5)), int(g.choice([64, 128])),
            int(g.choice([1, 2, 4, 8, 16])), ctx, str(g.choice(["fp16", "bf16"])), False)


_inputs_cache = {}


def case_inputs(case, seed: int):
    """Host inputs of a case: (pool, q bits [L][B][Hq][D], tables [B][stride],
    ctx, scale).  Pool tensors are drawn as the harness draws them for a
    device pool (K of every layer, then V, one sub-stream each).  The last
    few cases drawn are kept (drawing the largest takes seconds); callers
    must not modify them."""
    key = (case_id(case), tuple(case[6]), case[1], seed)
    if key not in _inputs_cache:
        if len(_inputs_cache) >= 4:
            _inputs_cache.pop(next(iter(_inputs_cache)))
        _inputs_cache[key] = _draw_inputs(case, seed)
    return _inputs_cache[key]


def _draw_inputs(case, seed: int):
    num_layers, num_blocks, bs, kv_heads, head_dim, group, ctx, dtype, vpos = case
    tile = bs * kv_heads * head_dim * 2
    draw = [wl.values16(seed, wl.SRC_VALUES, num_blocks * tile // 2, dtype, sub=idx)
            for idx in range(2 * num_layers)]
    if vpos:
        for idx in range(num_layers, 2 * num_layers):
            draw[idx] = draw[idx] & np.uint16(0x7FFF)
    tiles = [d.view(np.uint8).reshape(num_blocks, tile) for d in draw]
    pool = HostPool(tiles[:num_layers], tiles[num_layers:], bs, kv_heads * head_dim * 2)
    q_heads = kv_heads * group
    batch = len(ctx)
    stride = max(1, max(-(-c // bs) for c in ctx))
    g = wl.stream(seed, wl.EXTRA)
    tables = np.stack([g.choice(num_blocks, stride, replace=False) for _ in range(batch)]).astype(np.int32)
    q = wl.values16(seed, wl.APPEND_VALUES, num_layers * batch * q_heads * head_dim, dtype).reshape(
        num_layers, batch, q_heads, head_dim)
    return pool, q, tables, list(ctx), 1.0 / math.sqrt(head_dim)


def decode16(bits: np.ndarray, dtype: str) -> np.ndarray:
    bits = np.asarray(bits, np.uint16)
    if dtype == "fp16":
        return bits.view(np.float16).astype(np.float64)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def abs_v_pool(pool: HostPool) -> HostPool:
    """The pool with every V element's sign bit cleared (|V|)."""
    v = [(a.view(np.uint16) & np.uint16(0x7FFF)).view(np.uint8) for a in pool.v]
    return HostPool(pool.k, v, pool.block_size, pool.slot_bytes)


def depth(n):
    """Longest chain of fp32 additions behind an output of an n-token
    sequence (see the module docstring)."""
    n = np.asarray(n, np.float64)
    return 16.0 + 2.0 * np.ceil(np.minimum(n, PART_TOKENS) / 64.0) + 4.0 + np.ceil(n / PART_TOKENS)


def weight_sum(pool: HostPool, kv_heads: int, head_dim: int, dtype: str, q, tables, ctx, scale):
    """W[l][b][h] = sum_t exp(score_t - max_t score_t), in float64 from the
    gathered keys (1 for an empty sequence)."""
    q = np.asarray(q, np.uint16)
    num_layers, batch, q_heads, _ = q.shape
    group = q_heads // kv_heads
    bs = pool.block_size
    out = np.ones((num_layers, batch, q_heads, 1))
    for l in range(num_layers):
        keys = pool.k[l].view(np.uint16).reshape(pool.num_blocks, bs, kv_heads, head_dim)
        for b in range(batch):
            n = ctx[b]
            if n <= 0:
                continue
            t = np.arange(n)
            blocks = np.asarray(tables[b])[t // bs]
            for h in range(q_heads):
                kt = decode16(keys[blocks, t % bs, h // group], dtype)             # [n][D]
                sc = scale * (kt @ decode16(q[l, b, h], dtype))
                out[l, b, h, 0] = np.exp(sc - sc.max()).sum()
    return out


def tolerance(orc, pool: HostPool, kv_heads: int, head_dim: int, dtype: str, q, tables, ctx, scale):
    """Per-element bound on |kernel - oracle| (see the module docstring)."""
    A = orc.decode_attention(abs_v_pool(pool), kv_heads, head_dim, dtype, q, tables, ctx, scale)
    S = scale * np.abs(decode16(q, dtype)).sum(axis=-1, keepdims=True)          # [L][B][Hq][1]
    n = np.asarray(ctx, np.float64)[None, :, None, None]
    rel = EPS_P[dtype] + LAMBDA * U32 * (2.0 * np.sqrt(depth(n)) + 4.0 * (math.sqrt(head_dim) + 2.0) * S + 2.0)
    if dtype == "fp16":
        W = weight_sum(pool, kv_heads, head_dim, dtype, q, tables, ctx, scale)
        lo = LAMBDA * np.sqrt(n) * U32 / 2 / W
    else:
        lo = 0.0
    return A * rel + lo + U32


def excess(got, want, tol) -> np.ndarray:
    """|got - want| / tol: the bound holds where this is at most 1."""
    return np.abs(np.asarray(got, np.float64) - want) / tol


def items(ctx):
    """The (sequence, first token, end token) items of a call, in launch order."""
    out = []
    for b, n in enumerate(ctx):
        for t in range(0, n, PART_TOKENS):
            out.append((b, t, min(n, t + PART_TOKENS)))
    return out


def drop_tokens(tables, ctx, block_size: int, b: int, lo: int, hi: int):
    """Tables and lengths of the same call with tokens [lo, hi) of sequence b
    removed.  lo is a multiple of the block size and hi is one too unless it
    is the sequence's end, so whole blocks go; attention does not depend on
    the order of the tokens, so this is attention over the rest."""
    assert lo % block_size == 0 and (hi % block_size == 0 or hi == ctx[b])
    row = list(tables[b, :-(-ctx[b] // block_size)])
    keep = row[:lo // block_size] + row[-(-hi // block_size):]
    new = np.zeros_like(tables)
    new[:] = tables
    new[b, :] = 0
    new[b, :len(keep)] = keep
    lens = list(ctx)
    lens[b] = ctx[b] - (hi - lo)
    return new, lens


def default_oracle():
    return oracle.default()
