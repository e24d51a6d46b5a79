"""Every plausible single mistake planted in a copy of the CPU oracle must
fail at least one pin: evidence that the pins can tell a wrong oracle from a
right one.  The mistakes are planted in temporary copies of the oracle's C
source and of its Python replay code; the oracle itself is never changed."""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import oracle

# (name, text in the oracle's source, replacement, which occurrence)
MUTANTS = [
    ("plan_dst_reversed", "out_dst[k] = dst_free_list[k];", "out_dst[k] = dst_free_list[n - 1 - k];", 0),
    ("plan_src_no_offset", "out_src[k] = src_table[first_block + k];", "out_src[k] = src_table[k];", 0),
    ("plan_walk_inclusive", "for (int64_t t = from_tok; t < to_tok; t++) {",
     "for (int64_t t = from_tok; t <= to_tok; t++) {", 0),
    ("plan_enospc_off_by_one", "if (n > dst_free_len)", "if (n >= dst_free_len)", 0),
    ("plan_rejects_final_partial", "if (to_tok % bs != 0 && to_tok != len)", "if (to_tok % bs != 0)", 0),
    ("plan_no_boundary_check", "if (from_tok % bs != 0)", "if (0)", 0),
    ("plan_no_dst_duplicate_check", "if (dst_free_list[a] == dst_free_list[b])", "if (0)", 0),
    ("plan_no_src_duplicate_check", "if (src_table[first_block + a] == src_table[first_block + b])",
     "if (0)", 0),
    ("plan_erange_missed", "if (src_table[first_block + k] < 0 || dst_free_list[k] < 0)",
     "if (src_table[first_block + k] < -1 || dst_free_list[k] < -5)", 0),
    ("plan_short_table_accepted", "if (src_table_len < blocks_of_len)",
     "if (src_table_len < blocks_of_len - 1)", 0),
    ("plan_out_cap_unchecked", "if (n > out_cap)", "if (n > out_cap + 1)", 0),
    ("copy_pairs_misaligned", "src_k[l] + (int64_t)map_src[i] * tile_bytes",
     "src_k[l] + (int64_t)map_src[n - 1 - i] * tile_bytes", 0),
    ("copy_v_from_k", "src_v[l] + (int64_t)map_src[i] * tile_bytes",
     "src_k[l] + (int64_t)map_src[i] * tile_bytes", 0),
    ("copy_drops_last_layer", "for (int32_t l = 0; l < num_layers; l++) {\n            memcpy(dst_k[l]",
     "for (int32_t l = 0; l < num_layers - 1; l++) {\n            memcpy(dst_k[l]", 0),
    ("pack_transposed", "int64_t slot = ((int64_t)l * 2 + kv) * n + i;",
     "int64_t slot = (i * 2 + kv) * num_layers + l;", 0),
    ("unpack_reversed", "memcpy(pool[l] + (int64_t)blocks[i] * tile_bytes,",
     "memcpy(pool[l] + (int64_t)blocks[n - 1 - i] * tile_bytes,", 0),
    ("write_tokens_slot_shift", "+ (t % bs) * slot_bytes;", "+ ((t + 1) % bs) * slot_bytes;", 0),
    ("write_tokens_kv_swapped", "uint8_t *const *pool = (kv == 0) ? pool_k : pool_v;",
     "uint8_t *const *pool = (kv == 0) ? pool_v : pool_k;", 2),
    ("mismatch_skips_v", "if (memcmp(a_v[l] + off_a, b_v[l] + off_b, (size_t)slot_bytes) != 0)",
     "if (0)", 0),
    ("mismatch_skips_last_token", "for (int64_t t = 0; t < len; t++) {\n        for (int32_t l = 0;",
     "for (int64_t t = 0; t < len - 1; t++) {\n        for (int32_t l = 0;", 0),
    ("attn_head_map", "int32_t g = h / group;", "int32_t g = h % kv_heads;", 0),
    ("attn_no_scale", "                    s *= scale;\n", "", 0),
    ("attn_denominator_counts", "denom += w;", "denom += 1.0;", 0),
    ("attn_drops_last_token", "for (int32_t t = 0; t < ctx[b]; t++) {\n                    int64_t row",
     "for (int32_t t = 0; t < ctx[b] - 1; t++) {\n                    int64_t row", 1),
    ("attn_v_from_k", "o[d] += w * elem(pool_v[l]", "o[d] += w * elem(pool_k[l]", 0),
    ("half_exponent_bias", "exp - 25", "exp - 24", 0),
    ("half_subnormal_scale", "ldexp((double)frac, -24)", "ldexp((double)frac, -25)", 0),
    ("attn_row_slot", "+ t % block_size) * kv_heads + g;", "+ t % block_size) * kv_heads;", 0),
    ("layout_hnd_is_nhd", "index = (h * bs + t) * head_dim + d;", "index = (t * heads + h) * head_dim + d;", 0),
    ("layout_hcnx_group_swapped", "index = ((h * groups + d / x) * bs + t) * x + d % x;",
     "index = ((h * groups + d % x) * bs + t) * x + d / x;", 0),
    ("layout_hcnx_x_fixed", "int64_t x = 16 / elem_bytes;", "int64_t x = 8;", 0),
    ("layout_hdn_head_inner", "index = (h * head_dim + d) * bs + t;", "index = (d * heads + h) * bs + t;", 0),
    ("copy_layout_v_takes_k_layout", "d + oracle_layout_offset(dst_layouts[kv]",
     "d + oracle_layout_offset(dst_layouts[0]", 0),
    ("copy_layout_ignores_src_layout", "s + oracle_layout_offset(src_layouts[kv]",
     "s + oracle_layout_offset(dst_layouts[kv]", 0),
    ("write_tokens_layout_block_index", "oracle_layout_offset(layouts[kv], t % bs, h, e,",
     "oracle_layout_offset(layouts[kv], t / bs, h, e,", 0),
    ("mismatch_layout_b_read_as_a", "tb + oracle_layout_offset(b_layouts[kv]",
     "tb + oracle_layout_offset(a_layouts[kv]", 0),
    ("unpack_layout_reads_pool_layout", "s + oracle_layout_offset(staging_layouts[kv]",
     "s + oracle_layout_offset(pool_layouts[kv]", 0),
    ("unpack_layout_slot_order", "const uint8_t *s = staging + (((int64_t)l * 2 + kv) * n + i) * tile_bytes;",
     "const uint8_t *s = staging + ((i * 2 + kv) * num_layers + l) * tile_bytes;", 0),
]

# Mistakes in the Python side of the oracle (the multi-stage replay and the
# stage schedule of Llumnix §4.2), planted in a copy of oracle/__init__.py.
PY_MUTANTS = [
    ("replay_free_list_not_advanced", "free = free[len(md):]", "free = free"),
    ("replay_appends_dropped", "self.write_tokens(src, src_table, ev[1], ev[2])", "pass"),
    ("replay_table_from_sources", "dst_table.extend(int(x) for x in md)", "dst_table.extend(int(x) for x in ms)"),
    ("schedule_final_whole_blocks", "end = length if final else (length // block_size) * block_size",
     "end = (length // block_size) * block_size"),
    ("schedule_restarts_each_stage", "        copied = end", "        copied = 0"),
    ("replay_layout_appends_dropped",
     "self.write_tokens_layout(src, layouts[0], src_table, ev[1], ev[2], *layouts[2:])", "pass"),
    ("replay_layout_copy_unconverted", "self.copy_layout(src, layouts[0], dst, layouts[1], ms, md, *layouts[2:])",
     "self.copy(src, dst, ms, md)"),
]

RUNNER = r"""
import sys
sys.path[:0] = [sys.argv[1], sys.argv[2]]
import pins
from oracle import Oracle
orc = Oracle(sys.argv[3])
for pin in pins.ALL_PINS:
    try:
        pin(orc)
    except Exception:            # a wrong result, or an error where none is due
        print("FAILED", pin.__name__, flush=True)
print("DONE", flush=True)
"""


def _run_pins(root, tests_dir, lib):
    """Pins that fail on one mutant, run in a process of its own: a mutant
    that writes outside its buffers may kill that process, which counts as
    caught (the pins cannot pass on it)."""
    res = subprocess.run([sys.executable, "-c", RUNNER, root, tests_dir, lib],
                         capture_output=True, text=True, timeout=600)
    lines = res.stdout.splitlines()
    failed = [ln.split()[1] for ln in lines if ln.startswith("FAILED ")]
    if res.returncode != 0 or "DONE" not in lines:
        failed.append(f"process died ({res.returncode})")
    return failed


def _mutate(src, old, new, which):
    parts = src.split(old)
    assert len(parts) > which + 1, f"mutation site not found: {old!r}"
    return old.join(parts[:which + 1]) + new + old.join(parts[which + 1:])


def test_every_planted_mistake_fails_a_pin():
    src = open(oracle.SOURCE).read()
    tests_dir = os.path.dirname(os.path.abspath(__file__))
    root = os.path.dirname(tests_dir)
    with tempfile.TemporaryDirectory() as tmp:
        libs = {}
        for name, old, new, which in MUTANTS:
            path = os.path.join(tmp, name + ".c")
            with open(path, "w") as f:
                f.write(_mutate(src, old, new, which))
            libs[name] = oracle.build(path, os.path.join(tmp, name + ".so"), quiet=True)
        with ThreadPoolExecutor(max_workers=6) as pool:
            futures = {name: pool.submit(_run_pins, root, tests_dir, lib) for name, lib in libs.items()}
            caught = {name: f.result() for name, f in futures.items()}
    missed = [name for name, failed in caught.items() if not failed]
    assert not missed, f"mutants no pin catches: {missed}"


def test_every_planted_replay_mistake_fails_a_pin():
    py_src = open(os.path.join(os.path.dirname(oracle.SOURCE), "__init__.py")).read()
    tests_dir = os.path.dirname(os.path.abspath(__file__))
    lib = oracle.LIBRARY if os.path.exists(oracle.LIBRARY) else oracle.build()   # the unchanged C oracle
    with tempfile.TemporaryDirectory() as tmp:
        roots = {}
        for name, old, new in PY_MUTANTS:
            root = os.path.join(tmp, name)
            os.makedirs(os.path.join(root, "oracle"))
            with open(os.path.join(root, "oracle", "__init__.py"), "w") as f:
                f.write(_mutate(py_src, old, new, 0))
            roots[name] = root
        with ThreadPoolExecutor(max_workers=6) as pool:
            futures = {name: pool.submit(_run_pins, root, tests_dir, lib) for name, root in roots.items()}
            caught = {name: f.result() for name, f in futures.items()}
    missed = [name for name, failed in caught.items() if not failed]
    assert not missed, f"replay mutants no pin catches: {missed}"
