"""The library from plain C, without Python or torch: a C program allocates
two small pools with hipMalloc, fills them, plans and copies one stage
through llmig.h, and checks every tile byte for byte (mapped tiles equal
their sources, the rest of the destination unchanged)."""
import os
import subprocess

import pytest

from paper_2406_03243_amd import llmig

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

C_PROGRAM = r"""
#define __HIP_PLATFORM_AMD__ 1
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include "llmig.h"

enum { L = 3, NB = 64, BS = 16, H = 2, D = 72, E = 2 };   /* 4608-byte tiles: a partial last row */

static uint8_t pattern(int pool, int plane, size_t byte) { return (uint8_t)(byte * 131u + plane * 17u + pool * 101u + (byte >> 8)); }

int main(void)
{
    const size_t tile = (size_t)BS * H * D * E, tensor = tile * NB;
    uint64_t kp[2][L], vp[2][L];
    uint8_t *host = malloc(tensor), *got = malloc(tensor), *want = malloc(tensor);
    for (int p = 0; p < 2; ++p)
        for (int l = 0; l < L; ++l)
            for (int kv = 0; kv < 2; ++kv) {
                void *d = NULL;
                if (hipMalloc(&d, tensor) != hipSuccess) return 10;
                for (size_t b = 0; b < tensor; ++b) host[b] = pattern(p, 2 * l + kv, b);
                if (hipMemcpy(d, host, tensor, hipMemcpyHostToDevice) != hipSuccess) return 11;
                (kv ? vp : kp)[p][l] = (uint64_t)(uintptr_t)d;
            }
    llmig_pool *pool[2];
    for (int p = 0; p < 2; ++p) {
        llmig_pool_desc desc = {L, NB, BS, H, D, E, kp[p], vp[p], LLMIG_LAYOUT_NHD, LLMIG_LAYOUT_NHD};
        if (llmig_pool_create(&desc, &pool[p]) != LLMIG_OK) return 12;
    }
    /* a request of 90 tokens (6 blocks) migrated in one final stage */
    const int32_t table[6] = {40, 3, 17, 63, 0, 28};
    const int32_t free_list[8] = {5, 60, 33, 12, 1, 47, 9, 22};
    int32_t ms[8], md[8];
    int64_t n = 0;
    if (llmig_plan(table, 6, free_list, 8, 90, 0, 90, BS, ms, md, 8, &n) != LLMIG_OK || n != 6) return 13;
    if (llmig_stage(pool[0], pool[1], ms, md, n, 0, NULL) != LLMIG_OK) return 14;
    if (hipDeviceSynchronize() != hipSuccess) return 15;
    for (int l = 0; l < L; ++l)
        for (int kv = 0; kv < 2; ++kv) {
            const uint64_t d = (kv ? vp : kp)[1][l];
            if (hipMemcpy(got, (void *)(uintptr_t)d, tensor, hipMemcpyDeviceToHost) != hipSuccess) return 16;
            for (size_t b = 0; b < tensor; ++b) want[b] = pattern(1, 2 * l + kv, b);
            for (int64_t i = 0; i < n; ++i)
                for (size_t b = 0; b < tile; ++b)
                    want[(size_t)md[i] * tile + b] = pattern(0, 2 * l + kv, (size_t)ms[i] * tile + b);
            if (memcmp(got, want, tensor) != 0) {
                printf("layer %d %c differs\n", l, kv ? 'V' : 'K');
                return 17;
            }
        }
    for (int p = 0; p < 2; ++p) llmig_pool_destroy(pool[p]);
    printf("ok %lld pairs\n", (long long)n);
    return 0;
}
"""


@pytest.mark.gpu
def test_stage_from_plain_c(tmp_path):
    src = tmp_path / "client.c"
    src.write_text(C_PROGRAM)
    exe = tmp_path / "client"
    lib_dir = os.path.dirname(llmig.LIBRARY)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                    "-I", "/opt/rocm/include", str(src), "-o", str(exe), "-L", lib_dir, "-lllmig",
                    "-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath," + lib_dir + ":/opt/rocm/lib"], check=True)
    print("[case] plain C client: one 6-pair stage", flush=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, (res.returncode, res.stdout, res.stderr)
    assert res.stdout.strip() == "ok 6 pairs"
