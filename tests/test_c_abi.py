"""The boundary from plain C: include/purlin.h compiles as C99 (no C++ or
torch types), a C program links against the library, builds host-only plans
through it and reads their tables, and the status codes of invalid calls
match the header.  Runs on the CPU (host-only plans launch nothing)."""

import os
import shutil
import subprocess

import pytest

from paper_2609_36954_amd import purlin as PL

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

C_SOURCE = r"""
#include <stdio.h>
#include <string.h>
#include "purlin.h"

static int fail(const char* what) { printf("FAIL %s\n", what); return 1; }

int main(void) {
    purlin_plan_t plan = NULL;
    purlin_policy pol;
    uint64_t n = 0, in_b = 0, out_b = 0, sched = 0, stride = 0;
    const purlin_desc* table = NULL;
    uint64_t phase_begin[3];

    /* AllReduce, P = 8, bf16, 1 Mi elements per rank, chunk 64 KiB, host only */
    memset(&pol, 0, sizeof pol);
    pol.ar_mode = 1;
    pol.fanout = 1; /* one copy descriptor per destination */
    if (purlin_plan_ex(PURLIN_ALLREDUCE, 8, 1u << 20, PURLIN_BF16, 65536, &pol, PURLIN_PLAN_HOST_ONLY, &plan) != PURLIN_OK)
        return fail("plan");
    if (purlin_plan_info(plan, &n, &in_b, &out_b, &sched) != PURLIN_OK) return fail("info");
    if (in_b != (1u << 21) || out_b != (1u << 21)) return fail("bytes per rank");
    if (purlin_plan_descriptors(plan, &table, &n, &stride) != PURLIN_OK) return fail("descriptors");
    if (stride != sizeof(purlin_desc) || sizeof(purlin_desc) != 64) return fail("descriptor size");
    /* compose<ReduceScatter, AllGather>: 8 partitions x 4 chunks reduced, then copied to the 7 other ranks */
    if (n != 32 + 32 * 7) return fail("descriptor count");
    if (table[0].kind != PURLIN_KIND_REDUCE || table[0].nsrc != 8) return fail("first descriptor");
    if (purlin_plan_items(plan, &table, &n, phase_begin) != PURLIN_OK) return fail("items");
    if (phase_begin[2] != n || phase_begin[0] != 0 || phase_begin[1] == 0) return fail("phases");
    if (purlin_exec(plan, NULL, NULL) != PURLIN_ERR_INVALID) return fail("exec of a host-only plan");
    purlin_plan_destroy(plan);
    purlin_plan_destroy(NULL);

    /* errors leave *out_plan NULL */
    plan = (purlin_plan_t)0x1;
    if (purlin_plan_ex(PURLIN_ALLREDUCE, 3, 1000, PURLIN_BF16, 64, NULL, PURLIN_PLAN_HOST_ONLY, &plan) !=
        PURLIN_ERR_INVALID || plan != NULL)
        return fail("count not a multiple of P");
    if (purlin_plan_v(PURLIN_ALLTOALLV, 4, 100, 400, PURLIN_FP32, 64, 1, NULL,
                      PURLIN_PLAN_HOST_ONLY | PURLIN_PLAN_COUNTS_TRANSPOSED, &plan) != PURLIN_OK)
        return fail("v plan");
    purlin_plan_destroy(plan);
    if (purlin_plan_v(PURLIN_ALLGATHERV, 4, 100, 400, PURLIN_FP32, 64, 1, NULL,
                      PURLIN_PLAN_HOST_ONLY | PURLIN_PLAN_COUNTS_TRANSPOSED, &plan) != PURLIN_ERR_INVALID)
        return fail("transposed counts on a non-AllToAllV plan");
    /* rank 3's share of a ReduceScatter: partition 3's four 64 KiB chunks, reduced into out_3 */
    if (purlin_plan_share(PURLIN_REDUCE_SCATTER, 8, -1, 3, 1u << 20, PURLIN_BF16, 65536, NULL, PURLIN_PLAN_HOST_ONLY,
                          &plan) != PURLIN_OK)
        return fail("share plan");
    if (purlin_plan_descriptors(plan, &table, &n, &stride) != PURLIN_OK || n != 4) return fail("share descriptors");
    if (table[0].dst_buf != 8 + 3 || table[0].ndst != 1 || table[0].nsrc != 8) return fail("share destination");
    purlin_plan_destroy(plan);
    if (purlin_plan_rooted(PURLIN_BROADCAST, 4, 4, 64, PURLIN_FP32, 64, NULL, PURLIN_PLAN_HOST_ONLY, &plan) !=
        PURLIN_ERR_INVALID)
        return fail("root out of range");
    {
        uint64_t ws = 0;
        if (purlin_pack_workspace_size(4096, 8, 256, &ws) != PURLIN_OK || ws == 0) return fail("pack workspace");
        if (purlin_pack_dedup_workspace_size(4096, 8, &ws) != PURLIN_OK || ws == 0) return fail("dedup workspace");
    }
    if (strcmp(purlin_status_string(PURLIN_OK), "ok") != 0) return fail("status string");
    printf("OK %s\n", purlin_version());
    return 0;
}
"""


def test_header_compiles_as_c99_and_the_library_links(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    lib = PL.LIB_PATH
    assert os.path.exists(lib), "library not built"
    src = tmp_path / "abi.c"
    src.write_text(C_SOURCE)
    exe = tmp_path / "abi"
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(ROOT, "include"), str(src),
           lib, "-Wl,-rpath," + os.path.dirname(lib), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.startswith("OK"), r.stdout + r.stderr
