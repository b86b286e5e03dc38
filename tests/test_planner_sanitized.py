"""The host planner under AddressSanitizer and UndefinedBehaviorSanitizer.

The planner (csrc/plan.cpp) has no HIP dependency, so it is built here with
g++ and the sanitizers (host code only) together with a small C++ driver
that plans every op over many shapes, policies and invalid arguments, and
checks that every descriptor stays inside the buffers it names.  Any memory
error, overflow or undefined behaviour aborts the driver."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_36954_amd", "csrc")

DRIVER = r"""
#include <cstdio>
#include <algorithm>
#include <cstdlib>
#include "plan.h"

using namespace purlin;

static int checked = 0;

static void check_bounds(const Plan& p) {
    const uint64_t P = uint64_t(p.P);
    for (const purlin_desc& d : p.items) {
        for (uint32_t j = 0; j < d.nsrc; ++j) {
            const uint64_t b = uint64_t(d.src_buf) + uint64_t(j) * d.src_step;
            if (b >= 2 * P) { std::printf("source buffer %llu out of range\n", (unsigned long long)b); std::abort(); }
            const uint64_t cap = b < P ? p.in_bytes : p.out_bytes;
            if (d.src_off + d.bytes > cap) { std::printf("source range beyond its buffer\n"); std::abort(); }
        }
        for (uint32_t j = 0; j < d.ndst; ++j) {
            const uint64_t b = uint64_t(d.dst_buf) + uint64_t(j) * d.dst_step;
            if (b < P || b >= 2 * P) { std::printf("destination buffer %llu out of range\n", (unsigned long long)b); std::abort(); }
            if (d.dst_off + d.bytes > p.out_bytes) { std::printf("destination range beyond its buffer\n"); std::abort(); }
        }
    }
    ++checked;
}

int main() {
    const purlin_op fixed[] = {PURLIN_ALLREDUCE, PURLIN_REDUCE_SCATTER, PURLIN_ALLGATHER, PURLIN_ALLTOALL};
    const purlin_op rooted[] = {PURLIN_BROADCAST, PURLIN_REDUCE, PURLIN_SCATTER, PURLIN_GATHER};
    const purlin_op vops[] = {PURLIN_ALLGATHERV, PURLIN_REDUCE_SCATTERV, PURLIN_ALLTOALLV};
    const int Ps[] = {1, 2, 3, 8, 16};
    const uint64_t Ms[] = {0, 1, 7, 64, 1000, 65536};
    const uint64_t chunks[] = {2, 4, 96, 4096, 1u << 20};
    for (purlin_op op : fixed)
        for (int P : Ps)
            for (uint64_t M : Ms)
                for (uint64_t c : chunks)
                    for (int dt = 0; dt < 2; ++dt) {
                        const uint64_t per_part = (M * (dt ? 2 : 4) + c - 1) / c;  // chunks per partition
                        if (per_part * uint64_t(P) * uint64_t(P) > 20000) continue;  // keep the run short
                        for (uint32_t mode = 0; mode <= 3; ++mode)
                            for (uint32_t fan = 0; fan <= 2; ++fan) {
                                purlin_policy pol{};
                                pol.ar_mode = mode;
                                pol.fanout = fan;
                                pol.item_bytes = (mode + fan) % 2 ? 256 : 0;
                                Plan p;
                                const purlin_status st = build_plan(op, P, -1, M * uint64_t(P), purlin_dtype(dt), c, &pol,
                                                                    PURLIN_PLAN_HOST_ONLY, p);
                                if (st == PURLIN_OK) check_bounds(p);
                            }
                    }
    for (purlin_op op : rooted)
        for (int P : Ps)
            for (uint64_t M : Ms)
                for (int root = -1; root <= P; ++root) {
                    Plan p;
                    if (build_plan(op, P, root, M * uint64_t(P), PURLIN_BF16, 512, nullptr, PURLIN_PLAN_HOST_ONLY, p) ==
                        PURLIN_OK)
                        check_bounds(p);
                }
    for (purlin_op op : fixed)
        for (int P : Ps)
            for (int share = -1; share <= P; ++share)
                for (uint32_t mode = 0; mode <= 3; ++mode) {
                    purlin_policy pol{};
                    pol.ar_mode = mode;
                    Plan p;
                    if (build_plan(op, P, -1, 1000 * uint64_t(P), PURLIN_BF16, 96, &pol, PURLIN_PLAN_HOST_ONLY, p,
                                   share) == PURLIN_OK) {
                        check_bounds(p);
                        for (const purlin_desc& d : p.items)
                            if (share >= 0 && (d.ndst != 1 || d.dst_buf != uint32_t(P + share))) {
                                std::printf("a share writes another rank's output\n");
                                std::abort();
                            }
                    }
                }
    for (purlin_op op : rooted)
        for (int P : Ps)
            for (int share = 0; share < P; ++share) {
                Plan p;
                if (build_plan(op, P, P - 1, 64 * uint64_t(P), PURLIN_FP32, 32, nullptr, PURLIN_PLAN_HOST_ONLY, p,
                               share) == PURLIN_OK)
                    check_bounds(p);
            }
    for (purlin_op op : vops)
        for (int P : Ps)
            for (uint64_t in_cap : {uint64_t(0), uint64_t(5), uint64_t(1000), uint64_t(70000)})
                for (uint64_t out_cap : {uint64_t(0), uint64_t(3), uint64_t(1000), uint64_t(300000)})
                    for (uint64_t c : chunks) {
                        if ((std::max(in_cap, out_cap) * 4 + c - 1) / c * uint64_t(P) > 20000) continue;
                        Plan p;
                        const purlin_status st = build_plan_v(op, P, in_cap, out_cap, PURLIN_FP32, c, 1 + (c % 5),
                                                              nullptr, PURLIN_PLAN_HOST_ONLY, p);
                        if (st == PURLIN_OK) ++checked;
                    }
    // invalid arguments: every one must be rejected without touching anything
    Plan p;
    int rejected = 0;
    rejected += build_plan(purlin_op(99), 8, -1, 64, PURLIN_BF16, 64, nullptr, 0, p) != PURLIN_OK;
    rejected += build_plan(PURLIN_ALLREDUCE, 0, -1, 64, PURLIN_BF16, 64, nullptr, 0, p) != PURLIN_OK;
    rejected += build_plan(PURLIN_ALLREDUCE, 17, -1, 64, PURLIN_BF16, 64, nullptr, 0, p) != PURLIN_OK;
    rejected += build_plan(PURLIN_ALLREDUCE, 3, -1, 64, PURLIN_BF16, 64, nullptr, 0, p) != PURLIN_OK;
    rejected += build_plan(PURLIN_ALLREDUCE, 8, -1, 64, PURLIN_BF16, 3, nullptr, 0, p) != PURLIN_OK;
    rejected += build_plan(PURLIN_ALLREDUCE, 8, -1, ~uint64_t(0) - 7, PURLIN_BF16, 64, nullptr, 0, p) != PURLIN_OK;
    rejected += build_plan(PURLIN_ALLREDUCE, 8, -1, uint64_t(1) << 40, PURLIN_BF16, 2, nullptr, 0, p) != PURLIN_OK;
    rejected += build_plan_v(PURLIN_ALLTOALLV, 8, ~uint64_t(0), 64, PURLIN_BF16, 64, 1, nullptr, 0, p) != PURLIN_OK;
    rejected += build_plan_v(PURLIN_ALLGATHERV, 8, 64, 64, PURLIN_BF16, 64, 0, nullptr, 0, p) != PURLIN_OK;
    rejected += build_plan(PURLIN_ALLGATHER, 8, -1, 64, PURLIN_BF16, 64, nullptr, 0, p, 8) != PURLIN_OK;
    rejected += build_plan(PURLIN_ALLGATHER, 8, -1, 64, PURLIN_BF16, 64, nullptr, 0, p, -2) != PURLIN_OK;
    if (rejected != 11) { std::printf("an invalid plan was accepted\n"); return 1; }
    std::printf("OK %d plans\n", checked);
    return 0;
}
"""


def test_planner_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    drv = tmp_path / "driver.cpp"
    drv.write_text(DRIVER)
    exe = tmp_path / "planner_asan"
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "plan.cpp"), str(drv), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "sanitizer" in r.stderr.lower() and "cannot find" in r.stderr.lower():
        pytest.skip("sanitizer runtime not installed")
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600, env=env)
    assert r.returncode == 0 and r.stdout.startswith("OK"), (r.stdout + r.stderr)[-4000:]
