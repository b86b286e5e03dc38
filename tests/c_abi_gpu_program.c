/* A plain C program that drives the library through include/purlin.h and
 * the HIP runtime's C API only (no Python, no torch): the GPU leg of the
 * boundary tests.  It reads jobs from stdin, one per line,
 *
 *   coll <op> <P> <count> <dtype> <chunk_bytes> <prefix>
 *       reads <prefix>in<p>.bin (P files of the plan's input bytes), plans,
 *       executes on a stream of its own, writes <prefix>out<r>.bin
 *   moe <T> <H> <K> <E> <P> <prefix>
 *       reads <prefix>x.bin (bf16 [T,H]), <prefix>ids.bin (int32 [T,K]),
 *       <prefix>y.bin (bf16 [T*K,H]) and <prefix>g.bin (fp32 [T,K]); runs
 *       purlin_pack on x and purlin_unpack on y with pack's positions;
 *       writes <prefix>packed.bin, <prefix>pos.bin, <prefix>meta.bin
 *       (dest_counts, dest_offsets, expert_counts, expert_offsets, status)
 *       and <prefix>out.bin
 *
 * and prints "ok" when every job ran.  Any failing call prints the call and
 * its status and exits with 1. */

#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "purlin.h"

#define HIP_OK(call)                                                        \
    do {                                                                    \
        hipError_t e_ = (call);                                             \
        if (e_ != hipSuccess) {                                             \
            fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));      \
            exit(1);                                                        \
        }                                                                   \
    } while (0)

#define PURLIN_OK_(call)                                                    \
    do {                                                                    \
        purlin_status s_ = (call);                                          \
        if (s_ != PURLIN_OK) {                                              \
            fprintf(stderr, "%s: %s\n", #call, purlin_status_string(s_));   \
            exit(1);                                                        \
        }                                                                   \
    } while (0)

static void* read_file(const char* path, size_t bytes) {
    FILE* f = fopen(path, "rb");
    void* buf = malloc(bytes ? bytes : 1);
    if (!f || !buf || fread(buf, 1, bytes, f) != bytes) {
        fprintf(stderr, "cannot read %zu bytes from %s\n", bytes, path);
        exit(1);
    }
    fclose(f);
    return buf;
}

static void write_file(const char* path, const void* buf, size_t bytes) {
    FILE* f = fopen(path, "wb");
    if (!f || fwrite(buf, 1, bytes, f) != bytes) {
        fprintf(stderr, "cannot write %s\n", path);
        exit(1);
    }
    fclose(f);
}

static void* to_device(const char* path, size_t bytes) {
    void* host = read_file(path, bytes);
    void* dev = NULL;
    HIP_OK(hipMalloc(&dev, bytes ? bytes : 16));
    if (bytes) HIP_OK(hipMemcpy(dev, host, bytes, hipMemcpyHostToDevice));
    free(host);
    return dev;
}

static void to_file(const char* path, const void* dev, size_t bytes) {
    void* host = malloc(bytes ? bytes : 1);
    if (!host) exit(1);
    if (bytes) HIP_OK(hipMemcpy(host, dev, bytes, hipMemcpyDeviceToHost));
    write_file(path, host, bytes);
    free(host);
}

static int op_of(const char* name) {
    static const char* names[] = {"allreduce", "reduce_scatter", "allgather", "alltoall"};
    for (int i = 0; i < 4; ++i)
        if (strcmp(name, names[i]) == 0) return i;
    fprintf(stderr, "unknown op %s\n", name);
    exit(1);
}

static void run_collective(const char* op, int P, unsigned long long count, const char* dtype,
                           unsigned long long chunk, const char* prefix, hipStream_t stream) {
    purlin_plan_t plan = NULL;
    uint64_t n = 0, in_b = 0, out_b = 0, sched = 0;
    void* bufs[2 * PURLIN_MAX_RANKS];
    char path[4096];
    PURLIN_OK_(purlin_plan((purlin_op)op_of(op), P, count, strcmp(dtype, "bf16") == 0 ? PURLIN_BF16 : PURLIN_FP32,
                           chunk, &plan));
    PURLIN_OK_(purlin_plan_info(plan, &n, &in_b, &out_b, &sched));
    for (int p = 0; p < P; ++p) {
        snprintf(path, sizeof path, "%sin%d.bin", prefix, p);
        bufs[p] = to_device(path, in_b);
        HIP_OK(hipMalloc(&bufs[P + p], out_b ? out_b : 16));
        HIP_OK(hipMemset(bufs[P + p], 0xA5, out_b ? out_b : 16));
    }
    PURLIN_OK_(purlin_exec(plan, bufs, stream));
    HIP_OK(hipStreamSynchronize(stream));
    for (int r = 0; r < P; ++r) {
        snprintf(path, sizeof path, "%sout%d.bin", prefix, r);
        to_file(path, bufs[P + r], out_b);
    }
    for (int i = 0; i < 2 * P; ++i) HIP_OK(hipFree(bufs[i]));
    purlin_plan_destroy(plan);
}

static void run_moe(int T, int H, int K, int E, int P, const char* prefix, hipStream_t stream) {
    char path[4096];
    const size_t xb = (size_t)T * H * 2, ib = (size_t)T * K * 4;
    uint64_t wsb = 0;
    void *x, *ids, *y, *g, *packed, *pos, *out, *ws;
    int32_t *dest_counts, *dest_offsets, *expert_counts, *expert_offsets, *status;
    snprintf(path, sizeof path, "%sx.bin", prefix);
    x = to_device(path, xb);
    snprintf(path, sizeof path, "%sids.bin", prefix);
    ids = to_device(path, ib);
    snprintf(path, sizeof path, "%sy.bin", prefix);
    y = to_device(path, xb * K);
    snprintf(path, sizeof path, "%sg.bin", prefix);
    g = to_device(path, ib);
    HIP_OK(hipMalloc(&packed, xb * K + 16));
    HIP_OK(hipMalloc(&pos, ib + 16));
    HIP_OK(hipMalloc(&out, xb + 16));
    /* hipMalloc returns 256-byte aligned memory: every array meets the 16-byte rule */
    HIP_OK(hipMalloc((void**)&dest_counts, (size_t)P * 4));
    HIP_OK(hipMalloc((void**)&dest_offsets, (size_t)P * 4));
    HIP_OK(hipMalloc((void**)&expert_counts, (size_t)E * 4));
    HIP_OK(hipMalloc((void**)&expert_offsets, (size_t)E * 4));
    HIP_OK(hipMalloc((void**)&status, 4));
    PURLIN_OK_(purlin_pack_workspace_size(T, K, E, &wsb));
    HIP_OK(hipMalloc(&ws, wsb ? wsb : 16));
    PURLIN_OK_(purlin_pack(T, H, K, E, P, x, (const int32_t*)ids, packed, dest_counts, dest_offsets, expert_counts,
                           expert_offsets, (int32_t*)pos, status, ws, wsb, stream));
    PURLIN_OK_(purlin_unpack(T, H, K, y, (const int32_t*)pos, (const float*)g, out, NULL, stream));
    HIP_OK(hipStreamSynchronize(stream));
    snprintf(path, sizeof path, "%spacked.bin", prefix);
    to_file(path, packed, xb * K);
    snprintf(path, sizeof path, "%spos.bin", prefix);
    to_file(path, pos, ib);
    snprintf(path, sizeof path, "%sout.bin", prefix);
    to_file(path, out, xb);
    {
        int32_t* host = (int32_t*)malloc((size_t)(2 * P + 2 * E + 1) * 4);
        if (!host) exit(1);
        HIP_OK(hipMemcpy(host, dest_counts, (size_t)P * 4, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(host + P, dest_offsets, (size_t)P * 4, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(host + 2 * P, expert_counts, (size_t)E * 4, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(host + 2 * P + E, expert_offsets, (size_t)E * 4, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(host + 2 * P + 2 * E, status, 4, hipMemcpyDeviceToHost));
        snprintf(path, sizeof path, "%smeta.bin", prefix);
        write_file(path, host, (size_t)(2 * P + 2 * E + 1) * 4);
        free(host);
    }
    void* all[] = {x, ids, y, g, packed, pos, out, ws, dest_counts, dest_offsets, expert_counts, expert_offsets, status};
    for (size_t i = 0; i < sizeof all / sizeof all[0]; ++i) HIP_OK(hipFree(all[i]));
}

int main(void) {
    char line[8192], kind[32], a[64], d[16], prefix[4096];
    hipStream_t stream;
    HIP_OK(hipStreamCreate(&stream));
    while (fgets(line, sizeof line, stdin)) {
        if (sscanf(line, "%31s", kind) != 1) continue;
        if (strcmp(kind, "coll") == 0) {
            int P;
            unsigned long long count, chunk;
            if (sscanf(line, "coll %63s %d %llu %15s %llu %4095s", a, &P, &count, d, &chunk, prefix) != 6) return 2;
            run_collective(a, P, count, d, chunk, prefix, stream);
        } else if (strcmp(kind, "moe") == 0) {
            int T, H, K, E, P;
            if (sscanf(line, "moe %d %d %d %d %d %4095s", &T, &H, &K, &E, &P, prefix) != 6) return 2;
            run_moe(T, H, K, E, P, prefix, stream);
        } else {
            return 2;
        }
    }
    HIP_OK(hipStreamDestroy(stream));
    printf("ok\n");
    return 0;
}
