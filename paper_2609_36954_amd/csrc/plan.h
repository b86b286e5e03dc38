// Internal plan object shared by the planner (plan.cpp, host only) and the
// ABI glue (abi.hip).  Not part of the public ABI.
#pragma once

#include <cstdint>
#include <vector>

#include "purlin.h"

namespace purlin {

// One kernel launch of a plan: every work item of a phase has the same
// consume op and, for REDUCE, the same source count.
struct Phase {
    uint32_t kind = PURLIN_KIND_COPY;
    uint32_t nsrc = 1;
    uint32_t src_buf = 0;   // REDUCE phases: every item sums bufs[src_buf + p * src_step]
    uint32_t src_step = 0;
    bool nt_load = false;   // non-temporal (streaming) global loads
    bool nt_store = false;  // non-temporal (streaming) global stores
    uint64_t begin = 0;  // first work item
    uint64_t count = 0;  // work items
};

struct Plan {
    purlin_op op{};
    int P = 0;
    uint64_t count = 0;
    purlin_dtype dtype{};
    uint64_t chunk = 0;
    purlin_policy policy{};  // resolved: no "auto" fields left
    uint32_t flags = 0;

    int root = -1;           // rooted collectives only
    int share = -1;          // rank whose share this plan is, or -1 for all ranks' work
    uint32_t in_mask = 0;    // bit p: input p is read
    uint32_t out_mask = 0;   // bit r: output r is written
    uint64_t elem_bytes = 0;
    uint64_t in_bytes = 0;   // per rank
    uint64_t out_bytes = 0;  // per rank
    uint64_t sched_bytes = 0;

    std::vector<purlin_desc> descs;  // chunk descriptors
    std::vector<purlin_desc> items;  // work items (descriptors cut at item_bytes)
    int nphases = 0;
    Phase phases[2];

    // Variable-size collectives: capacities in elements, counts' unit.
    bool vop = false;
    uint64_t in_capacity = 0;
    uint64_t out_capacity = 0;
    uint64_t unit = 1;
    bool v_src_major = false;  // ALLTOALLV: descriptors cover each source's input

    // Single-launch AllReduce (ar_mode 3): one launch over all items.
    bool fused = false;
    uint64_t part_bytes = 0;
    uint64_t chunks_per_part = 0;
    uint64_t reduce_item_bytes = 0;  // cut size of the reduce items

    purlin_desc* d_items = nullptr;  // device copy of items (null for host-only plans)
    void* d_state = nullptr;         // fused plans: FusedState followed by the per-chunk counters
};

// Validates the request and fills `out` (host tables only).  Pure host code.
// Variable-size collectives (ALLGATHERV, REDUCE_SCATTERV, ALLTOALLV): the
// table covers a virtual index space: the gathered output (out_capacity),
// the partitioned input (in_capacity) or each destination's output
// (out_capacity); sizes are applied on the device.
purlin_status build_plan_v(purlin_op op, int P, uint64_t in_capacity, uint64_t out_capacity, purlin_dtype dtype,
                           uint64_t chunk, uint64_t unit, const purlin_policy* policy, uint32_t flags, Plan& out);

// `root` is -1 for the non-rooted collectives and a rank for the rooted ones.
// `share` >= 0 keeps only that rank's share of the work: the descriptors that
// write its output, each narrowed to that one destination (every rank pulls
// what it consumes).
purlin_status build_plan(purlin_op op, int P, int root, uint64_t count, purlin_dtype dtype, uint64_t chunk,
                         const purlin_policy* policy, uint32_t flags, Plan& out, int share = -1);

}  // namespace purlin
