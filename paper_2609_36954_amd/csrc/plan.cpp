// Host orchestrator: (op, P, count, dtype, chunk) -> chunk descriptors ->
// wavefront work items.  Pure host C++ (no HIP), so it runs and is tested
// on machines without a GPU.
//
// Paper passages (Purlin, arXiv 2609.36954):
//  - Section 3.1 / Listing 1: each collective is a consume op (copy or
//    reduce) between an input and an output layout; AllReduce is
//    compose<ReduceScatter, AllGather>, the AllGather consuming the
//    ReduceScatter result in place.
//  - Section 3.2 / Listing 2: work proceeds per chunk of a partition; a
//    packed output is addressed dst + offset, a scattered or transposed
//    output dst + peer * partBytes + offset; reduce consumes the chunk of
//    every rank, copy consumes one peer's chunk.
//  - Section 3.3, Eq. 3: throughput needs enough bytes in flight; here the
//    policy cuts descriptors into work items so that a launch has thousands
//    of independent wavefronts.

#include "plan.h"

#include <algorithm>
#include <new>

namespace purlin {
namespace {

constexpr uint64_t kMinItem = 1024;        // one 16-byte access per lane of a 64-wide wave
constexpr uint64_t kMaxItem = 64 * 1024;   // largest automatic work item
constexpr uint64_t kTargetItems = 4096;    // 16 wavefronts per CU on 256 CUs
// Traffic of a launch from which streaming item sizes and non-temporal hints
// win (measured on MI355X, P = 8: between 288 MiB, where cached accesses are
// faster, and 360 MiB, where they are 10-35% slower).
constexpr uint64_t kStreamingBytes = 320ull << 20;
constexpr uint64_t kAllReduceTwoPhaseBytes = 1ull << 30;  // one-phase traffic from which compose<RS, AG> wins
constexpr uint64_t kLastLevelCacheBytes = 256ull << 20;    // MI355X Infinity Cache (256 MB)
constexpr uint64_t kLargeCopyBytes = 4ull << 30;           // copy-phase traffic from which 2 KiB items win
constexpr uint64_t kLatencyNtStoreMin = 8ull << 20;  // written bytes per launch between which
constexpr uint64_t kLatencyNtStoreMax = 32ull << 20; // non-temporal stores win below streaming

uint64_t ceil_div(uint64_t a, uint64_t b) { return (a + b - 1) / b; }

uint64_t pow2_floor(uint64_t v) {
    uint64_t p = 1;
    while (p <= v / 2) p <<= 1;
    return p;
}

purlin_desc make_desc(uint32_t kind, uint32_t phase, uint32_t nsrc, uint32_t src_buf, uint32_t src_step,
                      uint32_t ndst, uint32_t dst_buf, uint32_t dst_step, uint64_t src_off, uint64_t dst_off,
                      uint64_t bytes, uint32_t part, uint32_t chunk) {
    purlin_desc d{};
    d.kind = kind;
    d.phase = phase;
    d.nsrc = nsrc;
    d.src_buf = src_buf;
    d.src_step = src_step;
    d.ndst = ndst;
    d.dst_buf = dst_buf;
    d.dst_step = dst_step;
    d.src_off = src_off;
    d.dst_off = dst_off;
    d.bytes = bytes;
    d.part = part;
    d.chunk = chunk;
    return d;
}

// Automatic work-item size for one phase.
//  - Phases that stream more than the last-level cache holds: a wave's
//    share is sized by the bytes it moves.  Measured on MI355X (256 MiB
//    per rank, P = 8): a reduce item reading ~32 KiB (4 KiB of output from
//    each of 8 sources), a multi-destination copy item writing ~256 KiB
//    (32 KiB to each of 8 destinations) and a one-to-one copy item of 4 KiB
//    run fastest; larger items leave too few wavefronts, smaller ones pay
//    per-item overhead.
//  - Copy phases that move 4 GiB or more (at P = 8: AllGather from
//    512 MiB per rank, AllToAll from 256 MiB): 2 KiB items, measured 3-6%
//    faster than the sizes above from 512 MiB per rank (and 10% slower for
//    AllGather at 256 MiB).  The waves in flight
//    then cover a narrower span of every destination buffer at a time.
//    Variable-size plans keep the sizes above: their waves also map each
//    item onto the run-time sizes, and 2 KiB items made the AllToAllV
//    exchanges 18-50% slower.
//  - Smaller phases (latency regime): aim at kTargetItems items of at
//    least one wave-wide 16-byte access per lane, one-to-one copies at most
//    4 KiB.
// Never above kMaxItem, and large enough to keep the item count under
// PURLIN_MAX_ITEMS.
uint64_t auto_item_bytes(uint64_t phase_bytes, uint64_t traffic, uint32_t kind, uint32_t nsrc, uint32_t ndst,
                         bool variable) {
    uint64_t item;
    if (traffic >= kStreamingBytes) {
        if (kind == PURLIN_KIND_REDUCE)
            item = pow2_floor(std::max<uint64_t>(1, (32 * 1024) / std::max<uint32_t>(1, nsrc)));
        else if (traffic >= kLargeCopyBytes && !variable)
            item = 2048;
        else if (ndst > 1)
            item = std::min<uint64_t>(32 * 1024, pow2_floor(std::max<uint64_t>(1, (256 * 1024) / ndst)));
        else
            item = 4096;  // one-to-one copies: many small items (AllToAll measured best at 4 KiB)
        item = std::max<uint64_t>(item, 2048);
    } else {
        item = pow2_floor(std::max<uint64_t>(1, phase_bytes / kTargetItems));
        // one-to-one copies keep their streaming size here too (Gather of
        // 128 MiB: 40.8 vs 45.0 µs with 32 KiB items; AllToAll of 16 MiB per
        // rank: 40.9 vs 42.6 µs; measured on MI355X, P = 8)
        if (kind == PURLIN_KIND_COPY && ndst == 1 && !variable) item = std::min<uint64_t>(item, 4096);
    }
    item = std::min(std::max(item, kMinItem), kMaxItem);
    const uint64_t floor_for_cap = ceil_div(phase_bytes, PURLIN_MAX_ITEMS / 2);
    if (item < floor_for_cap) item = ceil_div(floor_for_cap, 16) * 16;
    return item;
}

// Work-item size of a single-launch AllReduce (both of its phases): a
// quarter of a chunk, at most 32 KiB.  Every item claims a ticket, and a
// reduced chunk is published to its copies with write-through stores and a
// counter; measured on MI355X (P = 8, bf16), per call: at 256 MiB per rank
// 810 µs with 32 KiB items, 833 µs with 4 KiB and 1090 µs with quarter
// chunks of 256 KiB; at 128 x 8192 per rank (64 KiB chunks) 22.7 µs with
// quarter chunks, 26 µs with 4 KiB and 34 µs with 32 KiB items.
constexpr uint64_t kFusedMaxItem = 32 * 1024;
uint64_t fused_item_bytes(uint64_t chunk, uint64_t phase_bytes) {
    uint64_t item = std::max<uint64_t>(16, std::min(kFusedMaxItem, chunk / 4) / 16 * 16);
    const uint64_t floor_for_cap = ceil_div(phase_bytes, PURLIN_MAX_ITEMS / 2);
    if (item < floor_for_cap) item = ceil_div(floor_for_cap, 16) * 16;
    return item;
}

bool parse_policy(const purlin_policy* policy, purlin_policy& pol) {
    pol = purlin_policy{};
    if (!policy) return true;
    pol = *policy;
    if (pol.item_bytes % 16 != 0) return false;
    if (pol.fanout > 2 || pol.ar_mode > 3) return false;
    if (pol.load_hint > 2 || pol.store_hint > 2) return false;
    if (pol.copy_depth != 0 && pol.copy_depth != 1 && pol.copy_depth != 2 && pol.copy_depth != 4 &&
        pol.copy_depth != 8)
        return false;
    for (uint32_t r : pol.reserved)
        if (r != 0) return false;
    return true;
}

// Cuts out.descs into work items phase by phase, records the launches and
// resolves the cache hints.  Returns PURLIN_ERR_NOMEM past PURLIN_MAX_ITEMS
// or PURLIN_ERR_UNSUPPORTED if a phase mixes consume ops or source sets.
purlin_status cut_items(Plan& out, const purlin_policy& pol);

}  // namespace

purlin_status build_plan(purlin_op op, int P, int root, uint64_t count, purlin_dtype dtype, uint64_t chunk,
                         const purlin_policy* policy, uint32_t flags, Plan& out, int share) {
    if (op < PURLIN_ALLREDUCE || op > PURLIN_GATHER) return PURLIN_ERR_INVALID;
    const bool rooted = op >= PURLIN_BROADCAST;
    if (dtype != PURLIN_FP32 && dtype != PURLIN_BF16) return PURLIN_ERR_INVALID;
    if (P < 1 || P > PURLIN_MAX_RANKS) return PURLIN_ERR_INVALID;
    if (rooted ? (root < 0 || root >= P) : root != -1) return PURLIN_ERR_INVALID;
    if (share < -1 || share >= P) return PURLIN_ERR_INVALID;
    if (count % static_cast<uint64_t>(P) != 0) return PURLIN_ERR_INVALID;
    if (flags & ~(PURLIN_PLAN_HOST_ONLY | PURLIN_PLAN_SHARE_PUSH)) return PURLIN_ERR_INVALID;
    const bool push = (flags & PURLIN_PLAN_SHARE_PUSH) != 0;
    if (push && share < 0) return PURLIN_ERR_INVALID;
    if (push && (op == PURLIN_ALLREDUCE || op == PURLIN_REDUCE_SCATTER || op == PURLIN_REDUCE))
        return PURLIN_ERR_UNSUPPORTED;
    const uint64_t s = dtype == PURLIN_FP32 ? 4 : 2;
    if (chunk < s || chunk % s != 0) return PURLIN_ERR_INVALID;
    if (count > (uint64_t(1) << 58) / s) return PURLIN_ERR_INVALID;

    purlin_policy pol{};
    if (!parse_policy(policy, pol)) return PURLIN_ERR_INVALID;
    const uint64_t M = count / P;       // elements per partition
    const uint64_t part = M * s;        // partBytes
    const uint64_t Cp = part ? ceil_div(part, chunk) : 0;

    if (pol.fanout == 0) pol.fanout = 2;
    if (pol.copy_depth == 0) {
        // Copies keep 4 loads per lane in flight; on a grid capped at a
        // quarter or less of the CUs, 8 (measured on MI355X, AllGather at
        // 256 MiB/rank: 1.88 vs 1.77 TB/s on 16 workgroups, 5.12 vs 4.86 on
        // 64; 6.39 vs 6.11 uncapped with 4).
        pol.copy_depth = pol.max_workgroups && pol.max_workgroups <= 128 ? 8 : 4;
    }
    if (pol.max_workgroups && op == PURLIN_ALLREDUCE && pol.ar_mode == 3) return PURLIN_ERR_UNSUPPORTED;
    if (share >= 0 && op == PURLIN_ALLREDUCE) {
        // A rank's share of an AllReduce is its ReduceScatter partition and
        // the pulls of the others (compose<RS, AG>); the one-phase form would
        // have every rank reduce the whole buffer, and the single-launch form
        // coordinates ranks through counters in one GPU's memory.
        if (pol.ar_mode == 0) pol.ar_mode = 1;
        if (pol.ar_mode == 3) return PURLIN_ERR_UNSUPPORTED;
    }
    if (pol.ar_mode == 0) {
        // AllReduce: up to 48 MiB per rank (P = 8) one launch that reduces
        // each chunk once and writes it to all P outputs wins (no second
        // launch; 82 vs 128 µs at 32 MiB, 150 vs 196 µs at 48 MiB).  From
        // 64 MiB per rank the two-phase compose wins although it schedules
        // more bytes: phase 0 leaves the N*s reduced bytes in the last-level
        // cache and phase 1's copies read them back from there, while each
        // wave streams one direction at a time (744 vs 801 µs at 256 MiB).
        // Once those bytes no longer fit that cache, phase 1 reads them from
        // HBM and the one-phase form is ahead again (1662 vs 1677 µs at
        // 512 MiB per rank, 3299 vs 3372 µs at 1 GiB; measured on MI355X).
        const uint64_t one_phase_traffic = 2 * uint64_t(P) * count * s;
        const bool reduced_fits_cache = count * s <= kLastLevelCacheBytes;
        pol.ar_mode = one_phase_traffic >= kAllReduceTwoPhaseBytes && reduced_fits_cache ? 1 : 2;
    }

    out = Plan{};
    out.op = op;
    out.P = P;
    out.count = count;
    out.dtype = dtype;
    out.chunk = chunk;
    out.flags = flags;
    out.elem_bytes = s;
    out.root = rooted ? root : -1;
    const uint32_t all = (P >= 32) ? 0xFFFFFFFFu : ((1u << P) - 1u);
    const uint32_t root_bit = rooted ? (1u << root) : 0u;
    out.in_mask = all;
    out.out_mask = all;
    switch (op) {
        case PURLIN_ALLREDUCE:
        case PURLIN_ALLTOALL:
        case PURLIN_BROADCAST:
        case PURLIN_REDUCE:
            out.in_bytes = count * s;
            out.out_bytes = count * s;
            break;
        case PURLIN_REDUCE_SCATTER:
        case PURLIN_SCATTER:
            out.in_bytes = count * s;
            out.out_bytes = part;
            break;
        case PURLIN_ALLGATHER:
        case PURLIN_GATHER:
            out.in_bytes = part;
            out.out_bytes = count * s;
            break;
        default:
            return PURLIN_ERR_INVALID;  // variable-size ops go through build_plan_v
    }
    if (op == PURLIN_BROADCAST || op == PURLIN_SCATTER) out.in_mask = root_bit;
    if (op == PURLIN_REDUCE || op == PURLIN_GATHER) out.out_mask = root_bit;

    // Upper bound on descriptors before allocating anything.
    const uint64_t Pu = static_cast<uint64_t>(P);
    if (Cp > PURLIN_MAX_ITEMS || Cp * Pu * Pu * 2 > PURLIN_MAX_ITEMS) return PURLIN_ERR_NOMEM;

    const uint32_t in0 = 0, out0 = static_cast<uint32_t>(P);
    try {
        std::vector<purlin_desc>& D = out.descs;
        auto for_chunks = [&](uint32_t k, auto&& emit) {
            for (uint64_t c = 0; c < Cp; ++c) {
                const uint64_t off = c * chunk;
                const uint64_t len = std::min(chunk, part - off);
                emit(static_cast<uint32_t>(c), k * part + off, off, len);
            }
        };
        switch (op) {
            case PURLIN_REDUCE_SCATTER:
                // reduce, scattered -> packed: partition k of every input,
                // summed in rank order, lands at out_k + offset.
                for (uint32_t k = 0; k < Pu; ++k)
                    for_chunks(k, [&](uint32_t c, uint64_t scat, uint64_t pk, uint64_t len) {
                        D.push_back(make_desc(PURLIN_KIND_REDUCE, 0, P, in0, 1, 1, out0 + k, 0, scat, pk, len, k, c));
                    });
                break;
            case PURLIN_ALLGATHER:
                // copy, packed -> scattered: peer k's contribution lands at
                // out_r + k * partBytes + offset for every consumer r.
                for (uint32_t k = 0; k < Pu; ++k)
                    for_chunks(k, [&](uint32_t c, uint64_t scat, uint64_t pk, uint64_t len) {
                        if (pol.fanout == 2) {
                            D.push_back(make_desc(PURLIN_KIND_COPY, 0, 1, in0 + k, 0, P, out0, 1, pk, scat, len, k, c));
                        } else {
                            for (uint32_t r = 0; r < Pu; ++r)
                                D.push_back(make_desc(PURLIN_KIND_COPY, 0, 1, in0 + k, 0, 1, out0 + r, 0, pk, scat, len, k, c));
                        }
                    });
                break;
            case PURLIN_ALLTOALL:
                // copy, scattered -> transposed: consumer r takes partition r
                // of peer p and places it at out_r + p * partBytes + offset.
                for (uint32_t r = 0; r < Pu; ++r)
                    for (uint32_t p = 0; p < Pu; ++p)
                        for_chunks(r, [&](uint32_t c, uint64_t scat, uint64_t pk, uint64_t len) {
                            D.push_back(make_desc(PURLIN_KIND_COPY, 0, 1, in0 + p, 0, 1, out0 + r, 0, scat, p * part + pk, len, r, c));
                        });
                break;
            case PURLIN_BROADCAST:
                // compose<scatter, allGather> with the intermediate in
                // registers: each chunk of the root's partition k is read
                // once and written to every rank's partition k.
                for (uint32_t k = 0; k < Pu; ++k)
                    for_chunks(k, [&](uint32_t c, uint64_t scat, uint64_t, uint64_t len) {
                        D.push_back(make_desc(PURLIN_KIND_COPY, 0, 1, in0 + root, 0, P, out0, 1, scat, scat, len, k, c));
                    });
                break;
            case PURLIN_SCATTER:
                // copy, scattered -> packed: partition k of the root's input
                // lands at out_k + offset.
                for (uint32_t k = 0; k < Pu; ++k)
                    for_chunks(k, [&](uint32_t c, uint64_t scat, uint64_t pk, uint64_t len) {
                        D.push_back(make_desc(PURLIN_KIND_COPY, 0, 1, in0 + root, 0, 1, out0 + k, 0, scat, pk, len, k, c));
                    });
                break;
            case PURLIN_GATHER:
                // copy, packed -> scattered: rank p's contribution lands at
                // out_root + p * partBytes + offset.
                for (uint32_t p = 0; p < Pu; ++p)
                    for_chunks(p, [&](uint32_t c, uint64_t scat, uint64_t pk, uint64_t len) {
                        D.push_back(make_desc(PURLIN_KIND_COPY, 0, 1, in0 + p, 0, 1, out0 + root, 0, pk, scat, len, p, c));
                    });
                break;
            case PURLIN_REDUCE:
                // compose<reduceScatter, gather> with the intermediate in
                // registers: partition k of every input, summed in rank
                // order, lands at out_root + k * partBytes + offset.
                for (uint32_t k = 0; k < Pu; ++k)
                    for_chunks(k, [&](uint32_t c, uint64_t scat, uint64_t, uint64_t len) {
                        D.push_back(make_desc(PURLIN_KIND_REDUCE, 0, P, in0, 1, 1, out0 + root, 0, scat, scat, len, k, c));
                    });
                break;
            case PURLIN_ALLREDUCE:
                if (pol.ar_mode == 1 || pol.ar_mode == 3) {
                    // compose<ReduceScatter, AllGather> in place: phase 0
                    // reduces partition k into out_k's k-th partition (the
                    // intermediate Y_k), phase 1 copies it to every other rank.
                    for (uint32_t k = 0; k < Pu; ++k)
                        for_chunks(k, [&](uint32_t c, uint64_t scat, uint64_t, uint64_t len) {
                            D.push_back(make_desc(PURLIN_KIND_REDUCE, 0, P, in0, 1, 1, out0 + k, 0, scat, scat, len, k, c));
                        });
                    for (uint32_t k = 0; k < Pu; ++k)
                        for_chunks(k, [&](uint32_t c, uint64_t scat, uint64_t, uint64_t len) {
                            if (pol.fanout == 2) {
                                if (k > 0)
                                    D.push_back(make_desc(PURLIN_KIND_COPY, 1, 1, out0 + k, 0, k, out0, 1, scat, scat, len, k, c));
                                if (k + 1 < Pu)
                                    D.push_back(make_desc(PURLIN_KIND_COPY, 1, 1, out0 + k, 0, P - 1 - k, out0 + k + 1, 1,
                                                          scat, scat, len, k, c));
                            } else {
                                for (uint32_t r = 0; r < Pu; ++r)
                                    if (r != k)
                                        D.push_back(make_desc(PURLIN_KIND_COPY, 1, 1, out0 + k, 0, 1, out0 + r, 0, scat, scat, len, k, c));
                            }
                        });
                } else {
                    // One phase: each chunk of partition k is reduced once
                    // and written to every rank's output.
                    for (uint32_t k = 0; k < Pu; ++k)
                        for_chunks(k, [&](uint32_t c, uint64_t scat, uint64_t, uint64_t len) {
                            D.push_back(make_desc(PURLIN_KIND_REDUCE, 0, P, in0, 1, P, out0, 1, scat, scat, len, k, c));
                        });
                }
                break;
            default:
                return PURLIN_ERR_INVALID;
        }
        if (share >= 0 && push) {
            // Keep the copies that read in_share, as they are.
            std::vector<purlin_desc> kept;
            uint32_t out_mask = 0;
            for (const purlin_desc& d : D) {
                if (d.kind != PURLIN_KIND_COPY || d.nsrc != 1 || d.src_buf != in0 + static_cast<uint32_t>(share))
                    continue;
                for (uint32_t j = 0; j < d.ndst; ++j) out_mask |= 1u << (d.dst_buf + j * d.dst_step - out0);
                kept.push_back(d);
            }
            D.swap(kept);
            out.in_mask = D.empty() ? 0u : 1u << share;
            out.out_mask = out_mask;
            out.share = share;
        } else if (share >= 0) {
            // Keep what writes out_share, narrowed to that destination; the
            // buffer masks become the buffers the share reads or writes.
            const uint32_t mine = out0 + static_cast<uint32_t>(share);
            std::vector<purlin_desc> kept;
            uint32_t in_mask = 0, out_mask = 0;
            for (const purlin_desc& d : D) {
                bool writes = false;
                for (uint32_t j = 0; j < d.ndst; ++j) writes = writes || d.dst_buf + j * d.dst_step == mine;
                if (!writes) continue;
                purlin_desc n = d;
                n.ndst = 1;
                n.dst_buf = mine;
                n.dst_step = 0;
                for (uint32_t j = 0; j < n.nsrc; ++j) {
                    const uint32_t b = n.src_buf + j * n.src_step;
                    if (b < out0)
                        in_mask |= 1u << b;
                    else
                        out_mask |= 1u << (b - out0);
                }
                out_mask |= 1u << share;
                kept.push_back(n);
            }
            D.swap(kept);
            out.in_mask = in_mask;
            out.out_mask = out_mask;
            out.share = share;
        }
        out.policy = pol;
        out.part_bytes = part;
        out.chunks_per_part = Cp;
        out.fused = op == PURLIN_ALLREDUCE && pol.ar_mode == 3 && P > 1;

        const purlin_status st = cut_items(out, pol);
        if (st != PURLIN_OK) return st;
    } catch (const std::bad_alloc&) {
        out.descs.clear();
        out.items.clear();
        return PURLIN_ERR_NOMEM;
    }
    return PURLIN_OK;
}

namespace {

purlin_status cut_items(Plan& out, const purlin_policy& pol) {
    for (const purlin_desc& d : out.descs) out.sched_bytes += (uint64_t(d.nsrc) + d.ndst) * d.bytes;

    // Per-phase shape: bytes of the descriptors, bytes moved, fan-in/out.
    struct PhaseShape {
        uint64_t bytes = 0, traffic = 0, ndesc = 0;
        uint32_t kind = 0, nsrc = 0, ndst = 0;
        uint64_t item = 0;
    } shape[2];
    for (const purlin_desc& d : out.descs) {
        PhaseShape& sh = shape[d.phase];
        sh.bytes += d.bytes;
        sh.traffic += (uint64_t(d.nsrc) + d.ndst) * d.bytes;
        sh.kind = d.kind;
        sh.nsrc = std::max(sh.nsrc, d.nsrc);
        sh.ndst = std::max(sh.ndst, d.ndst);
        ++sh.ndesc;
    }
    // Cut descriptors into work items, phase by phase.
    uint64_t items_total = 0;
    for (uint32_t ph = 0; ph < 2; ++ph) {
        PhaseShape& sh = shape[ph];
        if (sh.ndesc == 0) continue;
        sh.item = pol.item_bytes ? pol.item_bytes
                  : out.fused    ? fused_item_bytes(out.chunk, sh.bytes)
                                 : auto_item_bytes(sh.bytes, sh.traffic, sh.kind, sh.nsrc, sh.ndst, out.vop);
        for (const purlin_desc& d : out.descs)
            if (d.phase == ph) items_total += ceil_div(d.bytes, sh.item);
        if (items_total > PURLIN_MAX_ITEMS) return PURLIN_ERR_NOMEM;
    }
    out.items.reserve(items_total);
    out.reduce_item_bytes = shape[0].item;
    for (uint32_t ph = 0; ph < 2; ++ph) {
        if (shape[ph].ndesc == 0) continue;
        const uint64_t item = shape[ph].item;
        Phase& phase = out.phases[out.nphases++];
        phase.begin = out.items.size();
        bool first = true;
        for (const purlin_desc& d : out.descs) {
            if (d.phase != ph) continue;
            if (first) {
                phase.kind = d.kind;
                phase.nsrc = d.nsrc;
                phase.src_buf = d.src_buf;
                phase.src_step = d.src_step;
                first = false;
            } else if (d.kind != phase.kind ||
                       (d.kind == PURLIN_KIND_REDUCE &&
                        (d.nsrc != phase.nsrc || d.src_buf != phase.src_buf || d.src_step != phase.src_step))) {
                return PURLIN_ERR_UNSUPPORTED;  // a phase is one kernel: one consume op, one source set
            }
            for (uint64_t o = 0; o < d.bytes; o += item) {
                purlin_desc w = d;
                w.src_off += o;
                w.dst_off += o;
                w.bytes = std::min(item, d.bytes - o);
                out.items.push_back(w);
            }
        }
        phase.count = out.items.size() - phase.begin;
        // Cache hints.  A stream that is touched once and is much larger
        // than the 256 MB last-level cache gains from non-temporal
        // accesses; which side gains was measured on MI355X: reads for
        // many-to-one (reduce), writes for one-to-many (multi-destination
        // copy), both for one-to-one copies.  A reduce also writes
        // non-temporally once its output is larger than that cache: the
        // output can no longer stay there for a next reader, and cached
        // stores of it run slower (P = 8, bf16, fresh output buffers: 1 GiB
        // per rank 72.2% of 8 TB/s against 68.7%, one-phase AllReduce 68.8
        // against 65.9%; at 256 MiB per rank the ReduceScatter's output
        // stays cached for the AllGather that reads it).  Phases whose
        // traffic fits the cache keep cached accesses so repeated calls hit
        // it.
        uint64_t traffic = 0, written = 0, max_ndst = 0;
        for (uint64_t i = phase.begin; i < out.items.size(); ++i) {
            traffic += (uint64_t(out.items[i].nsrc) + out.items[i].ndst) * out.items[i].bytes;
            written += uint64_t(out.items[i].ndst) * out.items[i].bytes;
            max_ndst = std::max<uint64_t>(max_ndst, out.items[i].ndst);
        }
        const bool streaming = traffic >= kStreamingBytes;
        bool auto_nt_load = false, auto_nt_store = false;
        if (streaming) {
            if (phase.kind == PURLIN_KIND_REDUCE) {
                auto_nt_load = true;
                auto_nt_store = written > kLastLevelCacheBytes;
            } else if (max_ndst > 1) {
                auto_nt_store = true;
            } else {
                auto_nt_load = auto_nt_store = true;
            }
        } else if (!out.vop) {
            // Below the streaming threshold, a launch that writes 8-32 MiB
            // runs faster with non-temporal stores when calls follow each
            // other (measured on MI355X, P = 8, bf16: AllReduce at
            // 1-4 MiB/rank 15-23% faster, AllGather and AllToAll 5-38%):
            // cached stores would leave that much dirty data in the XCDs'
            // L2 caches (32 MiB in all).  Smaller launches are bound by
            // launch latency and larger ones gain nothing.  Loads stay
            // cached.  (Variable-size launches tie both hints together and
            // keep the cached form here.)
            auto_nt_store = written >= kLatencyNtStoreMin && written <= kLatencyNtStoreMax;
        }
        phase.nt_load = pol.load_hint ? pol.load_hint == 2 : auto_nt_load;
        phase.nt_store = pol.store_hint ? pol.store_hint == 2 : auto_nt_store;
    }
    return PURLIN_OK;
}

}  // namespace

purlin_status build_plan_v(purlin_op op, int P, uint64_t in_capacity, uint64_t out_capacity, purlin_dtype dtype,
                           uint64_t chunk, uint64_t unit, const purlin_policy* policy, uint32_t flags, Plan& out) {
    if (op != PURLIN_ALLGATHERV && op != PURLIN_REDUCE_SCATTERV && op != PURLIN_ALLTOALLV) return PURLIN_ERR_INVALID;
    if (dtype != PURLIN_FP32 && dtype != PURLIN_BF16) return PURLIN_ERR_INVALID;
    if (P < 1 || P > PURLIN_MAX_RANKS) return PURLIN_ERR_INVALID;
    const uint32_t allowed = PURLIN_PLAN_HOST_ONLY | (op == PURLIN_ALLTOALLV ? PURLIN_PLAN_COUNTS_TRANSPOSED : 0u);
    if (flags & ~allowed) return PURLIN_ERR_INVALID;
    const uint64_t s = dtype == PURLIN_FP32 ? 4 : 2;
    if (chunk < s || chunk % s != 0) return PURLIN_ERR_INVALID;
    if (in_capacity > (uint64_t(1) << 58) / s || out_capacity > (uint64_t(1) << 58) / s) return PURLIN_ERR_INVALID;
    if (unit < 1 || unit > (uint64_t(1) << 31)) return PURLIN_ERR_INVALID;
    purlin_policy pol{};
    if (!parse_policy(policy, pol)) return PURLIN_ERR_INVALID;

    out = Plan{};
    out.op = op;
    out.P = P;
    // ALLTOALLV covers the side whose buffers are smaller: a receive buffer
    // sized for the worst case (every rank sending everything to one rank)
    // then adds no idle work items.
    const bool src_major = op == PURLIN_ALLTOALLV && in_capacity < out_capacity;
    const uint64_t space = (op == PURLIN_REDUCE_SCATTERV || src_major) ? in_capacity : out_capacity;
    out.count = space;
    out.dtype = dtype;
    out.chunk = chunk;
    out.flags = flags;
    out.elem_bytes = s;
    out.vop = true;
    out.in_capacity = in_capacity;
    out.out_capacity = out_capacity;
    out.v_src_major = src_major;
    out.unit = unit;
    out.in_bytes = in_capacity * s;
    out.out_bytes = out_capacity * s;
    out.in_mask = out.out_mask = (1u << P) - 1u;
    if (pol.fanout == 0) pol.fanout = 2;
    if (pol.ar_mode == 0) pol.ar_mode = 2;

    // The virtual index space: the gathered output (ALLGATHERV), the
    // partitioned input (REDUCE_SCATTERV), or each destination's output
    // (ALLTOALLV; each source's input when source-major), cut into chunks;
    // one descriptor per chunk.
    const uint64_t vbytes = space * s;
    const uint64_t Cv = vbytes ? ceil_div(vbytes, chunk) : 0;
    const uint64_t spaces = op == PURLIN_ALLTOALLV ? uint64_t(P) : 1;
    if (Cv > PURLIN_MAX_ITEMS || Cv * spaces > PURLIN_MAX_ITEMS) return PURLIN_ERR_NOMEM;
    const uint32_t out0 = static_cast<uint32_t>(P);
    try {
        for (uint32_t r = 0; r < spaces; ++r)
            for (uint64_t c = 0; c < Cv; ++c) {
                const uint64_t off = c * chunk, len = std::min(chunk, vbytes - off);
                if (op == PURLIN_ALLGATHERV)
                    out.descs.push_back(make_desc(PURLIN_KIND_COPY, 0, 1, 0, 0, P, out0, 1, off, off, len, 0,
                                                  static_cast<uint32_t>(c)));
                else if (op == PURLIN_REDUCE_SCATTERV)
                    out.descs.push_back(make_desc(PURLIN_KIND_REDUCE, 0, P, 0, 1, 1, out0, 0, off, off, len, 0,
                                                  static_cast<uint32_t>(c)));
                else if (src_major)  // source r's input; the sizes pick the output
                    out.descs.push_back(make_desc(PURLIN_KIND_COPY, 0, 1, r, 0, 1, out0, 1, off, off, len, r,
                                                  static_cast<uint32_t>(c)));
                else  // destination r's output; the sizes pick the input
                    out.descs.push_back(make_desc(PURLIN_KIND_COPY, 0, 1, 0, 0, 1, out0 + r, 0, off, off, len, r,
                                                  static_cast<uint32_t>(c)));
            }
        out.policy = pol;
        const purlin_status st = cut_items(out, pol);
        if (st != PURLIN_OK) return st;
    } catch (const std::bad_alloc&) {
        out.descs.clear();
        out.items.clear();
        return PURLIN_ERR_NOMEM;
    }
    return PURLIN_OK;
}

}  // namespace purlin
