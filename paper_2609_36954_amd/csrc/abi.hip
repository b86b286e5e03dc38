// extern "C" entry points declared in include/purlin.h: host-side argument
// validation (always complete before anything is enqueued), plan lifetime,
// and the launches.  Status codes only: no exception crosses the ABI.

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <mutex>
#include <new>

#include "kernels.h"
#include "plan.h"
#include "purlin.h"

struct purlin_plan_s {
    purlin::Plan plan;
};

// Workspace of the entry points that allocate nothing (purlin_pack_static):
// one copy per GPU, zero at load, held until the process ends.  In host
// code `scratch` names a host-side stand-in, never the device memory: the
// device address comes from hipGetSymbolAddress (static_scratch below).
static __device__ __align__(256) unsigned char scratch[PURLIN_STATIC_SCRATCH_BYTES];

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// [a, a + na) and [b, b + nb) share a byte.
bool overlaps(const void* a, uint64_t na, const void* b, uint64_t nb) {
    if (na == 0 || nb == 0) return false;
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
}

size_t fused_state_bytes(const purlin::Plan& p) {
    return sizeof(purlin::FusedState) + sizeof(uint64_t) * p.chunks_per_part * static_cast<uint64_t>(p.P);
}

// Device copies of a plan: its work items and, for a single-launch
// AllReduce, its zeroed state.  The uploads run on a private non-blocking
// stream that is drained before returning: no other stream, and no capture
// in progress on another stream, is waited for or disturbed.
purlin_status upload_plan(purlin::Plan& pl) {
    const size_t bytes = pl.items.size() * sizeof(purlin_desc);
    if (hipMalloc(reinterpret_cast<void**>(&pl.d_items), bytes) != hipSuccess) {
        pl.d_items = nullptr;
        return PURLIN_ERR_NOMEM;
    }
    const size_t sb = pl.fused ? fused_state_bytes(pl) : 0;
    if (sb && hipMalloc(&pl.d_state, sb) != hipSuccess) {
        pl.d_state = nullptr;
        (void)hipFree(pl.d_items);
        pl.d_items = nullptr;
        return PURLIN_ERR_NOMEM;
    }
    hipStream_t s = nullptr;
    bool ok = hipStreamCreateWithFlags(&s, hipStreamNonBlocking) == hipSuccess;
    ok = ok && hipMemcpyAsync(pl.d_items, pl.items.data(), bytes, hipMemcpyHostToDevice, s) == hipSuccess;
    ok = ok && (!sb || hipMemsetAsync(pl.d_state, 0, sb, s) == hipSuccess);
    ok = ok && hipStreamSynchronize(s) == hipSuccess;
    if (s) (void)hipStreamDestroy(s);
    if (!ok) {
        if (pl.d_state) (void)hipFree(pl.d_state);
        (void)hipFree(pl.d_items);
        pl.d_state = nullptr;
        pl.d_items = nullptr;
        return PURLIN_ERR_DEVICE;
    }
    return PURLIN_OK;
}

purlin_status make_plan(purlin_op op, int P, int root, uint64_t count, purlin_dtype dtype, uint64_t chunk,
                        const purlin_policy* policy, uint32_t flags, purlin_plan_t* out_plan, uint64_t v_unit = 0,
                        uint64_t v_out_capacity = 0, int share = -1) {
    if (!out_plan) return PURLIN_ERR_INVALID;
    *out_plan = nullptr;
    purlin_plan_s* h = new (std::nothrow) purlin_plan_s;
    if (!h) return PURLIN_ERR_NOMEM;
    purlin_status st;
    try {
        st = v_unit ? purlin::build_plan_v(op, P, count, v_out_capacity, dtype, chunk, v_unit, policy, flags, h->plan)
                    : purlin::build_plan(op, P, root, count, dtype, chunk, policy, flags, h->plan, share);
    } catch (...) {
        st = PURLIN_ERR_NOMEM;
    }
    if (st != PURLIN_OK) {
        delete h;
        return st;
    }
    purlin::Plan& pl = h->plan;
    if (!(flags & PURLIN_PLAN_HOST_ONLY) && !pl.items.empty()) {
        const purlin_status dst = upload_plan(pl);
        if (dst != PURLIN_OK) {
            delete h;
            return dst;
        }
    }
    *out_plan = h;
    return PURLIN_OK;
}

// Per-device address of `scratch` (below), looked up once per device.
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mu;

bool pack_limits_ok(int T, int H, int K, int E) {
    if (T < 0 || H < 1 || K < 1 || K > 64 || E < 1 || E > 4096) return false;
    return static_cast<int64_t>(T) * K < (int64_t(1) << 31) && purlin::moe_launch_fits(T, H);
}

// The one input/output overlap a plan allows: rank r's in-place layout,
// where every element is read and rewritten by the same wavefront (or, for
// AllReduce's second phase, rewritten after the first phase has read it).
//   ALLREDUCE, BROADCAST, REDUCE   in_r == out_r
//   REDUCE_SCATTER, SCATTER        out_r == in_r + r * out_bytes
//   ALLGATHER, GATHER              in_r == out_r + r * in_bytes
// Rooted ops only for the root's own pair; ALLTOALL and the variable-size
// ops never (an element there is rewritten before other waves read it).
bool in_place_pair(const purlin::Plan& p, int i, int r, const void* in, const void* out) {
    if (i != r || p.vop) return false;
    if (p.op >= PURLIN_BROADCAST && p.op <= PURLIN_GATHER && r != p.root) return false;
    const char* a = static_cast<const char*>(in);
    const char* b = static_cast<const char*>(out);
    switch (p.op) {
        case PURLIN_ALLREDUCE:
        case PURLIN_BROADCAST:
        case PURLIN_REDUCE:
            return a == b;
        case PURLIN_REDUCE_SCATTER:
        case PURLIN_SCATTER:
            return b == a + uint64_t(r) * p.out_bytes;
        case PURLIN_ALLGATHER:
        case PURLIN_GATHER:
            return a == b + uint64_t(r) * p.in_bytes;
        default:
            return false;
    }
}

// Host-side checks shared by purlin_exec and purlin_exec_v: non-null,
// aligned, no input/output overlap other than an in-place pair, no
// output/output overlap among used buffers.
purlin_status check_buffers(const purlin::Plan& p, void* const* bufs) {
    if (p.flags & PURLIN_PLAN_HOST_ONLY) return PURLIN_ERR_INVALID;
    if (!bufs) return PURLIN_ERR_INVALID;
    const int P = p.P;
    auto used = [&](int i) { return i < P ? ((p.in_mask >> i) & 1u) : ((p.out_mask >> (i - P)) & 1u); };
    for (int i = 0; i < 2 * P; ++i)
        if (used(i) && (!bufs[i] || !aligned16(bufs[i]))) return PURLIN_ERR_INVALID;
    for (int i = 0; i < P; ++i)
        for (int r = 0; r < P; ++r)
            if (used(i) && used(P + r) && overlaps(bufs[i], p.in_bytes, bufs[P + r], p.out_bytes) &&
                !in_place_pair(p, i, r, bufs[i], bufs[P + r]))
                return PURLIN_ERR_INVALID;
    for (int r = 0; r < P; ++r)
        for (int q = r + 1; q < P; ++q)
            if (used(P + r) && used(P + q) && overlaps(bufs[P + r], p.out_bytes, bufs[P + q], p.out_bytes))
                return PURLIN_ERR_INVALID;
    return PURLIN_OK;
}

// EP arguments shared by dispatch and combine: limits and the P ranks' pointers.
bool ep_limits_ok(int T, int H, int K, int E, int P, uint64_t capacity) {
    if (!pack_limits_ok(T, H, K, E)) return false;
    if (P < 1 || P > PURLIN_MAX_RANKS || P > E || E % P != 0) return false;
    if (capacity >= (uint64_t(1) << 31)) return false;
    return purlin::ep_launch_fits(T, H, P);
}

template <class Ptr>
bool all_aligned(Ptr const* v, int P) {
    if (!v) return false;
    for (int p = 0; p < P; ++p)
        if (!v[p] || !aligned16(v[p])) return false;
    return true;
}

// Every purlin_pack argument but the workspace.
purlin_status check_pack_args(int T, int H, int K, int E, int P, const void* x, const int32_t* ids,
                              const void* packed, const int32_t* dest_counts, const int32_t* dest_offsets,
                              const int32_t* expert_counts, const int32_t* expert_offsets, const int32_t* pos,
                              const int32_t* dev_status) {
    if (!pack_limits_ok(T, H, K, E)) return PURLIN_ERR_INVALID;
    if (P < 1 || P > E || E % P != 0) return PURLIN_ERR_INVALID;
    if (!dest_counts || !dest_offsets || !expert_counts) return PURLIN_ERR_INVALID;
    if (!aligned16(dest_counts) || !aligned16(dest_offsets) || !aligned16(expert_counts)) return PURLIN_ERR_INVALID;
    if (expert_offsets && !aligned16(expert_offsets)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    if (T > 0) {
        if (!x || !ids || !packed || !pos) return PURLIN_ERR_INVALID;
        if (!aligned16(x) || !aligned16(ids) || !aligned16(packed) || !aligned16(pos)) return PURLIN_ERR_INVALID;
        const uint64_t xb = uint64_t(T) * H * 2, pb = xb * K;
        if (overlaps(x, xb, packed, pb)) return PURLIN_ERR_INVALID;
    }
    return PURLIN_OK;
}

// purlin_pack after validation, with a workspace of at least
// pack_workspace_bytes(T, K, E) bytes.
purlin_status launch_pack_checked(int T, int H, int K, int E, int P, const void* x, const int32_t* ids, void* packed,
                                  int32_t* dest_counts, int32_t* dest_offsets, int32_t* expert_counts,
                                  int32_t* expert_offsets, int32_t* pos, int32_t* dev_status, void* workspace,
                                  void* stream) {
    const purlin::PackWorkspace ws = purlin::pack_workspace_carve(workspace, T, K, E);
    const hipError_t e = purlin::launch_pack(T, H, K, E, P, static_cast<const uint16_t*>(x), ids,
                                             static_cast<uint16_t*>(packed), dest_counts, dest_offsets,
                                             expert_counts, expert_offsets, pos, dev_status, ws,
                                             static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

// This device's address of `scratch`: looked up on the first call on each
// device (with that device current), then reused.
purlin_status static_scratch(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return PURLIN_ERR_DEVICE;
    if (dev < 0 || dev >= kMaxDevices) return PURLIN_ERR_UNSUPPORTED;
    void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_addr[dev].load(std::memory_order_relaxed);
        if (!p) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return PURLIN_ERR_DEVICE;
            g_scratch_addr[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return PURLIN_OK;
}

}  // namespace

extern "C" {

purlin_status purlin_plan(purlin_op op, int P, uint64_t count, purlin_dtype dtype, uint64_t chunk_bytes,
                          purlin_plan_t* out_plan) {
    return make_plan(op, P, -1, count, dtype, chunk_bytes, nullptr, 0, out_plan);
}

purlin_status purlin_plan_ex(purlin_op op, int P, uint64_t count, purlin_dtype dtype, uint64_t chunk_bytes,
                             const purlin_policy* policy, uint32_t flags, purlin_plan_t* out_plan) {
    return make_plan(op, P, -1, count, dtype, chunk_bytes, policy, flags, out_plan);
}

purlin_status purlin_plan_rooted(purlin_op op, int P, int root, uint64_t count, purlin_dtype dtype,
                                 uint64_t chunk_bytes, const purlin_policy* policy, uint32_t flags,
                                 purlin_plan_t* out_plan) {
    if (op < PURLIN_BROADCAST || op > PURLIN_GATHER) {
        if (out_plan) *out_plan = nullptr;
        return PURLIN_ERR_INVALID;
    }
    return make_plan(op, P, root, count, dtype, chunk_bytes, policy, flags, out_plan);
}

purlin_status purlin_plan_share(purlin_op op, int P, int root, int rank, uint64_t count, purlin_dtype dtype,
                                uint64_t chunk_bytes, const purlin_policy* policy, uint32_t flags,
                                purlin_plan_t* out_plan) {
    if (op < PURLIN_ALLREDUCE || op > PURLIN_GATHER || rank < 0 || rank >= P) {
        if (out_plan) *out_plan = nullptr;
        return PURLIN_ERR_INVALID;
    }
    return make_plan(op, P, root, count, dtype, chunk_bytes, policy, flags, out_plan, 0, 0, rank);
}

purlin_status purlin_plan_v(purlin_op op, int P, uint64_t in_capacity, uint64_t out_capacity, purlin_dtype dtype,
                            uint64_t chunk_bytes, uint64_t unit, const purlin_policy* policy, uint32_t flags,
                            purlin_plan_t* out_plan) {
    if (unit == 0) {
        if (out_plan) *out_plan = nullptr;
        return PURLIN_ERR_INVALID;
    }
    return make_plan(op, P, -1, in_capacity, dtype, chunk_bytes, policy, flags, out_plan, unit, out_capacity);
}

purlin_status purlin_plan_info(purlin_plan_t plan, uint64_t* n_desc, uint64_t* in_bytes_per_rank,
                               uint64_t* out_bytes_per_rank, uint64_t* sched_bytes) {
    if (!plan) return PURLIN_ERR_INVALID;
    const purlin::Plan& p = plan->plan;
    if (n_desc) *n_desc = p.descs.size();
    if (in_bytes_per_rank) *in_bytes_per_rank = p.in_bytes;
    if (out_bytes_per_rank) *out_bytes_per_rank = p.out_bytes;
    if (sched_bytes) *sched_bytes = p.sched_bytes;
    return PURLIN_OK;
}

purlin_status purlin_plan_descriptors(purlin_plan_t plan, const purlin_desc** table, uint64_t* n, uint64_t* stride) {
    if (!plan || !table || !n) return PURLIN_ERR_INVALID;
    *table = plan->plan.descs.data();
    *n = plan->plan.descs.size();
    if (stride) *stride = sizeof(purlin_desc);
    return PURLIN_OK;
}

purlin_status purlin_plan_items(purlin_plan_t plan, const purlin_desc** items, uint64_t* n, uint64_t phase_begin[3]) {
    if (!plan || !items || !n) return PURLIN_ERR_INVALID;
    const purlin::Plan& p = plan->plan;
    *items = p.items.data();
    *n = p.items.size();
    if (phase_begin) {
        // phase 0 always comes first; a plan has a phase 1 only as its second launch
        phase_begin[0] = 0;
        phase_begin[1] = p.nphases == 2 ? p.phases[1].begin : p.items.size();
        phase_begin[2] = p.items.size();
    }
    return PURLIN_OK;
}

purlin_status purlin_exec_v(purlin_plan_t plan, void* const* bufs, const int32_t* counts, int32_t* dev_status,
                            void* stream) {
    if (!plan) return PURLIN_ERR_INVALID;
    const purlin::Plan& p = plan->plan;
    if (!p.vop) return PURLIN_ERR_INVALID;
    if (p.flags & PURLIN_PLAN_HOST_ONLY) return PURLIN_ERR_INVALID;
    if (!counts || (reinterpret_cast<uintptr_t>(counts) & 3u)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    void* const no_bufs[2 * PURLIN_MAX_RANKS] = {};
    if (p.items.empty()) {
        // zero capacity: no buffer is touched (bufs is ignored and may be
        // NULL), but the sizes are still checked on the device when a status
        // word is given
        if (!dev_status) return PURLIN_OK;
        bufs = no_bufs;
    } else {
        const purlin_status st = check_buffers(p, bufs);
        if (st != PURLIN_OK) return st;
    }
    const purlin::Phase& ph = p.phases[0];
    const hipError_t e =
        purlin::launch_v(p.op, p.d_items, ph.count, p.P, p.dtype, ph.nt_load || ph.nt_store, bufs, counts,
                         (p.flags & PURLIN_PLAN_COUNTS_TRANSPOSED) != 0, p.v_src_major, dev_status, p.in_capacity,
                         p.out_capacity, p.unit, p.chunk, p.reduce_item_bytes ? p.reduce_item_bytes : p.chunk,
                         p.op == PURLIN_ALLTOALLV ? static_cast<uint32_t>(p.P) : 1u, p.policy.max_workgroups,
                         static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_exec(purlin_plan_t plan, void* const* bufs, void* stream) {
    if (!plan) return PURLIN_ERR_INVALID;
    const purlin::Plan& p = plan->plan;
    if (p.vop) return PURLIN_ERR_INVALID;  // sizes come with purlin_exec_v
    if (p.count == 0) return PURLIN_OK;
    const purlin_status st = check_buffers(p, bufs);
    if (st != PURLIN_OK) return st;
    const int P = p.P;

    hipStream_t s = static_cast<hipStream_t>(stream);
    if (p.fused) {
        auto* state = static_cast<purlin::FusedState*>(p.d_state);
        auto* ready = reinterpret_cast<uint64_t*>(state + 1);
        const uint64_t n = p.items.size();
        const uint64_t n_reduce = p.phases[0].count;
        const hipError_t e = purlin::launch_fused_allreduce(
            p.d_items, n, n_reduce, p.phases[0].nsrc, p.dtype, p.phases[0].nt_load, bufs, 2 * P, state, ready,
            p.part_bytes, p.chunk, p.reduce_item_bytes, p.chunks_per_part, s);
        return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
    }
    for (int i = 0; i < p.nphases; ++i) {
        const purlin::Phase& ph = p.phases[i];
        const hipError_t e =
            purlin::launch_phase(p.d_items + ph.begin, ph.count, ph.kind, ph.nsrc, ph.src_buf, ph.src_step, ph.nt_load,
                                 ph.nt_store, p.dtype, bufs, 2 * P, p.policy.max_workgroups, p.policy.copy_depth, s);
        if (e != hipSuccess) return PURLIN_ERR_DEVICE;
    }
    return PURLIN_OK;
}

purlin_status purlin_plan_device_error(purlin_plan_t plan, uint32_t* error) {
    if (!plan || !error) return PURLIN_ERR_INVALID;
    *error = 0;
    if (!plan->plan.d_state) return PURLIN_OK;
    if (hipDeviceSynchronize() != hipSuccess) return PURLIN_ERR_DEVICE;
    const auto* state = static_cast<const purlin::FusedState*>(plan->plan.d_state);
    if (hipMemcpy(error, &state->error, sizeof(uint32_t), hipMemcpyDeviceToHost) != hipSuccess)
        return PURLIN_ERR_DEVICE;
    return PURLIN_OK;
}

void purlin_plan_destroy(purlin_plan_t plan) {
    if (!plan) return;
    if (plan->plan.d_items) (void)hipFree(plan->plan.d_items);
    if (plan->plan.d_state) (void)hipFree(plan->plan.d_state);
    delete plan;
}

purlin_status purlin_pack_workspace_size(int T, int K, int E, uint64_t* bytes) {
    if (!bytes || T < 0 || K < 1 || K > 64 || E < 1 || E > 4096) return PURLIN_ERR_INVALID;
    if (static_cast<int64_t>(T) * K >= (int64_t(1) << 31)) return PURLIN_ERR_INVALID;
    *bytes = purlin::pack_workspace_bytes(T, K, E);
    return PURLIN_OK;
}

purlin_status purlin_pack_single_launch(int T, int H, int K, int E, int* single) {
    if (!single || !pack_limits_ok(T, H, K, E)) return PURLIN_ERR_INVALID;
    *single = purlin::pack_onepass_tokens(T, H, K, E) > 0 ? 1 : 0;
    return PURLIN_OK;
}

purlin_status purlin_pack(int T, int H, int K, int E, int P, const void* x, const int32_t* ids, void* packed,
                          int32_t* dest_counts, int32_t* dest_offsets, int32_t* expert_counts,
                          int32_t* expert_offsets, int32_t* pos, int32_t* dev_status, void* workspace,
                          uint64_t workspace_bytes, void* stream) {
    const purlin_status st =
        check_pack_args(T, H, K, E, P, x, ids, packed, dest_counts, dest_offsets, expert_counts, expert_offsets, pos,
                        dev_status);
    if (st != PURLIN_OK) return st;
    const uint64_t need = purlin::pack_workspace_bytes(T, K, E);
    if (workspace_bytes < need || (need && (!workspace || !aligned16(workspace)))) return PURLIN_ERR_INVALID;
    return launch_pack_checked(T, H, K, E, P, x, ids, packed, dest_counts, dest_offsets, expert_counts,
                               expert_offsets, pos, dev_status, workspace, stream);
}

purlin_status purlin_pack_meta(int T, int K, int E, int P, const int32_t* ids, int32_t* dest_counts,
                               int32_t* dest_offsets, int32_t* expert_counts, int32_t* expert_offsets,
                               int32_t* dev_status, void* workspace, uint64_t workspace_bytes, void* stream) {
    if (T < 0 || K < 1 || K > 64 || E < 1 || E > 4096 || static_cast<int64_t>(T) * K >= (int64_t(1) << 31))
        return PURLIN_ERR_INVALID;
    if (P < 1 || P > E || E % P != 0) return PURLIN_ERR_INVALID;
    if (!dest_counts || !dest_offsets || !expert_counts) return PURLIN_ERR_INVALID;
    if (!aligned16(dest_counts) || !aligned16(dest_offsets) || !aligned16(expert_counts)) return PURLIN_ERR_INVALID;
    if (expert_offsets && !aligned16(expert_offsets)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    if (T > 0 && (!ids || !aligned16(ids))) return PURLIN_ERR_INVALID;
    const uint64_t need = purlin::pack_workspace_bytes(T, K, E);
    if (workspace_bytes < need || (need && (!workspace || !aligned16(workspace)))) return PURLIN_ERR_INVALID;
    const purlin::PackWorkspace ws = purlin::pack_workspace_carve(workspace, T, K, E);
    const hipError_t e = purlin::launch_pack_meta(T, K, E, P, ids, dest_counts, dest_offsets, expert_counts,
                                                  expert_offsets, dev_status, ws, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_pack_rows(int T, int H, int K, int E, const void* x, const int32_t* ids, void* packed,
                               int32_t* pos, const void* workspace, uint64_t workspace_bytes, void* stream) {
    if (!pack_limits_ok(T, H, K, E)) return PURLIN_ERR_INVALID;
    if (T > 0) {
        if (!x || !ids || !packed || !pos) return PURLIN_ERR_INVALID;
        if (!aligned16(x) || !aligned16(ids) || !aligned16(packed) || !aligned16(pos)) return PURLIN_ERR_INVALID;
        const uint64_t xb = uint64_t(T) * H * 2, pb = xb * K;
        if (overlaps(x, xb, packed, pb)) return PURLIN_ERR_INVALID;
    }
    const uint64_t need = purlin::pack_workspace_bytes(T, K, E);
    if (workspace_bytes < need || (need && (!workspace || !aligned16(workspace)))) return PURLIN_ERR_INVALID;
    const purlin::PackWorkspace ws = purlin::pack_workspace_carve(const_cast<void*>(workspace), T, K, E);
    const hipError_t e = purlin::launch_pack_rows(T, H, K, E, static_cast<const uint16_t*>(x), ids,
                                                  static_cast<uint16_t*>(packed), pos, ws,
                                                  static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_pack_static(int T, int H, int K, int E, int P, const void* x, const int32_t* ids, void* packed,
                                 int32_t* dest_counts, int32_t* dest_offsets, int32_t* expert_counts,
                                 int32_t* expert_offsets, int32_t* pos, int32_t* dev_status, void* stream) {
    purlin_status st = check_pack_args(T, H, K, E, P, x, ids, packed, dest_counts, dest_offsets, expert_counts,
                                       expert_offsets, pos, dev_status);
    if (st != PURLIN_OK) return st;
    if (purlin::pack_workspace_bytes(T, K, E) > PURLIN_STATIC_SCRATCH_BYTES) return PURLIN_ERR_INVALID;
    void* ws = nullptr;
    st = static_scratch(&ws);
    if (st != PURLIN_OK) return st;
    return launch_pack_checked(T, H, K, E, P, x, ids, packed, dest_counts, dest_offsets, expert_counts,
                               expert_offsets, pos, dev_status, ws, stream);
}

purlin_status purlin_pack_dedup_workspace_size(int T, int P, uint64_t* bytes) {
    if (!bytes || T < 0 || P < 1 || P > PURLIN_MAX_RANKS) return PURLIN_ERR_INVALID;
    *bytes = purlin::pack_dedup_workspace_bytes(T, P);
    return PURLIN_OK;
}

purlin_status purlin_pack_dedup(int T, int H, int K, int E, int P, const void* x, const int32_t* ids, void* packed,
                                int32_t* dest_counts, int32_t* dest_offsets, int32_t* row_of, int32_t* dev_status,
                                void* workspace, uint64_t workspace_bytes, void* stream) {
    if (!pack_limits_ok(T, H, K, E)) return PURLIN_ERR_INVALID;
    if (P < 1 || P > PURLIN_MAX_RANKS || P > E || E % P != 0) return PURLIN_ERR_INVALID;
    if (!dest_counts || !dest_offsets || !aligned16(dest_counts) || !aligned16(dest_offsets)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    const uint64_t need = purlin::pack_dedup_workspace_bytes(T, P);
    if (workspace_bytes < need || (need && (!workspace || !aligned16(workspace)))) return PURLIN_ERR_INVALID;
    if (T > 0) {
        if (!x || !ids || !packed || !row_of) return PURLIN_ERR_INVALID;
        if (!aligned16(x) || !aligned16(ids) || !aligned16(packed) || !aligned16(row_of)) return PURLIN_ERR_INVALID;
        const uint64_t xb = uint64_t(T) * H * 2, pb = xb * static_cast<uint64_t>(std::min(K, P));
        if (overlaps(x, xb, packed, pb)) return PURLIN_ERR_INVALID;
    }
    const hipError_t e = purlin::launch_pack_dedup(T, H, K, E, P, static_cast<const uint16_t*>(x), ids,
                                                   static_cast<uint16_t*>(packed), dest_counts, dest_offsets, row_of,
                                                   dev_status, workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_unpack_dedup(int T, int H, int P, int64_t rows, const void* y, const int32_t* row_of, void* out,
                                  int32_t* dev_status, void* stream) {
    if (T < 0 || H < 1 || P < 1 || P > PURLIN_MAX_RANKS) return PURLIN_ERR_INVALID;
    if (rows < 0 || rows >= (int64_t(1) << 31) || !purlin::moe_launch_fits(T, H)) return PURLIN_ERR_INVALID;
    if (static_cast<int64_t>(T) * P >= (int64_t(1) << 31)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    if (T > 0) {
        if (!row_of || !out || (rows > 0 && !y)) return PURLIN_ERR_INVALID;
        if (!aligned16(row_of) || !aligned16(out) || (y && !aligned16(y))) return PURLIN_ERR_INVALID;
        const uint64_t ob = uint64_t(T) * H * 2, yb = uint64_t(rows) * H * 2;
        if (rows > 0 && overlaps(y, yb, out, ob)) return PURLIN_ERR_INVALID;
    }
    const hipError_t e = purlin::launch_unpack_dedup(T, H, P, rows, static_cast<const uint16_t*>(y), row_of,
                                                     static_cast<uint16_t*>(out), dev_status,
                                                     static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_ep_dispatch_workspace_size(int T, int K, int E, int P, uint64_t* bytes) {
    if (!bytes || !pack_limits_ok(T, 1, K, E)) return PURLIN_ERR_INVALID;
    if (P < 1 || P > PURLIN_MAX_RANKS || P > E || E % P != 0) return PURLIN_ERR_INVALID;
    *bytes = purlin::ep_dispatch_workspace_bytes(T, K, E, P);
    return PURLIN_OK;
}

purlin_status purlin_ep_dispatch(int T, int H, int K, int E, int P, const void* const* x, const int32_t* const* ids,
                                 void* const* recv, uint64_t capacity, int32_t* counts, int32_t* recv_pos,
                                 int32_t* dev_status, void* workspace, uint64_t workspace_bytes, void* stream) {
    if (!ep_limits_ok(T, H, K, E, P, capacity)) return PURLIN_ERR_INVALID;
    if (!counts || (reinterpret_cast<uintptr_t>(counts) & 3u)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    const uint64_t need = purlin::ep_dispatch_workspace_bytes(T, K, E, P);
    if (workspace_bytes < need || (need && (!workspace || !aligned16(workspace)))) return PURLIN_ERR_INVALID;
    if (T > 0) {
        if (!all_aligned(x, P) || !all_aligned(ids, P) || !all_aligned(recv, P)) return PURLIN_ERR_INVALID;
        if (!recv_pos || (reinterpret_cast<uintptr_t>(recv_pos) & 3u)) return PURLIN_ERR_INVALID;
        const uint64_t xb = uint64_t(T) * H * 2, rb = capacity * uint64_t(H) * 2;
        for (int r = 0; r < P; ++r) {
            for (int q = r + 1; q < P; ++q)
                if (overlaps(recv[r], rb, recv[q], rb)) return PURLIN_ERR_INVALID;
            for (int p = 0; p < P; ++p)
                if (overlaps(recv[r], rb, x[p], xb)) return PURLIN_ERR_INVALID;
        }
    }
    const hipError_t e = purlin::launch_ep_dispatch(
        T, H, K, E, P, reinterpret_cast<const uint16_t* const*>(x), ids, reinterpret_cast<uint16_t* const*>(recv),
        static_cast<int64_t>(capacity), counts, recv_pos, dev_status, workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_ep_combine(int T, int H, int K, int E, int P, const void* const* y, uint64_t capacity,
                                const int32_t* const* ids, const int32_t* recv_pos, const float* const* gates,
                                void* const* out, int32_t* dev_status, void* stream) {
    if (!ep_limits_ok(T, H, K, E, P, capacity)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    if (T > 0) {
        if (!all_aligned(ids, P) || !all_aligned(gates, P) || !all_aligned(out, P)) return PURLIN_ERR_INVALID;
        if (capacity > 0 && !all_aligned(y, P)) return PURLIN_ERR_INVALID;
        if (!recv_pos || (reinterpret_cast<uintptr_t>(recv_pos) & 3u)) return PURLIN_ERR_INVALID;
        const uint64_t ob = uint64_t(T) * H * 2, yb = capacity * uint64_t(H) * 2;
        for (int p = 0; p < P; ++p) {
            for (int q = p + 1; q < P; ++q)
                if (overlaps(out[p], ob, out[q], ob)) return PURLIN_ERR_INVALID;
            for (int r = 0; r < P && capacity > 0; ++r)
                if (overlaps(out[p], ob, y[r], yb)) return PURLIN_ERR_INVALID;
        }
    }
    const hipError_t e = purlin::launch_ep_combine(
        T, H, K, E, P, reinterpret_cast<const uint16_t* const*>(y), static_cast<int64_t>(capacity), ids, recv_pos,
        gates, reinterpret_cast<uint16_t* const*>(out), dev_status, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_ep_dispatch_dedup_workspace_size(int T, int P, uint64_t* bytes) {
    if (!bytes || T < 0 || P < 1 || P > PURLIN_MAX_RANKS) return PURLIN_ERR_INVALID;
    *bytes = purlin::ep_dispatch_dedup_workspace_bytes(T, P);
    return PURLIN_OK;
}

purlin_status purlin_ep_dispatch_dedup(int T, int H, int K, int E, int P, const void* const* x,
                                       const int32_t* const* ids, void* const* recv, uint64_t capacity,
                                       int32_t* counts, int32_t* recv_row, int32_t* dev_status, void* workspace,
                                       uint64_t workspace_bytes, void* stream) {
    if (!ep_limits_ok(T, H, K, E, P, capacity)) return PURLIN_ERR_INVALID;
    if (!counts || (reinterpret_cast<uintptr_t>(counts) & 3u)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    const uint64_t need = purlin::ep_dispatch_dedup_workspace_bytes(T, P);
    if (workspace_bytes < need || (need && (!workspace || !aligned16(workspace)))) return PURLIN_ERR_INVALID;
    if (T > 0) {
        if (!all_aligned(x, P) || !all_aligned(ids, P) || !all_aligned(recv, P)) return PURLIN_ERR_INVALID;
        if (!recv_row || (reinterpret_cast<uintptr_t>(recv_row) & 3u)) return PURLIN_ERR_INVALID;
        const uint64_t xb = uint64_t(T) * H * 2, rb = capacity * uint64_t(H) * 2;
        for (int r = 0; r < P; ++r) {
            for (int q = r + 1; q < P; ++q)
                if (overlaps(recv[r], rb, recv[q], rb)) return PURLIN_ERR_INVALID;
            for (int p = 0; p < P; ++p)
                if (overlaps(recv[r], rb, x[p], xb)) return PURLIN_ERR_INVALID;
        }
    }
    const hipError_t e = purlin::launch_ep_dispatch_dedup(
        T, H, K, E, P, reinterpret_cast<const uint16_t* const*>(x), ids, reinterpret_cast<uint16_t* const*>(recv),
        static_cast<int64_t>(capacity), counts, recv_row, dev_status, workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_ep_combine_dedup(int T, int H, int P, const void* const* y, uint64_t capacity,
                                      const int32_t* recv_row, void* const* out, int32_t* dev_status, void* stream) {
    if (T < 0 || H < 1 || P < 1 || P > PURLIN_MAX_RANKS) return PURLIN_ERR_INVALID;
    if (capacity >= (uint64_t(1) << 31) || !purlin::ep_launch_fits(T, H, P)) return PURLIN_ERR_INVALID;
    if (static_cast<int64_t>(T) * P >= (int64_t(1) << 31)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    if (T > 0) {
        if (!all_aligned(out, P)) return PURLIN_ERR_INVALID;
        if (capacity > 0 && !all_aligned(y, P)) return PURLIN_ERR_INVALID;
        if (!recv_row || (reinterpret_cast<uintptr_t>(recv_row) & 3u)) return PURLIN_ERR_INVALID;
        const uint64_t ob = uint64_t(T) * H * 2, yb = capacity * uint64_t(H) * 2;
        for (int p = 0; p < P; ++p) {
            for (int q = p + 1; q < P; ++q)
                if (overlaps(out[p], ob, out[q], ob)) return PURLIN_ERR_INVALID;
            for (int r = 0; r < P && capacity > 0; ++r)
                if (overlaps(out[p], ob, y[r], yb)) return PURLIN_ERR_INVALID;
        }
    }
    const hipError_t e = purlin::launch_ep_combine_dedup(
        T, H, P, reinterpret_cast<const uint16_t* const*>(y), static_cast<int64_t>(capacity), recv_row,
        reinterpret_cast<uint16_t* const*>(out), dev_status, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_unpack(int T, int H, int K, const void* y, const int32_t* pos, const float* gates, void* out,
                            int32_t* dev_status, void* stream) {
    if (T < 0 || H < 1 || K < 1 || K > 64) return PURLIN_ERR_INVALID;
    if (static_cast<int64_t>(T) * K >= (int64_t(1) << 31) || !purlin::moe_launch_fits(T, H)) return PURLIN_ERR_INVALID;
    if (dev_status && (reinterpret_cast<uintptr_t>(dev_status) & 3u)) return PURLIN_ERR_INVALID;
    if (T > 0) {
        if (!y || !pos || !gates || !out) return PURLIN_ERR_INVALID;
        if (!aligned16(y) || !aligned16(pos) || !aligned16(gates) || !aligned16(out)) return PURLIN_ERR_INVALID;
        const uint64_t ob = uint64_t(T) * H * 2, yb = ob * K;
        if (overlaps(y, yb, out, ob)) return PURLIN_ERR_INVALID;
    }
    const hipError_t e = purlin::launch_unpack(T, H, K, static_cast<const uint16_t*>(y), pos, gates,
                                               static_cast<uint16_t*>(out), dev_status,
                                               static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_stream_copy(void* dst, const void* src, uint64_t bytes, void* stream) {
    if (bytes % 16) return PURLIN_ERR_INVALID;
    if (bytes == 0) return PURLIN_OK;
    if (!dst || !src || !aligned16(dst) || !aligned16(src)) return PURLIN_ERR_INVALID;
    if (overlaps(dst, bytes, src, bytes)) return PURLIN_ERR_INVALID;
    const hipError_t e = purlin::launch_stream_copy(dst, src, bytes, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_stream(void* const* dst, int ndst, const void* const* src, int nsrc, uint64_t bytes, void* sink,
                            uint32_t hints, void* stream) {
    if (hints & ~uint32_t(PURLIN_STREAM_NT_LOAD | PURLIN_STREAM_NT_STORE)) return PURLIN_ERR_INVALID;
    if (nsrc < 0 || ndst < 0 || nsrc > PURLIN_MAX_RANKS || ndst > PURLIN_MAX_RANKS || nsrc + ndst == 0)
        return PURLIN_ERR_INVALID;
    if (bytes % 16) return PURLIN_ERR_INVALID;
    if (bytes == 0) return PURLIN_OK;
    if ((nsrc && !src) || (ndst && !dst)) return PURLIN_ERR_INVALID;
    if (ndst == 0 && (!sink || !aligned16(sink))) return PURLIN_ERR_INVALID;
    for (int p = 0; p < nsrc; ++p)
        if (!src[p] || !aligned16(src[p])) return PURLIN_ERR_INVALID;
    for (int j = 0; j < ndst; ++j) {
        if (!dst[j] || !aligned16(dst[j])) return PURLIN_ERR_INVALID;
        for (int p = 0; p < nsrc; ++p)
            if (overlaps(dst[j], bytes, src[p], bytes)) return PURLIN_ERR_INVALID;
        for (int k = 0; k < j; ++k)
            if (overlaps(dst[j], bytes, dst[k], bytes)) return PURLIN_ERR_INVALID;
    }
    const hipError_t e = purlin::launch_stream(dst, ndst, src, nsrc, bytes, sink, hints, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_stream_timed(void* const* dst, int ndst, const void* const* src, int nsrc, uint64_t bytes,
                                  void* sink, uint32_t hints, uint64_t* rec, uint64_t rec_entries, uint64_t* groups,
                                  void* stream) {
    if (nsrc < 0 || nsrc > PURLIN_MAX_RANKS || bytes % 16) return PURLIN_ERR_INVALID;
    const uint64_t g = purlin::stream_groups(nsrc, bytes);
    if (groups) *groups = g;
    if (!rec) return PURLIN_OK;
    if (g == 0) return purlin_stream(dst, ndst, src, nsrc, bytes, sink, hints, stream);
    if (!aligned16(rec) || rec_entries < purlin::kRecPerGroup * (g + 1)) return PURLIN_ERR_INVALID;
    if (overlaps(rec, rec_entries * 8, sink, 16)) return PURLIN_ERR_INVALID;
    for (int j = 0; j < ndst && dst; ++j)
        if (overlaps(rec, rec_entries * 8, dst[j], bytes)) return PURLIN_ERR_INVALID;
    // the stream's own checks, then the timed launch
    if (hints & ~uint32_t(PURLIN_STREAM_NT_LOAD | PURLIN_STREAM_NT_STORE)) return PURLIN_ERR_INVALID;
    if (ndst < 0 || ndst > PURLIN_MAX_RANKS || nsrc + ndst == 0) return PURLIN_ERR_INVALID;
    if ((nsrc && !src) || (ndst && !dst)) return PURLIN_ERR_INVALID;
    if (ndst == 0 && (!sink || !aligned16(sink))) return PURLIN_ERR_INVALID;
    for (int p = 0; p < nsrc; ++p)
        if (!src[p] || !aligned16(src[p])) return PURLIN_ERR_INVALID;
    for (int j = 0; j < ndst; ++j) {
        if (!dst[j] || !aligned16(dst[j])) return PURLIN_ERR_INVALID;
        for (int p = 0; p < nsrc; ++p)
            if (overlaps(dst[j], bytes, src[p], bytes)) return PURLIN_ERR_INVALID;
        for (int k = 0; k < j; ++k)
            if (overlaps(dst[j], bytes, dst[k], bytes)) return PURLIN_ERR_INVALID;
    }
    const hipError_t e =
        purlin::launch_stream(dst, ndst, src, nsrc, bytes, sink, hints, static_cast<hipStream_t>(stream), rec);
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

purlin_status purlin_pack_timed(int T, int H, int K, int E, int P, const void* x, const int32_t* ids, void* packed,
                                int32_t* dest_counts, int32_t* dest_offsets, int32_t* expert_counts,
                                int32_t* expert_offsets, int32_t* pos, int32_t* dev_status, uint64_t* rec,
                                uint64_t rec_entries, uint64_t* groups, void* stream) {
    if (!pack_limits_ok(T, H, K, E)) return PURLIN_ERR_INVALID;
    const int tw = purlin::pack_onepass_tokens(T, H, K, E);
    if (tw == 0) return PURLIN_ERR_UNSUPPORTED;
    const uint64_t g = (static_cast<uint64_t>(T) + tw - 1) / tw;
    if (groups) *groups = g;
    if (!rec) return PURLIN_OK;
    const purlin_status st = check_pack_args(T, H, K, E, P, x, ids, packed, dest_counts, dest_offsets, expert_counts,
                                             expert_offsets, pos, dev_status);
    if (st != PURLIN_OK) return st;
    if (!aligned16(rec) || rec_entries < purlin::kRecPerGroup * (g + 1)) return PURLIN_ERR_INVALID;
    if (overlaps(rec, rec_entries * 8, packed, uint64_t(T) * K * H * 2)) return PURLIN_ERR_INVALID;
    const purlin::PackWorkspace ws{};  // the one-launch form uses none
    const hipError_t e = purlin::launch_pack(T, H, K, E, P, static_cast<const uint16_t*>(x), ids,
                                             static_cast<uint16_t*>(packed), dest_counts, dest_offsets,
                                             expert_counts, expert_offsets, pos, dev_status, ws,
                                             static_cast<hipStream_t>(stream), rec);
    return e == hipSuccess ? PURLIN_OK : PURLIN_ERR_DEVICE;
}

const char* purlin_status_string(purlin_status status) {
    switch (status) {
        case PURLIN_OK: return "ok";
        case PURLIN_ERR_INVALID: return "invalid argument";
        case PURLIN_ERR_UNSUPPORTED: return "unsupported";
        case PURLIN_ERR_NOMEM: return "out of memory or descriptor table too large";
        case PURLIN_ERR_DEVICE: return "device error";
    }
    return "unknown status";
}

const char* purlin_version(void) { return "0.1.0"; }

}  // extern "C"
