// Internal launch entry points of the HIP kernels (exec.hip, moe.hip),
// called by the ABI glue (abi.hip) after host-side validation.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "purlin.h"

namespace purlin {

// Timing records of the measurement entry points (purlin_stream_timed,
// purlin_pack_timed): entry 0..3 = {wall-clock rate in kHz, workgroups, 0,
// 0}; then per workgroup b, entries 4(b+1)..: {XCD (the XCC id register),
// wall clock at entry, wall clock when its metadata was done (its entry for
// a stream), wall clock once all its stores have completed}.
constexpr uint64_t kRecPerGroup = 4;

__device__ __forceinline__ uint32_t xcc_id() {
    uint32_t v;
    __asm__ volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
    return v & 0xFu;
}

// Launch one phase: `n` work items starting at device pointer `items`, all
// of consume op `kind`.  The items of a REDUCE phase all sum the same `nsrc`
// sources bufs[src_buf + p * src_step].  `bufs` holds the 2P buffer pointers.
// nt_load / nt_store select non-temporal global loads / stores.
// Plain copy of `bytes` (a multiple of 16) from src to dst.
hipError_t launch_stream_copy(void* dst, const void* src, uint64_t bytes, hipStream_t stream);
// Reference stream: dst_j[i] = XOR_p src_p[i] per 16-byte vector (see purlin_stream).
hipError_t launch_stream(void* const* dst, int ndst, const void* const* src, int nsrc, uint64_t bytes, void* sink,
                         uint32_t hints, hipStream_t stream, uint64_t* rec = nullptr);
// Workgroups of one launch_stream grid.
uint64_t stream_groups(int nsrc, uint64_t bytes);
// The wall-clock rate of the current device in kHz (0 if unknown).
uint64_t wall_clock_khz();

hipError_t launch_phase(const purlin_desc* items, uint64_t n, uint32_t kind, uint32_t nsrc, uint32_t src_buf,
                        uint32_t src_step, bool nt_load, bool nt_store, purlin_dtype dtype, void* const* bufs,
                        int nbufs, uint32_t max_workgroups, uint32_t copy_depth, hipStream_t stream);

// Device state of a single-launch AllReduce plan (zeroed at plan creation).
struct FusedState {
    // Items claimed over all launches, one counter per partition of the
    // waves (workgroup index mod 8), each on its own 128-byte line: the
    // waves of partition k claim the items of partition k, nk per launch,
    // so launch e's tickets of counter k are [e*nk, (e+1)*nk).
    uint64_t tickets[8 * 16];
    uint32_t error;  // set if a wait gave up (bounded spin)
    uint32_t pad[31];
};

// One launch for a whole AllReduce: items [0, n_reduce) reduce partition k
// into out_k, the rest copy it to the other ranks once its chunk is done.
hipError_t launch_fused_allreduce(const purlin_desc* items, uint64_t n, uint64_t n_reduce, uint32_t nsrc,
                                  purlin_dtype dtype, bool streaming, void* const* bufs, int nbufs, FusedState* state,
                                  uint64_t* ready, uint64_t part_bytes, uint64_t chunk_bytes, uint64_t item_bytes,
                                  uint64_t chunks_per_part, hipStream_t stream);

// Variable-size collectives: one launch; sizes read from device `counts`
// (int32, in units of `unit` elements).  `status` (optional) receives 0 or
// 1 (invalid sizes: the call then writes nothing).  The n items form
// `spaces` equal spaces, each a run of chunks cut at item_bytes.
hipError_t launch_v(purlin_op op, const purlin_desc* items, uint64_t n, int P, purlin_dtype dtype, bool streaming,
                    void* const* bufs, const int32_t* counts, bool counts_transposed, bool source_major,
                    int32_t* status, uint64_t in_capacity, uint64_t out_capacity, uint64_t unit, uint64_t chunk,
                    uint64_t item_bytes, uint32_t spaces, uint32_t max_workgroups, hipStream_t stream);

struct PackWorkspace {
    int32_t* tile_base;  // [ntiles * E]: per-tile expert counts, then row bases
    int32_t* lrank;      // [T * K]: rank of (t, k) among its tile's tokens of the same expert
    int32_t* tile_err;   // [ntiles]
};

constexpr int kPackTileTokens = 64;  // one 64-bit token mask per expert and tile

uint64_t pack_workspace_bytes(int T, int K, int E);
bool moe_launch_fits(int T, int H);  // the pack/unpack grids for T tokens of H elements are launchable
PackWorkspace pack_workspace_carve(void* base, int T, int K, int E);

// Tokens per workgroup of the one-pass pack for this shape, or 0 when
// launch_pack takes the three launches (metadata tiles, scan, rows).
int pack_onepass_tokens(int T, int H, int K, int E);

hipError_t launch_pack(int T, int H, int K, int E, int P, const uint16_t* x, const int32_t* ids,
                       uint16_t* packed, int32_t* dest_counts, int32_t* dest_offsets, int32_t* expert_counts,
                       int32_t* expert_offsets, int32_t* pos, int32_t* dev_status, const PackWorkspace& ws,
                       hipStream_t stream, uint64_t* rec = nullptr);

// The two halves of launch_pack: the metadata (reads ids; fills the
// workspace and the count/offset outputs; given the token matrix, also
// reads it ahead into the caches) and the rows (reads x, ids and the
// workspace; writes packed and pos).
hipError_t launch_pack_meta(int T, int K, int E, int P, const int32_t* ids, int32_t* dest_counts,
                            int32_t* dest_offsets, int32_t* expert_counts, int32_t* expert_offsets, int32_t* dev_status,
                            const PackWorkspace& ws, hipStream_t stream, const void* prefetch = nullptr,
                            uint64_t prefetch_bytes = 0);
hipError_t launch_pack_rows(int T, int H, int K, int E, const uint16_t* x, const int32_t* ids, uint16_t* packed,
                            int32_t* pos, const PackWorkspace& ws, hipStream_t stream);

hipError_t launch_unpack(int T, int H, int K, const uint16_t* y, const int32_t* pos, const float* gates,
                         uint16_t* out, int32_t* dev_status, hipStream_t stream);

// De-duplicated dispatch: one row per (token, destination rank).  The
// workspace holds per-tile destination counts (then bases), each token's
// rank among its tile's tokens per destination, and per-tile error flags.
uint64_t pack_dedup_workspace_bytes(int T, int P);

hipError_t launch_pack_dedup(int T, int H, int K, int E, int P, const uint16_t* x, const int32_t* ids,
                             uint16_t* packed, int32_t* dest_counts, int32_t* dest_offsets, int32_t* row_of,
                             int32_t* dev_status, void* workspace, hipStream_t stream);

hipError_t launch_unpack_dedup(int T, int H, int P, int64_t rows, const uint16_t* y, const int32_t* row_of,
                               uint16_t* out, int32_t* dev_status, hipStream_t stream);

// Expert-parallel dispatch / combine over P ranks (per-rank pointer arrays
// of P host-held device pointers).  The dispatch workspace holds every
// rank's pack workspace, destination offsets, expert counts and status word.
uint64_t ep_dispatch_workspace_bytes(int T, int K, int E, int P);
bool ep_launch_fits(int T, int H, int P);

hipError_t launch_ep_dispatch(int T, int H, int K, int E, int P, const uint16_t* const* x, const int32_t* const* ids,
                              uint16_t* const* recv, int64_t capacity, int32_t* counts, int32_t* recv_pos,
                              int32_t* dev_status, void* workspace, hipStream_t stream);

hipError_t launch_ep_combine(int T, int H, int K, int E, int P, const uint16_t* const* y, int64_t capacity,
                             const int32_t* const* ids, const int32_t* recv_pos, const float* const* gates,
                             uint16_t* const* out, int32_t* dev_status, hipStream_t stream);

// The de-duplicated one-pass dispatch / combine (one row per token and
// owning rank; recv_row is [P, T, P]).
uint64_t ep_dispatch_dedup_workspace_bytes(int T, int P);

hipError_t launch_ep_dispatch_dedup(int T, int H, int K, int E, int P, const uint16_t* const* x,
                                    const int32_t* const* ids, uint16_t* const* recv, int64_t capacity,
                                    int32_t* counts, int32_t* recv_row, int32_t* dev_status, void* workspace,
                                    hipStream_t stream);

hipError_t launch_ep_combine_dedup(int T, int H, int P, const uint16_t* const* y, int64_t capacity,
                                   const int32_t* recv_row, uint16_t* const* out, int32_t* dev_status,
                                   hipStream_t stream);

}  // namespace purlin
