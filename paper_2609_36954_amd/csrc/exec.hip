// Datapath executor for gfx950: each 64-wide wavefront takes one work item
// (a slice of a chunk descriptor) and moves its bytes.
//
// Paper passages (Purlin, arXiv 2609.36954):
//  - Section 3.3 / Listing 3: the datapath offers copy (move one contiguous
//    byte range) and reduce (combine n equally sized typed sources into one
//    destination); both share one load path and differ only in the step
//    applied to the data once it is in registers.
//  - Section 3.3, Eq. 2: a reduction keeps one FP32 accumulator per output
//    element, starts it at zero and adds rank 0, 1, ..., n-1 in that order,
//    converting each term to FP32 and the sum back to the element type once;
//    throughput comes from many accumulators across elements, never from
//    reassociating across ranks.
//  - Section 3.3, Eq. 3 and Section 2.2, Eq. 1: bandwidth needs bytes in
//    flight.  The paper stages through shared memory with asynchronous
//    copies on its GPUs; here each lane keeps U (copy) or U*nsrc (reduce)
//    independent 16-byte global loads in flight before consuming any, and
//    thousands of wavefronts run at once, which is what HBM3E needs.  No
//    LDS is involved: the data is used once, straight from registers.

#include "kernels.h"

#include <algorithm>

namespace purlin {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;


struct ExecArgs {
    const purlin_desc* items;
    uint64_t n_items;
    uint64_t wave_stride;  // wavefronts in the grid: a wave takes items w, w + stride, ...
    char* bufs[2 * PURLIN_MAX_RANKS];
    // Sources of a REDUCE phase, resolved on the host: every item of such a
    // phase names the same sources (bufs[src_buf + p * src_step]), so the
    // kernel reads them at constant argument offsets instead of issuing one
    // dependent indexed lookup per source.
    char* srcs[PURLIN_MAX_RANKS];
};

// Loads in flight per lane: U vectors for a copy, U * NSRC for a reduce.
constexpr int kCopyUnroll = 4;
constexpr int reduce_unroll(int nsrc) { return nsrc >= 16 ? 1 : (nsrc >= 8 ? 2 : (nsrc >= 4 ? 4 : 8)); }

__device__ __forceinline__ uint32_t wave_index() {
    return __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + threadIdx.x / kWave);
}

__device__ __forceinline__ uint32_t lane_index() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ int64_t readlane64(int64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(v), lane);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(static_cast<uint64_t>(v) >> 32), lane);
    return static_cast<int64_t>((uint64_t(hi) << 32) | lo);
}

// 16-byte global access; NT selects the non-temporal (streaming) form,
// which tells the caches the line will not be reused.
template <bool NT>
__device__ __forceinline__ u32x4 load16(const char* p) {
    if constexpr (NT)
        return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    else
        return *reinterpret_cast<const u32x4*>(p);
}

template <bool NT>
__device__ __forceinline__ void store16(char* p, u32x4 v) {
    if constexpr (NT)
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
    else
        *reinterpret_cast<u32x4*>(p) = v;
}

// bf16 element 2m of a 32-bit word sits in its low half (little endian).
__device__ __forceinline__ float bf16_low(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_high(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// binary32 -> bf16, round to nearest, ties to even.  Adding 0x7FFF plus the
// lowest kept bit carries into the kept half exactly when the dropped half
// is above one half, or equal to it with an odd kept half; a carry out of
// the significand steps the exponent, and past the largest finite value it
// gives the infinity encoding.  NaNs become quiet NaNs keeping sign and the
// top payload bits.
__device__ __forceinline__ uint32_t to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    const uint32_t rounded = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    const uint32_t quiet_nan = (u >> 16) | 0x40u;
    return (u & 0x7FFFFFFFu) > 0x7F800000u ? quiet_nan : rounded;
}

__device__ __forceinline__ char* dst_ptr(const ExecArgs& a, const purlin_desc& d, uint32_t j) {
    return a.bufs[d.dst_buf + j * d.dst_step] + d.dst_off;
}

// Bytes [from, to) of an item, 2 bytes per lane step (every element width
// and offset here is a multiple of 2).
__device__ __forceinline__ void copy_bytes2(const ExecArgs& a, const purlin_desc& d, const char* src, uint64_t from,
                                            uint64_t to, uint32_t lane) {
    for (uint64_t b = from + 2 * lane; b < to; b += 2 * kWave) {
        const uint16_t v = *reinterpret_cast<const uint16_t*>(src + b);
        for (uint32_t j = 0; j < d.ndst; ++j) *reinterpret_cast<uint16_t*>(dst_ptr(a, d, j) + b) = v;
    }
}

// One COPY work item, executed by the whole wave.
template <int U, bool NTL, bool NTS>
__device__ __forceinline__ void run_copy(const ExecArgs& a, const purlin_desc& d, uint32_t lane) {
    const char* src = a.bufs[d.src_buf] + d.src_off;
    if (((d.src_off | d.dst_off) & 15) != 0) {
        copy_bytes2(a, d, src, 0, d.bytes, lane);
        return;
    }
    const uint64_t nvec = d.bytes >> 4;
    uint64_t base = 0;
    for (; base + U * kWave <= nvec; base += U * kWave) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = load16<NTL>(src + (base + u * kWave + lane) * 16);
        for (uint32_t j = 0; j < d.ndst; ++j) {
            char* dst = dst_ptr(a, d, j);
#pragma unroll
            for (int u = 0; u < U; ++u) store16<NTS>(dst + (base + u * kWave + lane) * 16, v[u]);
        }
    }
    for (uint64_t i = base + lane; i < nvec; i += kWave) {
        const u32x4 v = load16<NTL>(src + i * 16);
        for (uint32_t j = 0; j < d.ndst; ++j) store16<NTS>(dst_ptr(a, d, j) + i * 16, v);
    }
    copy_bytes2(a, d, src, nvec * 16, d.bytes, lane);
}

template <int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void exec_copy(ExecArgs a) {
    // One item per wave unless the grid is capped (then the waves stride).
    // Items are taken last to first: a copy phase usually reads what a
    // reduce phase (AllReduce's first phase, or a ReduceScatter called just
    // before an AllGather) wrote first to last, so its last-written chunks,
    // the ones still in the 256 MB last-level cache, are read before the
    // cache turns over (read in the order written, a buffer a little larger
    // than the cache misses on every line).  Measured on MI355X, P = 8,
    // bf16, 256 MiB per rank: AllGather after ReduceScatter 385-390 ->
    // 365 us, AllReduce 755 -> 741 us; the order does not change the result.
    for (uint64_t i = wave_index(); i < a.n_items; i += a.wave_stride) {
        const purlin_desc d = a.items[a.n_items - 1 - i];
        run_copy<U, NTL, NTS>(a, d, lane_index());
    }
}

// Eq. 2 on one 16-byte vector of every source: 8 bf16 or 4 fp32 elements.
template <int NSRC, bool BF16>
__device__ __forceinline__ u32x4 rank_order_sum(const u32x4 (&v)[NSRC]) {
    u32x4 o;
    if constexpr (BF16) {
        float acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
#pragma unroll
        for (int p = 0; p < NSRC; ++p) {
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                acc[2 * m] = acc[2 * m] + bf16_low(v[p][m]);
                acc[2 * m + 1] = acc[2 * m + 1] + bf16_high(v[p][m]);
            }
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) o[m] = to_bf16(acc[2 * m]) | (to_bf16(acc[2 * m + 1]) << 16);
    } else {
        float acc[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) acc[m] = 0.0f;
#pragma unroll
        for (int p = 0; p < NSRC; ++p) {
#pragma unroll
            for (int m = 0; m < 4; ++m) acc[m] = acc[m] + __uint_as_float(v[p][m]);
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) o[m] = __float_as_uint(acc[m]);
    }
    return o;
}

// Element-at-a-time reduction of bytes [from, to) of an item.
template <int NSRC, bool BF16>
__device__ __forceinline__ void reduce_elems(const ExecArgs& a, const purlin_desc& d, const char* const (&src)[NSRC],
                                             uint64_t from, uint64_t to, uint32_t lane) {
    constexpr uint64_t S = BF16 ? 2 : 4;
    for (uint64_t b = from + S * lane; b < to; b += S * kWave) {
        float acc = 0.0f;
#pragma unroll
        for (int p = 0; p < NSRC; ++p) {
            const float x = BF16 ? __uint_as_float(uint32_t(*reinterpret_cast<const uint16_t*>(src[p] + b)) << 16)
                                 : *reinterpret_cast<const float*>(src[p] + b);
            acc = acc + x;
        }
        for (uint32_t j = 0; j < d.ndst; ++j) {
            char* dst = dst_ptr(a, d, j) + b;
            if constexpr (BF16)
                *reinterpret_cast<uint16_t*>(dst) = static_cast<uint16_t>(to_bf16(acc));
            else
                *reinterpret_cast<float*>(dst) = acc;
        }
    }
}

// One REDUCE work item, executed by the whole wave.
template <int NSRC, bool BF16, int U, bool NTL, bool NTS>
__device__ __forceinline__ void run_reduce(const ExecArgs& a, const purlin_desc& d, uint32_t lane) {
    const char* src[NSRC];
#pragma unroll
    for (int p = 0; p < NSRC; ++p) src[p] = a.srcs[p] + d.src_off;
    // Unaligned items, and bf16 items of fewer than 12 vectors, go element
    // by element: a wavefront with at most 8 of its lanes active runs the
    // bf16 widening and rounding about 0.8 us slower (measured on MI355X,
    // P = 8: 128-byte items 2.5 us, 192-byte items 1.8 us per graph-replayed
    // call; the same 128 bytes over 16 or 64 lanes 1.65 us).
    if (((d.src_off | d.dst_off) & 15) != 0 || (BF16 && d.bytes < 12 * 16)) {
        reduce_elems<NSRC, BF16>(a, d, src, 0, d.bytes, lane);
        return;
    }
    const uint64_t nvec = d.bytes >> 4;
    uint64_t base = 0;
    for (; base + U * kWave <= nvec; base += U * kWave) {
        u32x4 v[U][NSRC];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int p = 0; p < NSRC; ++p) v[u][p] = load16<NTL>(src[p] + (base + u * kWave + lane) * 16);
        u32x4 o[U];
#pragma unroll
        for (int u = 0; u < U; ++u) o[u] = rank_order_sum<NSRC, BF16>(v[u]);
        for (uint32_t j = 0; j < d.ndst; ++j) {
            char* dst = dst_ptr(a, d, j);
#pragma unroll
            for (int u = 0; u < U; ++u) store16<NTS>(dst + (base + u * kWave + lane) * 16, o[u]);
        }
    }
    for (uint64_t i = base + lane; i < nvec; i += kWave) {
        u32x4 v[NSRC];
#pragma unroll
        for (int p = 0; p < NSRC; ++p) v[p] = load16<NTL>(src[p] + i * 16);
        const u32x4 o = rank_order_sum<NSRC, BF16>(v);
        for (uint32_t j = 0; j < d.ndst; ++j) store16<NTS>(dst_ptr(a, d, j) + i * 16, o);
    }
    reduce_elems<NSRC, BF16>(a, d, src, nvec * 16, d.bytes, lane);
}

template <int NSRC, bool BF16, int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void exec_reduce(ExecArgs a) {
    for (uint64_t i = wave_index(); i < a.n_items; i += a.wave_stride) {
        const purlin_desc d = a.items[i];
        run_reduce<NSRC, BF16, U, NTL, NTS>(a, d, lane_index());
    }
}

// ---------------------------------------------------------------------------
// Single-launch AllReduce: compose<ReduceScatter, AllGather> with the gather
// of each chunk released by the completion of that chunk's reduction
// (Algorithm 1's reduce and gather roles, notify and consume of Section 3.2)
// inside one launch.  All ranks share one address space, so there is no
// staging; the notification is a per-chunk counter of finished reduce items.
//
// * Items are split into 8 partitions like the waves (item i and wave w in
//   partition (i / 4) % 8 and (w / 4) % 8, so every partition has as many
//   waves as items), and the waves of a partition claim its items in table
//   order through the partition's ticket counter.  Every reduce item
//   precedes every copy item in the table, so in each partition the reduce
//   items are claimed first, by running waves, and reduce items never wait;
//   a copy waits only for reduce items, which are therefore all claimed
//   (in every partition) or running.  Every wait ends.  Eight counters
//   spread the claims (one device-scope atomic each, about 12-15 ns apart on
//   one address under contention).
// * Nothing is ever reset (the epochs of Section 4.2).  Each launch has
//   exactly n waves and each claims one ticket, and launches of a plan are
//   ordered on its stream, so launch e's tickets of partition k are
//   [e*nk, (e+1)*nk): the ticket gives both the epoch and the item.  Chunk
//   (k, c) is ready in launch e when its cumulative counter reaches
//   (e + 1) * (its reduce items).
// * Publication without L2 write-backs: the 8 XCDs' L2 caches are not
//   coherent with each other, so a reduced chunk is written with the sc1
//   (device-coherent, write-through) policy and read back by its copies
//   with the same policy; a reduce wave waits for its own stores to
//   complete before it bumps the chunk's counter.  Items with bytes outside
//   whole 16-byte vectors (unaligned or short) take the plain paths with an
//   agent-scope release (an L2 write-back) or acquire (an L2 invalidation),
//   the design this replaced for every item: measured on MI355X (P = 8,
//   bf16, 256 MiB per rank, 32 KiB items) 1346 -> 810 us.
// * Waits are bounded: a wave that waits longer than kSpinLimit sleeps
//   records an error in the state block and gives up its item, so the
//   launch always drains (and the epochs stay consistent).
struct FusedArgs {
    FusedState* state;
    uint64_t* ready;         // [P * chunks_per_part] finished reduce items, cumulative
    uint64_t n_reduce;       // items [0, n_reduce) reduce, the rest copy
    uint64_t part_bytes;     // partition bytes
    uint64_t chunk_bytes;
    uint64_t item_bytes;     // cut size of the reduce items
    uint64_t chunks_per_part;
};

constexpr uint32_t kSpinLimit = 1u << 24;

__device__ __forceinline__ uint64_t reduce_items_of_chunk(const FusedArgs& f, uint32_t c) {
    const uint64_t off = uint64_t(c) * f.chunk_bytes;
    const uint64_t len = min(f.chunk_bytes, f.part_bytes - off);
    return (len + f.item_bytes - 1) / f.item_bytes;
}

// 16-byte accesses with the sc1 (device-coherent) cache policy, through a
// raw buffer resource over [base, base + bytes) (bytes < 2^31).  Word 3 of
// the resource selects 32-bit data for untyped (raw) accesses on gfx9-family
// chips; the last argument of the access is its cache policy, sc1 = 16.
constexpr int kRawBufferWord3 = 0x00020000;
constexpr int kPolicySc1 = 16;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coh_rsrc(const char* base, uint64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), 0, static_cast<int>(bytes), kRawBufferWord3);
}
__device__ __forceinline__ void store16_coh(__amdgpu_buffer_rsrc_t r, uint64_t off, u32x4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(v, r, static_cast<int>(off), 0, kPolicySc1);
}
__device__ __forceinline__ u32x4 load16_coh(__amdgpu_buffer_rsrc_t r, uint64_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, kPolicySc1);
}
// Reduce item, whole 16-byte vectors only, written through to the coherence point.
template <int NSRC, bool BF16, int U, bool NTL>
__device__ __forceinline__ void run_reduce_coh(const ExecArgs& a, const purlin_desc& d, uint32_t lane) {
    const char* src[NSRC];
#pragma unroll
    for (int p = 0; p < NSRC; ++p) src[p] = a.srcs[p] + d.src_off;
    const uint64_t nvec = d.bytes >> 4;
    uint64_t base = 0;
    for (; base + U * kWave <= nvec; base += U * kWave) {
        u32x4 v[U][NSRC];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int p = 0; p < NSRC; ++p) v[u][p] = load16<NTL>(src[p] + (base + u * kWave + lane) * 16);
        u32x4 o[U];
#pragma unroll
        for (int u = 0; u < U; ++u) o[u] = rank_order_sum<NSRC, BF16>(v[u]);
        for (uint32_t j = 0; j < d.ndst; ++j) {
            const __amdgpu_buffer_rsrc_t r = coh_rsrc(dst_ptr(a, d, j), d.bytes);
#pragma unroll
            for (int u = 0; u < U; ++u) store16_coh(r, (base + u * kWave + lane) * 16, o[u]);
        }
    }
    for (uint64_t i = base + lane; i < nvec; i += kWave) {
        u32x4 v[NSRC];
#pragma unroll
        for (int p = 0; p < NSRC; ++p) v[p] = load16<NTL>(src[p] + i * 16);
        const u32x4 o = rank_order_sum<NSRC, BF16>(v);
        for (uint32_t j = 0; j < d.ndst; ++j) store16_coh(coh_rsrc(dst_ptr(a, d, j), d.bytes), i * 16, o);
    }
}
// Copy item, whole 16-byte vectors only, its source read at the coherence point.
template <int U, bool NTS>
__device__ __forceinline__ void run_copy_coh(const ExecArgs& a, const purlin_desc& d, uint32_t lane) {
    const __amdgpu_buffer_rsrc_t rs = coh_rsrc(a.bufs[d.src_buf] + d.src_off, d.bytes);
    const uint64_t nvec = d.bytes >> 4;
    uint64_t base = 0;
    for (; base + U * kWave <= nvec; base += U * kWave) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = load16_coh(rs, (base + u * kWave + lane) * 16);
        for (uint32_t j = 0; j < d.ndst; ++j) {
            char* dst = dst_ptr(a, d, j);
#pragma unroll
            for (int u = 0; u < U; ++u) store16<NTS>(dst + (base + u * kWave + lane) * 16, v[u]);
        }
    }
    for (uint64_t i = base + lane; i < nvec; i += kWave) {
        const u32x4 v = load16_coh(rs, i * 16);
        for (uint32_t j = 0; j < d.ndst; ++j) store16<NTS>(dst_ptr(a, d, j) + i * 16, v);
    }
}

template <int NSRC, bool BF16, bool STREAM>
__global__ __launch_bounds__(kBlock) void exec_fused_allreduce(ExecArgs a, FusedArgs f) {
    const uint32_t w = wave_index();
    if (w >= a.n_items) return;  // exactly n_items waves claim
    const uint32_t lane = lane_index();
    FusedState* st = f.state;
    const uint64_t n = a.n_items;
    const uint32_t k = (w / kWavesPerBlock) % 8;
    const uint64_t full = n / 32, rem = n % 32;
    const uint64_t nk = full * 4 + (rem > uint64_t(k) * 4 ? min(rem - uint64_t(k) * 4, uint64_t(4)) : 0);
    uint64_t ticket = 0;
    if (lane == 0) ticket = __hip_atomic_fetch_add(&st->tickets[k * 16], 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    ticket = static_cast<uint64_t>(readlane64(static_cast<int64_t>(ticket), 0));
    const uint64_t epoch = ticket / nk;
    const uint64_t jj = ticket - epoch * nk;
    const uint64_t i = ((jj / 4) * 8 + k) * 4 + jj % 4;
    {
        const purlin_desc d = a.items[i];
        uint64_t* ready = f.ready + uint64_t(d.part) * f.chunks_per_part + d.chunk;
        const bool whole = ((d.src_off | d.dst_off | d.bytes) & 15) == 0 && !(BF16 && d.bytes < 12 * 16) &&
                           d.bytes < (uint64_t(1) << 31);
        if (i < f.n_reduce) {
            if (whole) {
                run_reduce_coh<NSRC, BF16, reduce_unroll(NSRC), STREAM>(a, d, lane);
                __builtin_amdgcn_s_waitcnt(0);  // the write-through stores have completed
            } else {
                run_reduce<NSRC, BF16, reduce_unroll(NSRC), STREAM, false>(a, d, lane);
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            }
            if (lane == 0) __hip_atomic_fetch_add(ready, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            const uint64_t target = (epoch + 1) * reduce_items_of_chunk(f, d.chunk);
            uint32_t spins = 0;
            bool ok = true;
            while (__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(
                       __hip_atomic_load(ready, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target))) {
                if (++spins > kSpinLimit) {
                    ok = false;
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
            }
            if (ok && whole) {
                run_copy_coh<kCopyUnroll, STREAM>(a, d, lane);
            } else if (ok) {
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                run_copy<kCopyUnroll, false, STREAM>(a, d, lane);
            } else if (lane == 0) {
                __hip_atomic_store(&st->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
}


template <int NSRC, bool BF16>
void launch_reduce_hints(dim3 grid, hipStream_t stream, const ExecArgs& a, bool ntl, bool nts) {
    constexpr int U = reduce_unroll(NSRC);
    if (ntl && nts)
        hipLaunchKernelGGL((exec_reduce<NSRC, BF16, U, true, true>), grid, dim3(kBlock), 0, stream, a);
    else if (ntl)
        hipLaunchKernelGGL((exec_reduce<NSRC, BF16, U, true, false>), grid, dim3(kBlock), 0, stream, a);
    else if (nts)
        hipLaunchKernelGGL((exec_reduce<NSRC, BF16, U, false, true>), grid, dim3(kBlock), 0, stream, a);
    else
        hipLaunchKernelGGL((exec_reduce<NSRC, BF16, U, false, false>), grid, dim3(kBlock), 0, stream, a);
}

template <int NSRC>
void launch_reduce(dim3 grid, hipStream_t stream, const ExecArgs& a, bool bf16, bool ntl, bool nts) {
    if (bf16)
        launch_reduce_hints<NSRC, true>(grid, stream, a, ntl, nts);
    else
        launch_reduce_hints<NSRC, false>(grid, stream, a, ntl, nts);
}

template <int U>
void launch_copy_u(dim3 grid, hipStream_t stream, const ExecArgs& a, bool ntl, bool nts) {
    if (ntl && nts)
        hipLaunchKernelGGL((exec_copy<U, true, true>), grid, dim3(kBlock), 0, stream, a);
    else if (ntl)
        hipLaunchKernelGGL((exec_copy<U, true, false>), grid, dim3(kBlock), 0, stream, a);
    else if (nts)
        hipLaunchKernelGGL((exec_copy<U, false, true>), grid, dim3(kBlock), 0, stream, a);
    else
        hipLaunchKernelGGL((exec_copy<U, false, false>), grid, dim3(kBlock), 0, stream, a);
}

// `depth`: 16-byte loads in flight per lane (1, 2, 4, 8; 0 = kCopyUnroll).
void launch_copy(dim3 grid, hipStream_t stream, const ExecArgs& a, bool ntl, bool nts, uint32_t depth) {
    switch (depth) {
        case 1: launch_copy_u<1>(grid, stream, a, ntl, nts); break;
        case 2: launch_copy_u<2>(grid, stream, a, ntl, nts); break;
        case 8: launch_copy_u<8>(grid, stream, a, ntl, nts); break;
        default: launch_copy_u<kCopyUnroll>(grid, stream, a, ntl, nts); break;
    }
}

// ---------------------------------------------------------------------------
// Variable-size collectives (the V layouts of Section 3.1): partition sizes
// are read from device memory at run time.  The work items cover a fixed
// virtual index space sized by the plan's capacity; each wave maps its range
// onto (source, destination, offset) from prefix sums over at most 16
// counts (P x P for AllToAllV), which every wave forms in registers.  Sizes
// that are negative or exceed the capacity make every wave skip the call
// (all waves reach the same verdict); wave 0 reports it.
// ---------------------------------------------------------------------------
struct VArgs {
    const int32_t* counts;  // P (AllGatherV, ReduceScatterV) or P*P row-major (AllToAllV)
    int32_t* status;        // optional: 0, or 1 for invalid sizes
    uint64_t in_cap;        // elements every input holds
    uint64_t out_cap;       // elements every output holds
    uint64_t unit;          // elements per count
    uint32_t P;
    uint32_t elem_bytes;
    uint32_t transposed;  // AllToAllV: counts are column-major
    uint32_t src_major;   // AllToAllV: items cover each source's input
};

// Lane p < P holds count p (elements); returns whether every count is >= 0
// and fits `part_cap`, and their sum fits `total_cap`.
__device__ __forceinline__ bool load_counts(const VArgs& v, uint32_t lane, int64_t part_cap, int64_t total_cap,
                                            int64_t& c) {
    c = 0;
    if (lane < v.P) c = static_cast<int64_t>(v.counts[lane]) * static_cast<int64_t>(v.unit);
    bool ok = true;
    int64_t total = 0;  // each term is checked against a capacity first, so this cannot overflow
    for (uint32_t p = 0; p < v.P; ++p) {
        const int64_t cp = readlane64(c, p);
        const bool fits = cp >= 0 && cp <= part_cap;
        ok = ok && fits;
        total += fits ? cp : 0;
    }
    return ok && total <= total_cap;
}

__device__ __forceinline__ void report(const VArgs& v, uint32_t w, uint32_t lane, bool ok) {
    if (w == 0 && lane == 0 && v.status) *v.status = ok ? 0 : 1;
}

// The items of a variable-size plan cover every space's full capacity; only
// those that start below the space's run-time extent carry data.  A space's
// items are its chunks cut at `item` bytes, so how many start below an
// extent follows in closed form, and a fixed grid of waves strides over
// just those (the sizes are read once per wave, the AllToAllV matrix once
// per workgroup).
struct VGrid {
    uint64_t chunk;      // chunk bytes of the virtual space
    uint64_t item;       // work-item bytes (chunks are cut at this size)
    uint64_t per_chunk;  // items per full chunk
    uint64_t per_space;  // items per space (every space is cut alike)
    uint32_t waves;      // waves in the launch: the grid stride
};

__device__ __forceinline__ uint64_t active_items(const VGrid& g, uint64_t extent_bytes) {
    if (extent_bytes == 0) return 0;
    const uint64_t o = extent_bytes - 1;
    return min(g.per_space, (o / g.chunk) * g.per_chunk + (o % g.chunk) / g.item + 1);
}

// The first item of wave w is item w (when the run-time sizes make it
// active): its descriptor is loaded before the sizes are known, so that the
// wave's data loads wait on one memory round trip, not two.
__device__ __forceinline__ purlin_desc first_item(const ExecArgs& a, uint32_t w) {
    purlin_desc d{};
    if (w < a.n_items) d = a.items[w];
    return d;
}

template <bool STREAM>
__global__ __launch_bounds__(kBlock) void exec_allgatherv(ExecArgs a, VArgs v, VGrid g) {
    const uint32_t w = wave_index();
    if (w >= g.waves) return;
    const uint32_t lane = lane_index();
    const purlin_desc d0 = first_item(a, w);
    int64_t c;
    const bool ok = load_counts(v, lane, static_cast<int64_t>(v.in_cap), static_cast<int64_t>(v.out_cap), c);
    report(v, w, lane, ok);
    if (!ok) return;
    const uint64_t s = v.elem_bytes;
    int64_t total = 0;
    for (uint32_t p = 0; p < v.P; ++p) total += readlane64(c, p);
    const uint64_t n = active_items(g, uint64_t(total) * s);
    for (uint64_t i = w; i < n; i += g.waves) {
        const purlin_desc d = i == w ? d0 : a.items[i];
        const int64_t lo_v = static_cast<int64_t>(d.src_off / s), hi_v = lo_v + static_cast<int64_t>(d.bytes / s);
        int64_t off = 0;
        for (uint32_t p = 0; p < v.P; ++p) {
            const int64_t cp = readlane64(c, p);
            const int64_t x = max(lo_v, off), y = min(hi_v, off + cp);
            if (x < y) {
                purlin_desc sub = d;
                sub.src_buf = p;
                sub.ndst = v.P;
                sub.dst_buf = v.P;
                sub.dst_step = 1;
                sub.src_off = uint64_t(x - off) * s;
                sub.dst_off = uint64_t(x) * s;
                sub.bytes = uint64_t(y - x) * s;
                run_copy<kCopyUnroll, false, STREAM>(a, sub, lane);
            }
            off += cp;
        }
    }
}

template <int NSRC, bool BF16, bool STREAM>
__global__ __launch_bounds__(kBlock) void exec_reducescatterv(ExecArgs a, VArgs v, VGrid g) {
    const uint32_t w = wave_index();
    if (w >= g.waves) return;
    const uint32_t lane = lane_index();
    const purlin_desc d0 = first_item(a, w);
    int64_t c;
    const bool ok = load_counts(v, lane, static_cast<int64_t>(v.out_cap), static_cast<int64_t>(v.in_cap), c);
    report(v, w, lane, ok);
    if (!ok) return;
    const uint64_t s = v.elem_bytes;
    int64_t total = 0;
    for (uint32_t r = 0; r < v.P; ++r) total += readlane64(c, r);
    const uint64_t n = active_items(g, uint64_t(total) * s);
    for (uint64_t i = w; i < n; i += g.waves) {
        const purlin_desc d = i == w ? d0 : a.items[i];
        const int64_t lo_v = static_cast<int64_t>(d.src_off / s), hi_v = lo_v + static_cast<int64_t>(d.bytes / s);
        int64_t off = 0;
        for (uint32_t r = 0; r < v.P; ++r) {
            const int64_t cr = readlane64(c, r);
            const int64_t x = max(lo_v, off), y = min(hi_v, off + cr);
            if (x < y) {
                purlin_desc sub = d;
                sub.ndst = 1;
                sub.dst_buf = v.P + r;
                sub.dst_step = 0;
                sub.src_off = uint64_t(x) * s;
                sub.dst_off = uint64_t(x - off) * s;
                sub.bytes = uint64_t(y - x) * s;
                run_reduce<NSRC, BF16, reduce_unroll(NSRC), STREAM, false>(a, sub, lane);
            }
            off += cr;
        }
    }
}

// AllToAllV.  counts[p * P + r] = elements rank p sends to rank r
// (counts[r * P + p] when transposed).  Space k is destination k's output,
// whose pieces come from the sources in rank order, or (source-major)
// source k's input, whose pieces go to the destinations in rank order; an
// item covers bytes [src_off, src_off + bytes) of space d.part.  The P x P
// sizes are staged once per workgroup in LDS, row-major; lane q checks row
// q (what q sends) and column q (what q receives), and for each item forms
// piece q of the item's space: its length and where it starts on the other
// side.
template <bool STREAM>
__global__ __launch_bounds__(kBlock) void exec_alltoallv(ExecArgs a, VArgs v, VGrid g) {
    __shared__ int64_t m[PURLIN_MAX_RANKS * PURLIN_MAX_RANKS];
    const uint32_t P = v.P;
    const int64_t unit = static_cast<int64_t>(v.unit);
    for (uint32_t i = threadIdx.x; i < P * P; i += kBlock) {
        const uint32_t src = v.transposed ? (i % P) * P + i / P : i;
        m[i] = static_cast<int64_t>(v.counts[src]) * unit;
    }
    __syncthreads();
    const uint32_t w = wave_index();
    if (w >= g.waves) return;
    const uint32_t lane = lane_index();
    const bool src_major = v.src_major != 0;
    const int64_t in_cap = static_cast<int64_t>(v.in_cap), out_cap = static_cast<int64_t>(v.out_cap);
    const int64_t cap = max(in_cap, out_cap);
    bool ok = true;
    int64_t extent = 0;  // lane q: elements in space q
    if (lane < P) {
        int64_t row = 0, col = 0;  // each term is checked against a capacity first: no overflow
        for (uint32_t j = 0; j < P; ++j) {
            int64_t x = m[lane * P + j];
            if (x < 0 || x > cap) {
                ok = false;
                x = 0;
            }
            row += x;
            int64_t y = m[j * P + lane];
            if (y < 0 || y > cap) y = 0;  // reported by lane j's row
            col += y;
        }
        ok = ok && row <= in_cap && col <= out_cap;
        extent = src_major ? row : col;
    }
    const bool all_ok = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(__all(ok)));
    report(v, w, lane, all_ok);
    if (!all_ok) return;
    const uint64_t s = v.elem_bytes;
    // active items per space, and their exclusive prefix over spaces
    const uint64_t act = lane < P ? active_items(g, uint64_t(extent) * s) : 0;
    uint64_t before = 0, n = 0;
    for (uint32_t q = 0; q < P; ++q) {
        const uint64_t aq = static_cast<uint64_t>(readlane64(static_cast<int64_t>(act), q));
        if (q < lane) before += aq;
        n += aq;
    }
    for (uint64_t i = w; i < n; i += g.waves) {
        // space k: the number of spaces that end at or before active item i
        const uint32_t k = __popcll(__ballot(lane < P && before + act <= i));
        const uint64_t first = static_cast<uint64_t>(readlane64(static_cast<int64_t>(before), k));
        const purlin_desc d = a.items[uint64_t(k) * g.per_space + (i - first)];
        // piece `lane` of space k: destination-major, source lane's part for
        // k (m[lane][k]) starting at sum_{j<k} m[lane][j] in in_lane;
        // source-major, k's part for destination lane (m[k][lane]) landing at
        // sum_{j<k} m[j][lane] in out_lane
        int64_t other = 0, c = 0;
        if (lane < P) {
            for (uint32_t j = 0; j < P; ++j) {
                const int64_t e = src_major ? m[j * P + lane] : m[lane * P + j];
                if (j < k) other += e;
                if (j == k) c = e;
            }
        }
        const int64_t lo_v = static_cast<int64_t>(d.src_off / s), hi_v = lo_v + static_cast<int64_t>(d.bytes / s);
        int64_t base = 0;
        for (uint32_t q = 0; q < P; ++q) {
            const int64_t cq = readlane64(c, q), oq = readlane64(other, q);
            const int64_t x = max(lo_v, base), y = min(hi_v, base + cq);
            if (x < y) {
                purlin_desc sub = d;
                sub.ndst = 1;
                sub.dst_step = 0;
                if (src_major) {
                    sub.src_buf = k;
                    sub.dst_buf = P + q;
                    sub.src_off = uint64_t(x) * s;
                    sub.dst_off = uint64_t(oq + (x - base)) * s;
                } else {
                    sub.src_buf = q;
                    sub.dst_buf = P + k;
                    sub.src_off = uint64_t(oq + (x - base)) * s;
                    sub.dst_off = uint64_t(x) * s;
                }
                sub.bytes = uint64_t(y - x) * s;
                run_copy<kCopyUnroll, STREAM, STREAM>(a, sub, lane);
            }
            base += cq;
        }
    }
}

template <int NSRC>
void launch_fused_n(dim3 grid, hipStream_t stream, const ExecArgs& a, const FusedArgs& f, bool bf16, bool stream_hint) {
    if (bf16) {
        if (stream_hint)
            hipLaunchKernelGGL((exec_fused_allreduce<NSRC, true, true>), grid, dim3(kBlock), 0, stream, a, f);
        else
            hipLaunchKernelGGL((exec_fused_allreduce<NSRC, true, false>), grid, dim3(kBlock), 0, stream, a, f);
    } else {
        if (stream_hint)
            hipLaunchKernelGGL((exec_fused_allreduce<NSRC, false, true>), grid, dim3(kBlock), 0, stream, a, f);
        else
            hipLaunchKernelGGL((exec_fused_allreduce<NSRC, false, false>), grid, dim3(kBlock), 0, stream, a, f);
    }
}

}  // namespace

hipError_t launch_fused_allreduce(const purlin_desc* items, uint64_t n, uint64_t n_reduce, uint32_t nsrc,
                                  purlin_dtype dtype, bool streaming, void* const* bufs, int nbufs, FusedState* state,
                                  uint64_t* ready, uint64_t part_bytes, uint64_t chunk_bytes, uint64_t item_bytes,
                                  uint64_t chunks_per_part, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    if (n >= (uint64_t(1) << 32)) return hipErrorInvalidValue;
    ExecArgs a{};
    a.items = items;
    a.n_items = n;
    for (int i = 0; i < nbufs && i < 2 * PURLIN_MAX_RANKS; ++i) a.bufs[i] = static_cast<char*>(bufs[i]);
    for (uint32_t p = 0; p < nsrc && p < PURLIN_MAX_RANKS; ++p) a.srcs[p] = static_cast<char*>(bufs[p]);
    FusedArgs f{state, ready, n_reduce, part_bytes, chunk_bytes, item_bytes, chunks_per_part};
    const dim3 grid(static_cast<uint32_t>((n + kWavesPerBlock - 1) / kWavesPerBlock));
    const bool bf16 = dtype == PURLIN_BF16;
    (void)hipGetLastError();
    switch (nsrc) {
#define PURLIN_FUSED_CASE(k) \
    case k: launch_fused_n<k>(grid, stream, a, f, bf16, streaming); break;
        PURLIN_FUSED_CASE(1) PURLIN_FUSED_CASE(2) PURLIN_FUSED_CASE(3) PURLIN_FUSED_CASE(4)
        PURLIN_FUSED_CASE(5) PURLIN_FUSED_CASE(6) PURLIN_FUSED_CASE(7) PURLIN_FUSED_CASE(8)
        PURLIN_FUSED_CASE(9) PURLIN_FUSED_CASE(10) PURLIN_FUSED_CASE(11) PURLIN_FUSED_CASE(12)
        PURLIN_FUSED_CASE(13) PURLIN_FUSED_CASE(14) PURLIN_FUSED_CASE(15) PURLIN_FUSED_CASE(16)
#undef PURLIN_FUSED_CASE
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_v(purlin_op op, const purlin_desc* items, uint64_t n, int P, purlin_dtype dtype, bool streaming,
                    void* const* bufs, const int32_t* counts, bool counts_transposed, bool source_major,
                    int32_t* status, uint64_t in_capacity, uint64_t out_capacity, uint64_t unit, uint64_t chunk,
                    uint64_t item_bytes, uint32_t spaces, uint32_t max_workgroups, hipStream_t stream) {
    if (chunk == 0 || item_bytes == 0 || spaces == 0 || n % spaces != 0) return hipErrorInvalidValue;
    ExecArgs a{};
    a.items = items;
    a.n_items = n;
    for (int i = 0; i < 2 * P && i < 2 * PURLIN_MAX_RANKS; ++i) a.bufs[i] = static_cast<char*>(bufs[i]);
    for (int p = 0; p < P && p < PURLIN_MAX_RANKS; ++p) a.srcs[p] = static_cast<char*>(bufs[p]);
    VArgs v{counts, status, in_capacity, out_capacity, unit, static_cast<uint32_t>(P), dtype == PURLIN_FP32 ? 4u : 2u,
            counts_transposed ? 1u : 0u, source_major ? 1u : 0u};
    // Waves stride over the active items.  Measured on MI355X (P = 8,
    // 256 MiB/rank and the expert-parallel exchanges): copies run best with
    // a grid of half as many waves as items -- as fast as one wave per item
    // when the sizes fill the capacity, and 1.4x faster when they fill 40%
    // of it (fewer waves that find nothing) -- while ReduceScatterV, whose
    // waves carry P loads per vector, runs best with one wave per item.  At
    // least one wave: it validates the sizes and writes the status even
    // when the plan has no items (zero capacity).
    const uint64_t per_wave = op == PURLIN_REDUCE_SCATTERV ? 1 : 2;
    uint64_t waves = std::max<uint64_t>(1, (n + per_wave - 1) / per_wave);
    if (max_workgroups) waves = std::min<uint64_t>(waves, uint64_t(max_workgroups) * kWavesPerBlock);
    VGrid g{chunk, item_bytes, (chunk + item_bytes - 1) / item_bytes, n / spaces, static_cast<uint32_t>(waves)};
    const dim3 grid(static_cast<uint32_t>((waves + kWavesPerBlock - 1) / kWavesPerBlock));
    const bool bf16 = dtype == PURLIN_BF16;
    (void)hipGetLastError();
    if (op == PURLIN_ALLGATHERV) {
        if (streaming)
            hipLaunchKernelGGL((exec_allgatherv<true>), grid, dim3(kBlock), 0, stream, a, v, g);
        else
            hipLaunchKernelGGL((exec_allgatherv<false>), grid, dim3(kBlock), 0, stream, a, v, g);
    } else if (op == PURLIN_ALLTOALLV) {
        if (streaming)
            hipLaunchKernelGGL((exec_alltoallv<true>), grid, dim3(kBlock), 0, stream, a, v, g);
        else
            hipLaunchKernelGGL((exec_alltoallv<false>), grid, dim3(kBlock), 0, stream, a, v, g);
    } else if (op == PURLIN_REDUCE_SCATTERV) {
        switch (P) {
#define PURLIN_RSV_CASE(k)                                                                                      \
    case k:                                                                                                     \
        if (bf16 && streaming)                                                                                  \
            hipLaunchKernelGGL((exec_reducescatterv<k, true, true>), grid, dim3(kBlock), 0, stream, a, v, g);     \
        else if (bf16)                                                                                          \
            hipLaunchKernelGGL((exec_reducescatterv<k, true, false>), grid, dim3(kBlock), 0, stream, a, v, g);    \
        else if (streaming)                                                                                     \
            hipLaunchKernelGGL((exec_reducescatterv<k, false, true>), grid, dim3(kBlock), 0, stream, a, v, g);    \
        else                                                                                                    \
            hipLaunchKernelGGL((exec_reducescatterv<k, false, false>), grid, dim3(kBlock), 0, stream, a, v, g);   \
        break;
            PURLIN_RSV_CASE(1) PURLIN_RSV_CASE(2) PURLIN_RSV_CASE(3) PURLIN_RSV_CASE(4)
            PURLIN_RSV_CASE(5) PURLIN_RSV_CASE(6) PURLIN_RSV_CASE(7) PURLIN_RSV_CASE(8)
            PURLIN_RSV_CASE(9) PURLIN_RSV_CASE(10) PURLIN_RSV_CASE(11) PURLIN_RSV_CASE(12)
            PURLIN_RSV_CASE(13) PURLIN_RSV_CASE(14) PURLIN_RSV_CASE(15) PURLIN_RSV_CASE(16)
#undef PURLIN_RSV_CASE
            default: return hipErrorInvalidValue;
        }
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

namespace {

// A plain 16-byte copy with no descriptors: each lane moves kCopyUnroll
// vectors 256 lanes apart, one workgroup 16 KiB.  It is the reference
// stream for the executor's copies.
__global__ __launch_bounds__(kBlock) void stream_copy(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                     uint64_t nvec) {
    const uint64_t base = uint64_t(blockIdx.x) * (kBlock * kCopyUnroll) + threadIdx.x;
    u32x4 v[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
        const uint64_t i = base + uint64_t(u) * kBlock;
        if (i < nvec) v[u] = src[i];
    }
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
        const uint64_t i = base + uint64_t(u) * kBlock;
        if (i < nvec) dst[i] = v[u];
    }
}

// Reference streams (not steps of the method): every 16-byte vector i of
// the range is the XOR of the NS sources' vectors i (NS = 0: the vector
// {i, i, i, i}), stored to each of the ND destinations; with ND = 0 the
// vectors are only read (a store to `sink` that the data cannot trigger in
// practice keeps the loads alive).  A workgroup moves U * 256 vectors
// (U = 2 with 8 or more sources, else 4), every load of a lane in flight
// before its stores; NTL / NTS select the non-temporal forms.
struct StreamArgs {
    const u32x4* src[PURLIN_MAX_RANKS];
    u32x4* dst[PURLIN_MAX_RANKS];
    u32x4* sink;
    uint64_t nvec;
    int nsrc, ndst;
    uint64_t* rec;  // timing records, or null
    uint64_t rate_khz;
};

constexpr int stream_unroll(int nsrc) { return nsrc >= 8 ? 2 : 4; }

// NS, ND < 0: counts taken from the arguments.  U vectors per lane.  The
// cache hints are template parameters: a run-time choice between the two
// load forms can be folded into one plain load by the compiler.
template <int NS, int ND, int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void stream_nm(StreamArgs a) {
    const int ns = NS >= 0 ? NS : a.nsrc, nd = ND >= 0 ? ND : a.ndst;
    const uint64_t t_entry = a.rec ? wall_clock64() : 0;
    const uint64_t base = uint64_t(blockIdx.x) * (kBlock * U) + threadIdx.x;
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint64_t i = base + uint64_t(u) * kBlock;
        v[u] = u32x4{uint32_t(i), uint32_t(i), uint32_t(i), uint32_t(i)};
        if (ns > 0 && i < a.nvec) {
            v[u] = load16<NTL>(reinterpret_cast<const char*>(a.src[0] + i));
            for (int p = 1; p < ns; ++p) v[u] ^= load16<NTL>(reinterpret_cast<const char*>(a.src[p] + i));
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint64_t i = base + uint64_t(u) * kBlock;
        if (i >= a.nvec) continue;
        if (nd == 0) {
            if (v[u][0] == 0x9E3779B9u && v[u][1] == 0x7F4A7C15u && v[u][2] == 0xF39CC060u) *a.sink = v[u];
        } else {
            for (int j = 0; j < nd; ++j) store16<NTS>(reinterpret_cast<char*>(a.dst[j] + i), v[u]);
        }
    }
    if (a.rec) {
        __builtin_amdgcn_s_waitcnt(0);  // this thread's loads and stores have completed
        __syncthreads();
        if (threadIdx.x == 0) {
            uint64_t* r = a.rec + kRecPerGroup * (uint64_t(blockIdx.x) + 1);
            r[0] = xcc_id();
            r[1] = t_entry;
            r[2] = t_entry;
            r[3] = wall_clock64();
            if (blockIdx.x == 0) {
                a.rec[0] = a.rate_khz;
                a.rec[1] = gridDim.x;
            }
        }
    }
}

// One purlin_stream launch: the kernel instantiated for its source and
// destination counts (the measured mixes) or the generic one.
template <bool NTL, bool NTS>
void launch_stream_mix(const StreamArgs& a, dim3 grid, hipStream_t stream) {
    const int ns = a.nsrc, nd = a.ndst;
    if (ns == 1 && nd == 0)
        hipLaunchKernelGGL((stream_nm<1, 0, stream_unroll(1), NTL, NTS>), grid, dim3(kBlock), 0, stream, a);
    else if (ns == 0 && nd == 1)
        hipLaunchKernelGGL((stream_nm<0, 1, stream_unroll(0), NTL, NTS>), grid, dim3(kBlock), 0, stream, a);
    else if (ns == 1 && nd == 1)
        hipLaunchKernelGGL((stream_nm<1, 1, stream_unroll(1), NTL, NTS>), grid, dim3(kBlock), 0, stream, a);
    else if (ns == 8 && nd == 1)
        hipLaunchKernelGGL((stream_nm<8, 1, stream_unroll(8), NTL, NTS>), grid, dim3(kBlock), 0, stream, a);
    else if (ns == 1 && nd == 8)
        hipLaunchKernelGGL((stream_nm<1, 8, stream_unroll(1), NTL, NTS>), grid, dim3(kBlock), 0, stream, a);
    else if (ns >= 8)
        hipLaunchKernelGGL((stream_nm<-1, -1, stream_unroll(8), NTL, NTS>), grid, dim3(kBlock), 0, stream, a);
    else
        hipLaunchKernelGGL((stream_nm<-1, -1, stream_unroll(1), NTL, NTS>), grid, dim3(kBlock), 0, stream, a);
}

}  // namespace

hipError_t launch_stream_copy(void* dst, const void* src, uint64_t bytes, hipStream_t stream) {
    const uint64_t nvec = bytes / 16;
    if (nvec == 0) return hipSuccess;
    const uint64_t per_block = uint64_t(kBlock) * kCopyUnroll;
    const uint64_t blocks = (nvec + per_block - 1) / per_block;
    if (blocks > 0xffffffffull) return hipErrorInvalidValue;
    (void)hipGetLastError();
    hipLaunchKernelGGL(stream_copy, dim3(static_cast<uint32_t>(blocks)), dim3(kBlock), 0, stream,
                       static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), nvec);
    return hipGetLastError();
}

uint64_t stream_groups(int nsrc, uint64_t bytes) {
    const uint64_t per_block = uint64_t(kBlock) * stream_unroll(nsrc);
    return (bytes / 16 + per_block - 1) / per_block;
}

uint64_t wall_clock_khz() {
    int dev = 0, khz = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) return 0;
    return khz > 0 ? static_cast<uint64_t>(khz) : 0;
}

hipError_t launch_stream(void* const* dst, int ndst, const void* const* src, int nsrc, uint64_t bytes, void* sink,
                         uint32_t hints, hipStream_t stream, uint64_t* rec) {
    StreamArgs a{};
    a.rec = rec;
    a.rate_khz = rec ? wall_clock_khz() : 0;
    for (int p = 0; p < nsrc; ++p) a.src[p] = static_cast<const u32x4*>(src[p]);
    for (int j = 0; j < ndst; ++j) a.dst[j] = static_cast<u32x4*>(dst[j]);
    a.sink = static_cast<u32x4*>(sink);
    a.nvec = bytes / 16;
    a.nsrc = nsrc;
    a.ndst = ndst;
    if (a.nvec == 0) return hipSuccess;
    const uint64_t per_block = uint64_t(kBlock) * stream_unroll(nsrc);
    const uint64_t blocks = (a.nvec + per_block - 1) / per_block;
    if (blocks > 0xffffffffull) return hipErrorInvalidValue;
    const dim3 grid(static_cast<uint32_t>(blocks));
    (void)hipGetLastError();
    switch (hints & (PURLIN_STREAM_NT_LOAD | PURLIN_STREAM_NT_STORE)) {
        case 0: launch_stream_mix<false, false>(a, grid, stream); break;
        case PURLIN_STREAM_NT_LOAD: launch_stream_mix<true, false>(a, grid, stream); break;
        case PURLIN_STREAM_NT_STORE: launch_stream_mix<false, true>(a, grid, stream); break;
        default: launch_stream_mix<true, true>(a, grid, stream); break;
    }
    return hipGetLastError();
}

hipError_t launch_phase(const purlin_desc* items, uint64_t n, uint32_t kind, uint32_t nsrc, uint32_t src_buf,
                        uint32_t src_step, bool nt_load, bool nt_store, purlin_dtype dtype, void* const* bufs,
                        int nbufs, uint32_t max_workgroups, uint32_t copy_depth, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    ExecArgs a{};
    a.items = items;
    a.n_items = n;
    for (int i = 0; i < nbufs && i < 2 * PURLIN_MAX_RANKS; ++i) a.bufs[i] = static_cast<char*>(bufs[i]);
    if (kind == PURLIN_KIND_REDUCE) {
        for (uint32_t p = 0; p < nsrc && p < PURLIN_MAX_RANKS; ++p) {
            const uint64_t b = uint64_t(src_buf) + uint64_t(p) * src_step;
            if (b >= uint64_t(nbufs)) return hipErrorInvalidValue;
            a.srcs[p] = static_cast<char*>(bufs[b]);
        }
    }
    uint64_t blocks = (n + kWavesPerBlock - 1) / kWavesPerBlock;
    if (max_workgroups) blocks = std::min<uint64_t>(blocks, max_workgroups);
    if (blocks > 0xffffffffull) return hipErrorInvalidValue;
    a.wave_stride = blocks * kWavesPerBlock;
    const dim3 grid(static_cast<uint32_t>(blocks));
    (void)hipGetLastError();
    if (kind == PURLIN_KIND_COPY) {
        launch_copy(grid, stream, a, nt_load, nt_store, copy_depth);
    } else {
        const bool bf16 = dtype == PURLIN_BF16;
        switch (nsrc) {
#define PURLIN_REDUCE_CASE(n) \
    case n: launch_reduce<n>(grid, stream, a, bf16, nt_load, nt_store); break;
            PURLIN_REDUCE_CASE(1) PURLIN_REDUCE_CASE(2) PURLIN_REDUCE_CASE(3) PURLIN_REDUCE_CASE(4)
            PURLIN_REDUCE_CASE(5) PURLIN_REDUCE_CASE(6) PURLIN_REDUCE_CASE(7) PURLIN_REDUCE_CASE(8)
            PURLIN_REDUCE_CASE(9) PURLIN_REDUCE_CASE(10) PURLIN_REDUCE_CASE(11) PURLIN_REDUCE_CASE(12)
            PURLIN_REDUCE_CASE(13) PURLIN_REDUCE_CASE(14) PURLIN_REDUCE_CASE(15) PURLIN_REDUCE_CASE(16)
#undef PURLIN_REDUCE_CASE
            default: return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

}  // namespace purlin
