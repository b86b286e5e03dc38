// MoE dispatch (pack) and combine (unpack) for gfx950.
//
// Expert parallelism dispatches tokens to the ranks that own their experts
// and combines the expert outputs (Purlin, arXiv 2609.36954: Section 2,
// Table 2); the per-destination segments are the scatteredV layout of
// Section 3.1.  The reduction in combine follows Eq. 2 with slots in place
// of ranks: one FP32 accumulator per output element, started at zero, terms
// added in ascending slot order, converted to bf16 once.
//
// Pack runs in three launches:
//   1. pack_tiles: one workgroup per tile of 64 tokens.  In LDS it builds,
//      for every expert, a 64-bit mask of the tile's tokens that chose it.
//      The rank of (t, k) among the tile's earlier tokens of the same expert
//      is a popcount of that mask below t; the tile's count per expert is
//      the mask's popcount.  Deterministic: no ordering depends on atomics.
//   2. pack_scan: one workgroup.  Exclusive prefix over tiles per expert,
//      expert totals, exclusive prefix over experts, destination
//      counts/offsets, and the error flag.  The per-tile counts are
//      rewritten in place into each tile's first row per expert.
//   3. pack_rows: one wavefront per (token, 1 KiB column slice).  Lane k
//      forms pos[t, k]; the wave then streams its slice of the token row
//      through registers and writes it to the K packed rows with 16-byte
//      stores.
// Extra workgroups of the first two launches read the token matrix ahead
// (when it is 8-128 MiB), so that the rows kernel finds it in the
// last-level cache.
// Unpack is one launch, one wavefront per (token, slice), slots in groups
// of 4 with all their 16-byte row loads in flight before the FP32
// accumulation.
//
// The de-duplicated variants (one row per token and destination rank) use
// the same structure with destinations in place of experts: pack_dedup is
// dedup_tiles, dedup_scan, dedup_rows; unpack_dedup is unpack_rows without
// gates, summing a token's rows in rank order.

#include "kernels.h"

#include <algorithm>
#include <type_traits>

namespace purlin {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kScanThreads = 1024;
constexpr int kMaxExperts = 4096;
constexpr int kMaxDedupRanks = 16;

// The id matrices of a metadata launch that covers several ranks at once
// (one grid row or workgroup per rank); a single-rank launch fills entry 0.
struct RankIds {
    const int32_t* ids[PURLIN_MAX_RANKS];
};

// Rank p's copy of a per-rank workspace array: the ranks' workspaces lie
// `stride` bytes apart (0 for a single rank).
template <class V>
__device__ __forceinline__ V* at_rank(V* base, uint64_t stride, int p) {
    using C = typename std::conditional<std::is_const<V>::value, const char*, char*>::type;
    return reinterpret_cast<V*>(reinterpret_cast<C>(base) + stride * static_cast<uint64_t>(p));
}

__device__ __forceinline__ uint32_t wave_index() {
    return __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + threadIdx.x / kWave);
}

__device__ __forceinline__ uint32_t lane_index() { return threadIdx.x & (kWave - 1); }

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

// binary32 -> bf16, round to nearest, ties to even (see the executor for
// the derivation); NaN -> quiet NaN with sign and top payload bits kept.
__device__ __forceinline__ uint32_t to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    const uint32_t rounded = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    const uint32_t quiet_nan = (u >> 16) | 0x40u;
    return (u & 0x7FFFFFFFu) > 0x7F800000u ? quiet_nan : rounded;
}

// A byte range that extra workgroups of a metadata launch read through the
// caches and drop: the token matrix, read while the latency-bound metadata
// leaves HBM idle, so that the rows kernel after it finds the matrix in the
// last-level cache and streams its writes alone.  `blocks` workgroups
// (after the launch's own) read [lo, hi) of `base`.
struct Prefetch {
    const char* base;
    uint64_t lo, hi;
    uint32_t blocks;
};

// Workgroup `part` of `parts` reads its share of p's range, 16-byte loads,
// four in flight per thread; the values only feed an empty asm statement,
// which keeps the loads without storing anything.
__device__ __forceinline__ void prefetch_part(const Prefetch& p, uint32_t part) {
    const uint64_t v0 = p.lo / 16, v1 = p.hi / 16;
    const uint64_t per = (v1 - v0 + p.blocks - 1) / p.blocks;
    const uint64_t lo = v0 + per * part, hi = min(v1, lo + per);
    const uint32_t nt = blockDim.x;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (uint64_t i = lo + threadIdx.x; i < hi; i += 4ull * nt) {
        u32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint64_t j = i + static_cast<uint64_t>(u) * nt;
            v[u] = j < hi ? load16<false>(p.base + j * 16) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) acc ^= v[u];
    }
    __asm__ volatile("" : : "v"(acc));
}

__global__ __launch_bounds__(kBlock) void pack_tiles(int T, int K, int E, RankIds rids, int32_t* __restrict__ tile_cnt,
                                                     int32_t* __restrict__ lrank, int32_t* __restrict__ tile_err,
                                                     uint64_t stride, Prefetch pf) {
    extern __shared__ unsigned long long masks[];  // [E]
    __shared__ int32_t tids[kPackTileTokens * 64];  // the tile's ids (K <= 64)
    __shared__ int err;
    const uint32_t ntiles = gridDim.x - pf.blocks;
    if (blockIdx.x >= ntiles) {
        prefetch_part(pf, blockIdx.x - ntiles);
        return;
    }
    const int tile = blockIdx.x;
    const int rank = blockIdx.y;
    const int32_t* ids = rids.ids[rank];
    tile_cnt = at_rank(tile_cnt, stride, rank);
    lrank = at_rank(lrank, stride, rank);
    tile_err = at_rank(tile_err, stride, rank);
    const int t0 = tile * kPackTileTokens;
    const int nt = min(kPackTileTokens, T - t0);
    const int n = nt * K;
    const int32_t* gids = ids + static_cast<int64_t>(t0) * K;

    for (int e = threadIdx.x; e < E; e += kBlock) masks[e] = 0ull;
    for (int j = threadIdx.x; j < n; j += kBlock) tids[j] = gids[j];
    if (threadIdx.x == 0) err = 0;
    __syncthreads();

    bool bad = false;
    for (int j = threadIdx.x; j < n; j += kBlock) {
        const int tl = j / K;
        const int k = j - tl * K;
        const int e = tids[j];
        if (e < 0 || e >= E) {
            bad = true;
            continue;
        }
        for (int k2 = 0; k2 < k; ++k2)
            if (tids[tl * K + k2] == e) bad = true;
        atomicOr(&masks[e], 1ull << tl);
    }
    if (bad) err = 1;  // every writer stores the same value
    __syncthreads();

    for (int j = threadIdx.x; j < n; j += kBlock) {
        const int tl = j / K;
        const int e = tids[j];
        int r = -1;
        if (e >= 0 && e < E) r = __popcll(masks[e] & ((1ull << tl) - 1ull));
        lrank[static_cast<int64_t>(t0) * K + j] = r;
    }
    for (int e = threadIdx.x; e < E; e += kBlock) tile_cnt[static_cast<int64_t>(tile) * E + e] = __popcll(masks[e]);
    if (threadIdx.x == 0) tile_err[tile] = err;
}

// Tile counts of one work unit kept in registers between the two passes.
constexpr int kScanBatch = 16;

// One workgroup per rank (workgroup p: rank p's tile counts, expert and
// destination outputs at p*E and p*P, status word p).
__global__ __launch_bounds__(kScanThreads) void pack_scan(int ntiles, int E, int P, int32_t* __restrict__ tile_cnt,
                                                          const int32_t* __restrict__ tile_err,
                                                          int32_t* __restrict__ expert_counts,
                                                          int32_t* __restrict__ expert_offsets,
                                                          int32_t* __restrict__ dest_counts,
                                                          int32_t* __restrict__ dest_offsets,
                                                          int32_t* __restrict__ dev_status, uint64_t stride,
                                                          Prefetch pf) {
    const uint32_t nscan = gridDim.x - pf.blocks;
    if (blockIdx.x >= nscan) {
        prefetch_part(pf, blockIdx.x - nscan);
        return;
    }
    __shared__ int32_t partial[kMaxExperts];  // per work unit (expert, tile slice)
    __shared__ int32_t total[kMaxExperts];    // per expert
    __shared__ int32_t offs[kMaxExperts];     // per expert, exclusive prefix
    __shared__ int32_t scan[kScanThreads / kWave];  // wave totals
    const int tid = threadIdx.x;
    const int rank = blockIdx.x;
    tile_cnt = at_rank(tile_cnt, stride, rank);
    tile_err = at_rank(tile_err, stride, rank);
    expert_counts += static_cast<int64_t>(rank) * E;
    if (expert_offsets) expert_offsets += static_cast<int64_t>(rank) * E;
    dest_counts += static_cast<int64_t>(rank) * P;
    dest_offsets += static_cast<int64_t>(rank) * P;
    if (dev_status) dev_status += rank;

    // error flags: one per thread when the tiles fit one pass (its load is
    // only consumed at the end, so it overlaps the count loads), else a loop
    int err0 = 0;
    if (ntiles <= kScanThreads && tid < ntiles) err0 = tile_err[tid];

    // Work units: tpe threads per expert when E is small, each owning a
    // contiguous slice of tiles; one unit per expert when E >= 1024.  A
    // unit whose slice fits kScanBatch keeps its counts in registers.
    // Unit u is (slice q = u / E, expert e = u % E): consecutive lanes read
    // and write consecutive experts of one tile row.
    const int tpe = E >= kScanThreads ? 1 : kScanThreads / E;
    const int units = E * tpe;
    const int span = (ntiles + tpe - 1) / tpe;
    const bool in_regs = span <= kScanBatch && units <= kScanThreads;

    int c[kScanBatch];
    for (int u = tid; u < units; u += kScanThreads) {
        const int q = u / E, e = u - q * E;
        const int lo = min(ntiles, q * span), hi = min(ntiles, lo + span);
        int sum = 0;
        for (int t = lo; t < hi; t += kScanBatch) {
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i) c[i] = (t + i < hi) ? tile_cnt[static_cast<int64_t>(t + i) * E + e] : 0;
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i) sum += c[i];
        }
        partial[u] = sum;
    }
    __syncthreads();
    for (int e = tid; e < E; e += kScanThreads) {
        int sum = 0;
        for (int q = 0; q < tpe; ++q) sum += partial[q * E + e];
        total[e] = sum;
    }
    __syncthreads();

    // Exclusive prefix over experts: each thread sums a run of consecutive
    // experts; the runs are combined by a cross-lane scan in every wave and
    // a scan of the wave totals.
    const int per = (E + kScanThreads - 1) / kScanThreads;
    int local = 0;
    for (int i = 0; i < per; ++i) {
        const int e = tid * per + i;
        if (e < E) local += total[e];
    }
    const uint32_t lane = tid & (kWave - 1), wave = tid / kWave;
    int incl = local;
    for (int off = 1; off < kWave; off <<= 1) {
        const int u = __shfl_up(incl, off);
        if (lane >= static_cast<uint32_t>(off)) incl += u;
    }
    if (lane == kWave - 1) scan[wave] = incl;
    __syncthreads();
    // this wave's base: the totals of the waves before it, summed across lanes
    int wave_base = lane < wave ? scan[lane] : 0;
    for (int off = kWave / 2; off > 0; off >>= 1) wave_base += __shfl_xor(wave_base, off);
    int run = wave_base + incl - local;
    for (int i = 0; i < per; ++i) {
        const int e = tid * per + i;
        if (e < E) {
            offs[e] = run;
            expert_counts[e] = total[e];
            if (expert_offsets) expert_offsets[e] = run;
            run += total[e];
        }
    }
    __syncthreads();

    // Rewrite each tile's count into the row of its first (t, k) per expert.
    for (int u = tid; u < units; u += kScanThreads) {
        const int q = u / E, e = u - q * E;
        const int lo = min(ntiles, q * span), hi = min(ntiles, lo + span);
        int base = offs[e];
        for (int q2 = 0; q2 < q; ++q2) base += partial[q2 * E + e];
        for (int t = lo; t < hi; t += kScanBatch) {
            if (!in_regs) {
#pragma unroll
                for (int i = 0; i < kScanBatch; ++i)
                    c[i] = (t + i < hi) ? tile_cnt[static_cast<int64_t>(t + i) * E + e] : 0;
            }
#pragma unroll
            for (int i = 0; i < kScanBatch; ++i) {
                if (t + i < hi) tile_cnt[static_cast<int64_t>(t + i) * E + e] = base;
                base += c[i];
            }
        }
    }

    // rank r's rows: its experts' offsets are contiguous, so its count is
    // the difference of two expert offsets
    const int L = E / P;
    for (int r = tid; r < P; r += kScanThreads) {
        const int end = r + 1 < P ? offs[(r + 1) * L] : offs[E - 1] + total[E - 1];
        dest_counts[r] = end - offs[r * L];
        dest_offsets[r] = offs[r * L];
    }

    int any = err0;
    if (ntiles > kScanThreads)
        for (int t = tid; t < ntiles; t += kScanThreads) any |= tile_err[t];
    any = __syncthreads_or(any);
    if (tid == 0 && dev_status) *dev_status = any ? 1 : 0;
}

// Stream one column slice of a token row (U * 64 16-byte vectors, U per
// lane) through registers into every slot j < nslots: dst_of(j) gives the
// destination row's base (wave-uniform), or null for none.  The row is read
// once from HBM.  Rows that are not a multiple of 16 bytes take one slice
// per token, 2 bytes per lane step.
template <int U, bool NTL, bool NTS, class DstOf>
__device__ __forceinline__ void copy_row_to_slots(const char* src, uint64_t row_bytes, uint32_t slice, int nslots,
                                                  uint32_t lane, DstOf dst_of) {
    if (row_bytes % 16 == 0) {
        const uint64_t nvec = row_bytes / 16;
        const uint64_t base = static_cast<uint64_t>(slice) * U * kWave;
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t i = base + u * kWave + lane;
            if (i < nvec) v[u] = load16<NTL>(src + i * 16);
        }
        for (int j = 0; j < nslots; ++j) {
            char* dst = dst_of(j);
            if (!dst) continue;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint64_t i = base + u * kWave + lane;
                if (i < nvec) store16<NTS>(dst + i * 16, v[u]);
            }
        }
    } else {
        const uint64_t H = row_bytes / 2;
        for (uint64_t h = lane; h < H; h += kWave) {
            const uint16_t v = reinterpret_cast<const uint16_t*>(src)[h];
            for (int j = 0; j < nslots; ++j) {
                char* dst = dst_of(j);
                if (dst) reinterpret_cast<uint16_t*>(dst)[h] = v;
            }
        }
    }
}

// One wavefront per (token, column slice): a slice is U * 64 16-byte
// vectors of the row, so each lane holds U vectors of it.  Every slice's
// wave forms the token's K positions (lane k forms pos[t, k]); the wave of
// slice 0 also stores them.
template <int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void pack_rows(int T, int H, int K, int E, int slices, const char* __restrict__ x,
                                                    const int32_t* __restrict__ ids,
                                                    const int32_t* __restrict__ tile_base,
                                                    const int32_t* __restrict__ lrank, int32_t* __restrict__ pos,
                                                    char* __restrict__ packed) {
    const uint32_t w = wave_index();
    const uint32_t t = w / slices;
    if (t >= static_cast<uint32_t>(T)) return;
    const uint32_t slice = w - t * slices;
    const uint32_t lane = lane_index();
    const int64_t rows = static_cast<int64_t>(T) * K;
    int p = -1;
    if (lane < static_cast<uint32_t>(K)) {
        const int64_t j = static_cast<int64_t>(t) * K + lane;
        const int e = ids[j];
        const int r = lrank[j];
        if (e >= 0 && e < E && r >= 0) {
            const int64_t q = static_cast<int64_t>(tile_base[static_cast<int64_t>(t / kPackTileTokens) * E + e]) + r;
            p = (q >= 0 && q < rows) ? static_cast<int>(q) : -1;
        }
        if (slice == 0) pos[j] = p;
    }
    const uint64_t row_bytes = static_cast<uint64_t>(H) * 2;
    copy_row_to_slots<U, NTL, NTS>(x + t * row_bytes, row_bytes, slice, K, lane, [&](int j) -> char* {
        const int pj = __builtin_amdgcn_readlane(p, j);
        return pj < 0 ? nullptr : packed + static_cast<uint64_t>(pj) * row_bytes;
    });
}

// ---------------------------------------------------------------------------
// The whole pack in one launch, for routings small enough that every
// workgroup can count all of them itself (T*K <= kOneMaxIds, E <=
// kOneMaxExperts) and hold its own tokens' rows in registers.  Workgroup b
// owns tokens [b*tw, b*tw + tw) and never waits for another workgroup:
//   1. it loads every id (4 to a vector) and its own ids;
//   2. it counts every id into LDS, split at its first token: before[e] =
//      ids of e in earlier tokens, after[e] = the rest (lane l adds into copy
//      l % C of the counters, C up to 16, so the routings' popular experts
//      do not serialise one LDS word: with Zipf(1.1) routing over 256
//      experts, expert 0 is in 86% of the tokens); it marks its own tokens
//      in one 64-bit mask per expert; then it issues the loads of its rows of
//      x (kOneVec 16-byte vectors per thread, non-temporal), which arrive
//      while it finishes the metadata;
//   3. expert totals, their exclusive prefix over experts, and the positions
//      of its own (t, k): offset[e] + before[e] + earlier own tokens of e;
//   4. it writes each vector of its rows to the K packed rows of its token,
//      each as soon as that vector has arrived.
// Workgroup 0 also writes the counts and offsets, checks every token for
// repeated ids (before its stores, whose queue its loads would otherwise
// wait behind; after them for K > 8) and writes the status word (it has seen
// every id, so it knows of out-of-range ones).  Ranks follow from counts, so the
// result is the same whatever the order of the LDS atomics.
constexpr int kOneThreads = 1024;
constexpr int kOneVec = 16;                               // x vectors per thread: 64 VGPRs
constexpr int kOneIdVec = 8;                              // id vectors (4 ids) per thread
constexpr int kOneMaxIds = kOneIdVec * 4 * kOneThreads;  // 32768
constexpr int kOneMaxExperts = kOneThreads;              // one expert per thread in the scan
constexpr int kOneMaxOwn = kOneThreads;                  // own (t, k) pairs: one per thread
constexpr int kOneUnrolledSlots = 8;                     // K up to this: the store loop unrolled
constexpr int kOneMaxCopies = 16;                        // counter copies (lanes modulo)
constexpr uint32_t kOneCopyBytes = 40u << 10;            // LDS for the counter copies (64 KiB in all)

constexpr int kDupTokens = 4;  // tokens per thread and round of the repeated-id check

// The ids of tokens t, t + kOneThreads, ... (kDupTokens of them, indexes
// clamped to the last token) into registers, all loads issued together.
template <int KMAX>
__device__ __forceinline__ void load_token_ids(int (&e)[kDupTokens][KMAX], const int32_t* __restrict__ ids, int T,
                                               int K, int t) {
#pragma unroll
    for (int i = 0; i < kDupTokens; ++i) {
        const int32_t* row = ids + static_cast<int64_t>(min(t + i * kOneThreads, T - 1)) * K;
#pragma unroll
        for (int k = 0; k < KMAX; ++k) e[i][k] = k < K ? row[k] : 0;
    }
}

// Whether any of those tokens holds an id twice among its K slots.
template <int KMAX>
__device__ __forceinline__ bool repeated_id(const int (&e)[kDupTokens][KMAX], int K) {
    bool dup = false;
#pragma unroll
    for (int i = 0; i < kDupTokens; ++i)
#pragma unroll
        for (int k = 1; k < KMAX; ++k)
#pragma unroll
            for (int k2 = 0; k2 < k; ++k2)
                if (k < K && e[i][k] == e[i][k2]) dup = true;
    return dup;
}

template <int KMAX, bool NTL, bool NTS>
__global__ __launch_bounds__(kOneThreads) void pack_onepass(int T, int K, int E, int P, int tw, uint32_t nvec,
                                                            int copies, const char* __restrict__ x,
                                                            const int32_t* __restrict__ ids,
                                                            char* __restrict__ packed, int32_t* __restrict__ pos,
                                                            int32_t* __restrict__ expert_counts,
                                                            int32_t* __restrict__ expert_offsets,
                                                            int32_t* __restrict__ dest_counts,
                                                            int32_t* __restrict__ dest_offsets,
                                                            int32_t* __restrict__ dev_status, uint64_t* rec,
                                                            uint64_t rate_khz) {
    // Counter copy c holds before[] at [c*S, c*S + E) and after[] at
    // [c*S + E, c*S + 2E); S = 2E + 1 is odd, so one expert's copies lie in
    // different LDS banks.
    extern __shared__ int32_t hist[];
    __shared__ int32_t cnt[2 * kOneMaxExperts];  // summed copies: before[e], then after[e]
    __shared__ int32_t offs[kOneMaxExperts];
    __shared__ unsigned long long masks[kOneMaxExperts];
    __shared__ int32_t own_pos[kOneMaxOwn];
    __shared__ int32_t wave_tot[kOneThreads / kWave];
    __shared__ int bad_any;

    const uint64_t t_entry = rec ? wall_clock64() : 0;
    const int tid = threadIdx.x;
    const int t0 = static_cast<int>(blockIdx.x) * tw;
    const int nt = min(tw, T - t0);
    const int n = T * K;
    const int first = t0 * K;  // this workgroup's first (t, k)
    const int nown = nt * K;
    const uint64_t row_bytes = static_cast<uint64_t>(nvec) * 16;
    const int S = 2 * E + 1;

    // 1. loads of the ids.  Every load is issued unconditionally (indexes
    // clamped into range, n >= 4), so the code is straight-line and each
    // use waits only for its own load.
    const int n4 = n / 4;
    u32x4 idv[kOneIdVec];
#pragma unroll
    for (int q = 0; q < kOneIdVec; ++q) {
        const int j = min(tid + q * kOneThreads, n4 - 1);
        idv[q] = *reinterpret_cast<const u32x4*>(ids + 4 * j);
    }
    const int tail = n - 4 * n4;
    const int tail_e = ids[min(4 * n4 + tid, n - 1)];
    const int own_e = ids[first + min(tid, nown - 1)];
    // Workgroup 0 checks every token for repeated ids (the status word).
    // With K <= KMAX the ids of a thread's first kDupTokens tokens are
    // loaded here, with the others, so that they arrive before any store is
    // queued behind which they would wait (later rounds, T > 4096, are
    // loaded after the counting, still before the stores).
    const bool dup_check = blockIdx.x == 0 && dev_status != nullptr && K > 1;
    int dupv[kDupTokens][KMAX > 0 ? KMAX : 1];
    if constexpr (KMAX > 0)
        if (dup_check) load_token_ids<KMAX>(dupv, ids, T, K, tid);
    for (int i = tid; i < copies * S; i += kOneThreads) hist[i] = 0;
    for (int e = tid; e < E; e += kOneThreads) masks[e] = 0ull;
    if (tid == 0) bad_any = 0;
    __syncthreads();

    // 2. count every id, split at this workgroup's first token
    bool bad = false;
    int32_t* h = hist + (tid & (copies - 1)) * S;
#pragma unroll
    for (int q = 0; q < kOneIdVec; ++q) {
        const int j = tid + q * kOneThreads;
        if (j < n4) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int e = static_cast<int>(idv[q][r]);
                if (e < 0 || e >= E)
                    bad = true;
                else
                    atomicAdd(&h[(4 * j + r >= first ? E : 0) + e], 1);
            }
        }
    }
    if (tid < tail) {
        if (tail_e < 0 || tail_e >= E)
            bad = true;
        else
            atomicAdd(&h[(4 * n4 + tid >= first ? E : 0) + tail_e], 1);
    }
    const int tl = tid / K;  // own token of (t, k) = (t0 + tl, tid % K)
    const bool own_ok = tid < nown && own_e >= 0 && own_e < E;
    if (own_ok) {
        const unsigned long long bit = 1ull << tl;
        if (atomicOr(&masks[own_e], bit) & bit) bad = true;  // repeated within the token
    }
    if constexpr (KMAX > 0) {
        if (dup_check) {
            if (repeated_id<KMAX>(dupv, K)) bad = true;
            for (int tb = tid + kDupTokens * kOneThreads; tb < T; tb += kDupTokens * kOneThreads) {
                load_token_ids<KMAX>(dupv, ids, T, K, tb);
                if (repeated_id<KMAX>(dupv, K)) bad = true;
            }
        }
    }
    // the rows: issued after the counting in program order (a wave whose
    // loads cannot all issue at once would otherwise stall the counting
    // behind them)
    __asm__ volatile("" ::: "memory");
    const uint32_t nv = static_cast<uint32_t>(nt) * nvec;
    const char* xs = x + static_cast<uint64_t>(t0) * row_bytes;
    u32x4 v[kOneVec];
#pragma unroll
    for (int u = 0; u < kOneVec; ++u) {
        const uint32_t i = min(static_cast<uint32_t>(u * kOneThreads + tid), nv - 1);
        v[u] = load16<NTL>(xs + static_cast<uint64_t>(i) * 16);
    }
    if (bad) bad_any = 1;  // every writer stores the same value
    __syncthreads();
    for (int e = tid; e < E; e += kOneThreads) {
        int before = 0, after = 0;
        for (int c = 0; c < copies; ++c) {
            before += hist[c * S + e];
            after += hist[c * S + E + e];
        }
        cnt[e] = before;
        cnt[E + e] = after;
    }
    __syncthreads();

    // 3. expert totals and their exclusive prefix: one expert per thread
    const int tot = tid < E ? cnt[tid] + cnt[E + tid] : 0;
    const uint32_t lane = tid & (kWave - 1), wave = tid / kWave;
    int incl = tot;
    for (int off = 1; off < kWave; off <<= 1) {
        const int w = __shfl_up(incl, off);
        if (lane >= static_cast<uint32_t>(off)) incl += w;
    }
    if (lane == kWave - 1) wave_tot[wave] = incl;
    __syncthreads();
    int wave_base = lane < wave ? wave_tot[lane] : 0;
    for (int off = kWave / 2; off > 0; off >>= 1) wave_base += __shfl_xor(wave_base, off);
    const int excl = wave_base + incl - tot;
    if (tid < E) offs[tid] = excl;
    if (blockIdx.x == 0 && tid < E) {
        expert_counts[tid] = tot;
        if (expert_offsets) expert_offsets[tid] = excl;
    }
    __syncthreads();
    if (blockIdx.x == 0 && tid < P) {
        const int L = E / P;
        const int end = tid + 1 < P ? offs[(tid + 1) * L] : offs[E - 1] + cnt[E - 1] + cnt[2 * E - 1];
        dest_counts[tid] = end - offs[tid * L];
        dest_offsets[tid] = offs[tid * L];
    }
    if (tid < nown) {
        int p = -1;
        if (own_ok) {
            const int64_t q = static_cast<int64_t>(offs[own_e]) + cnt[own_e] +
                              __popcll(masks[own_e] & ((1ull << tl) - 1ull));
            p = q < n ? static_cast<int>(q) : -1;
        }
        own_pos[tid] = p;
        pos[first + tid] = p;
    }
    __syncthreads();

    const uint64_t t_meta = rec ? wall_clock64() : 0;

    // 4. every vector of the rows to its token's K packed rows.  With
    // KMAX > 0 (K <= KMAX) the slots are unrolled, so the code stays
    // straight-line and each vector's stores wait only for that vector.
    uint32_t tok = static_cast<uint32_t>(tid) / nvec, col = static_cast<uint32_t>(tid) - tok * nvec;
    const uint32_t step_tok = kOneThreads / nvec, step_col = kOneThreads - step_tok * nvec;
#pragma unroll
    for (int u = 0; u < kOneVec; ++u) {
        const uint32_t i = static_cast<uint32_t>(u * kOneThreads + tid);
        const bool live = i < nv;
        const int32_t* pk = own_pos + min(tok, static_cast<uint32_t>(nt - 1)) * K;
        char* dst = packed + col * 16ull;
        if constexpr (KMAX > 0) {
            int pv[KMAX];
#pragma unroll
            for (int k = 0; k < KMAX; ++k) pv[k] = k < K ? pk[k] : -1;
#pragma unroll
            for (int k = 0; k < KMAX; ++k)
                if (live && pv[k] >= 0) store16<NTS>(dst + static_cast<uint64_t>(pv[k]) * row_bytes, v[u]);
        } else if (live) {
            for (int k = 0; k < K; ++k) {
                const int p = pk[k];
                if (p >= 0) store16<NTS>(dst + static_cast<uint64_t>(p) * row_bytes, v[u]);
            }
        }
        tok += step_tok;
        col += step_col;
        if (col >= nvec) {
            col -= nvec;
            ++tok;
        }
    }

    // workgroup 0: the status word.  With K <= KMAX its repeated-id check
    // ran before the stores (above); for larger K every token's row is
    // checked here, after the workgroup's rows.
    if (blockIdx.x == 0 && dev_status) {
        bool dup = false;
        if constexpr (KMAX == 0) {
            for (int t = tid; t < T; t += kOneThreads) {
                const int32_t* row = ids + static_cast<int64_t>(t) * K;
                for (int k = 1; k < K; ++k) {
                    const int e = row[k];
                    for (int k2 = 0; k2 < k; ++k2)
                        if (row[k2] == e) dup = true;
                }
            }
        }
        const int any = __syncthreads_or(dup || bad_any);
        if (tid == 0) *dev_status = any ? 1 : 0;
    }
    if (rec) {
        __builtin_amdgcn_s_waitcnt(0);  // this thread's stores have completed
        __syncthreads();
        if (tid == 0) {
            uint64_t* r = rec + kRecPerGroup * (uint64_t(blockIdx.x) + 1);
            r[0] = xcc_id();
            r[1] = t_entry;
            r[2] = t_meta;
            r[3] = wall_clock64();
            if (blockIdx.x == 0) {
                rec[0] = rate_khz;
                rec[1] = gridDim.x;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// De-duplicated dispatch: one row per (token, destination rank).
//   1. dedup_tiles: one workgroup per tile of 64 tokens stages the tile's
//      ids in LDS; then one wavefront, lane = token, forms each token's
//      destination mask (bit r: some expert of the token lives on rank r)
//      and checks the ids; per destination a ballot gives the tile's count
//      and each token's rank among the tile's tokens bound there (popcount
//      below the lane).
//   2. dedup_scan: one workgroup; wave r scans destination r's tile counts
//      in tile order with cross-lane prefix sums, rewriting them into tile
//      bases; then destination counts and offsets, and the error flag.
//   3. dedup_rows: one wavefront per (token, column slice); lane r < P forms
//      row_of[t, r], and the row is streamed once into each of its rows.
__global__ __launch_bounds__(kBlock) void dedup_tiles(int T, int K, int E, int P, RankIds rids,
                                                      int32_t* __restrict__ tile_cnt, int32_t* __restrict__ lrank,
                                                      int32_t* __restrict__ tile_err, uint64_t stride) {
    __shared__ int32_t tids[kWave * 64];  // the tile's ids (K <= 64), loaded by the whole workgroup
    const int tile = blockIdx.x;
    const int rank = blockIdx.y;
    const int32_t* ids = rids.ids[rank];
    tile_cnt = at_rank(tile_cnt, stride, rank);
    lrank = at_rank(lrank, stride, rank);
    tile_err = at_rank(tile_err, stride, rank);
    const int64_t t0 = static_cast<int64_t>(tile) * kWave;
    const int nt = static_cast<int>(min<int64_t>(kWave, T - t0));
    const int n = nt * K;
    const int32_t* gids = ids + t0 * K;
    for (int j = threadIdx.x; j < n; j += kBlock) tids[j] = gids[j];
    __syncthreads();
    if (threadIdx.x >= kWave) return;
    const uint32_t lane = threadIdx.x;
    const bool valid = static_cast<int>(lane) < nt;
    const int L = E / P;
    uint32_t mask = 0;
    bool bad = false;
    if (valid) {
        const int32_t* row = tids + lane * K;
        for (int k = 0; k < K; ++k) {
            const int e = row[k];
            if (e < 0 || e >= E) {
                bad = true;
                continue;
            }
            for (int k2 = 0; k2 < k; ++k2)
                if (row[k2] == e) bad = true;
            mask |= 1u << (e / L);
        }
    }
    const uint64_t below = (uint64_t(1) << lane) - 1u;
    const int64_t t = t0 + lane;
    for (int r = 0; r < P; ++r) {
        const bool has = valid && ((mask >> r) & 1u);
        const uint64_t b = __ballot(has);
        if (lane == 0) tile_cnt[static_cast<int64_t>(tile) * P + r] = __popcll(b);
        if (valid) lrank[t * P + r] = has ? __popcll(b & below) : -1;
    }
    const uint64_t eb = __ballot(bad);
    if (lane == 0) tile_err[tile] = eb != 0 ? 1 : 0;
}

// One workgroup per rank, as pack_scan.
__global__ __launch_bounds__(kScanThreads) void dedup_scan(int ntiles, int P, int32_t* __restrict__ tile_cnt,
                                                           const int32_t* __restrict__ tile_err,
                                                           int32_t* __restrict__ dest_counts,
                                                           int32_t* __restrict__ dest_offsets,
                                                           int32_t* __restrict__ dev_status, uint64_t stride) {
    __shared__ int32_t totals[kMaxDedupRanks];
    const uint32_t wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
    const int rank = blockIdx.x;
    tile_cnt = at_rank(tile_cnt, stride, rank);
    tile_err = at_rank(tile_err, stride, rank);
    dest_counts += static_cast<int64_t>(rank) * P;
    dest_offsets += static_cast<int64_t>(rank) * P;
    if (dev_status) dev_status += rank;
    int any = 0;
    for (int t = threadIdx.x; t < ntiles; t += kScanThreads) any |= tile_err[t];
    if (wave < static_cast<uint32_t>(P)) {
        const int r = static_cast<int>(wave);
        int carry = 0;
        for (int t0 = 0; t0 < ntiles; t0 += kWave) {
            const int t = t0 + static_cast<int>(lane);
            const int c = t < ntiles ? tile_cnt[static_cast<int64_t>(t) * P + r] : 0;
            int v = c;  // inclusive prefix over the 64 lanes
            for (int off = 1; off < kWave; off <<= 1) {
                const int u = __shfl_up(v, off);
                if (lane >= static_cast<uint32_t>(off)) v += u;
            }
            if (t < ntiles) tile_cnt[static_cast<int64_t>(t) * P + r] = carry + v - c;
            carry += __shfl(v, kWave - 1);
        }
        if (lane == 0) totals[r] = carry;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int r = 0; r < P; ++r) {
            dest_counts[r] = totals[r];
            dest_offsets[r] = run;
            run += totals[r];
        }
    }
    any = __syncthreads_or(any);
    if (threadIdx.x == 0 && dev_status) *dev_status = any ? 1 : 0;
}

template <int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void dedup_rows(int T, int H, int P, int slices, const char* __restrict__ x,
                                                     const int32_t* __restrict__ tile_base,
                                                     const int32_t* __restrict__ lrank,
                                                     const int32_t* __restrict__ dest_offsets,
                                                     int32_t* __restrict__ row_of, char* __restrict__ packed) {
    const uint32_t w = wave_index();
    const uint32_t t = w / slices;
    if (t >= static_cast<uint32_t>(T)) return;
    const uint32_t slice = w - t * slices;
    const uint32_t lane = lane_index();
    int row = -1;
    if (lane < static_cast<uint32_t>(P)) {
        const int64_t j = static_cast<int64_t>(t) * P + lane;
        const int lr = lrank[j];
        if (lr >= 0) row = dest_offsets[lane] + tile_base[static_cast<int64_t>(t / kWave) * P + lane] + lr;
        if (slice == 0) row_of[j] = row;
    }
    const uint64_t row_bytes = static_cast<uint64_t>(H) * 2;
    copy_row_to_slots<U, NTL, NTS>(x + t * row_bytes, row_bytes, slice, P, lane, [&](int j) -> char* {
        const int rj = __builtin_amdgcn_readlane(row, j);
        return rj < 0 ? nullptr : packed + static_cast<uint64_t>(rj) * row_bytes;
    });
}

__global__ void set_status(int32_t* status) { *status = 0; }

constexpr int kSlotGroup = 4;  // slots whose row loads are in flight together (4 measured 3% faster than 8 or 16)

// One column slice of one output row: acc = +0, then for each slot k in
// ascending order acc (+)= g_k (x) widen(row_k) (GATED) or acc (+)= row_k,
// with src_of(k) the slot's source row base (wave-uniform; null = no row)
// and g_k read from lane k of `g`; the rows of kSlotGroup slots are loaded
// together before their terms are added.  Then one RNE narrowing and a
// 16-byte store per vector.
template <int U, bool NTL, bool NTS, bool GATED, class SrcOf>
__device__ __forceinline__ void combine_slots(SrcOf src_of, float g, int K, char* dst, uint64_t row_bytes,
                                              uint32_t slice, uint32_t lane) {
    if (row_bytes % 16 == 0) {
        const uint64_t nvec = row_bytes / 16;
        const uint64_t base = static_cast<uint64_t>(slice) * U * kWave;
        float acc[U][8];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[u][e] = 0.0f;
        for (int k0 = 0; k0 < K; k0 += kSlotGroup) {
            u32x4 v[kSlotGroup][U];
            const char* rk[kSlotGroup];
#pragma unroll
            for (int kk = 0; kk < kSlotGroup; ++kk) {
                rk[kk] = (k0 + kk < K) ? src_of(k0 + kk) : nullptr;
                if (!rk[kk]) continue;
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const uint64_t i = base + u * kWave + lane;
                    if (i < nvec) v[kk][u] = load16<NTL>(rk[kk] + i * 16);
                }
            }
#pragma unroll
            for (int kk = 0; kk < kSlotGroup; ++kk) {
                if (!rk[kk]) continue;
                const float gk = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(g), k0 + kk));
#pragma unroll
                for (int u = 0; u < U; ++u) {
#pragma unroll
                    for (int m = 0; m < 4; ++m) {
                        const uint32_t wv = v[kk][u][m];
                        const float lo = __uint_as_float(wv << 16), hi = __uint_as_float(wv & 0xFFFF0000u);
                        if constexpr (GATED) {
                            acc[u][2 * m] = __fadd_rn(acc[u][2 * m], __fmul_rn(gk, lo));
                            acc[u][2 * m + 1] = __fadd_rn(acc[u][2 * m + 1], __fmul_rn(gk, hi));
                        } else {
                            acc[u][2 * m] = __fadd_rn(acc[u][2 * m], lo);
                            acc[u][2 * m + 1] = __fadd_rn(acc[u][2 * m + 1], hi);
                        }
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t i = base + u * kWave + lane;
            if (i < nvec) {
                u32x4 o;
#pragma unroll
                for (int m = 0; m < 4; ++m) o[m] = to_bf16(acc[u][2 * m]) | (to_bf16(acc[u][2 * m + 1]) << 16);
                store16<NTS>(dst + i * 16, o);
            }
        }
    } else {
        const uint64_t H = row_bytes / 2;
        for (uint64_t h = lane; h < H; h += kWave) {
            float acc = 0.0f;
            for (int k = 0; k < K; ++k) {
                const char* row = src_of(k);
                if (!row) continue;
                const float gk = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(g), k));
                const uint16_t hv = reinterpret_cast<const uint16_t*>(row)[h];
                const float v = __uint_as_float(uint32_t(hv) << 16);
                acc = __fadd_rn(acc, GATED ? __fmul_rn(gk, v) : v);
            }
            reinterpret_cast<uint16_t*>(dst)[h] = static_cast<uint16_t>(to_bf16(acc));
        }
    }
}

// One wavefront per (token, column slice) of the output row.  GATED: the
// combine of one row per (t, k), acc (+)= g[t, k] (x) row; otherwise the
// de-duplicated combine of one row per (t, rank), acc (+)= row, where a
// slot of -1 means "no row".  Slots name rows in [0, rows).
template <int U, bool NTL, bool NTS, bool GATED>
__global__ __launch_bounds__(kBlock) void unpack_rows(int T, int H, int K, int slices, int64_t rows,
                                                      const char* __restrict__ y, const int32_t* __restrict__ pos,
                                                      const float* __restrict__ gates, char* __restrict__ out,
                                                      int32_t* __restrict__ dev_status) {
    const uint32_t w = wave_index();
    const uint32_t t = w / slices;
    if (t >= static_cast<uint32_t>(T)) return;
    const uint32_t slice = w - t * slices;
    const uint32_t lane = lane_index();
    int p = -1;
    float g = 1.0f;
    if (lane < static_cast<uint32_t>(K)) {
        const int64_t j = static_cast<int64_t>(t) * K + lane;
        p = pos[j];
        if constexpr (GATED) g = gates[j];
        const bool absent = !GATED && p == -1;
        if (!absent && (p < 0 || p >= rows)) {
            if (dev_status && slice == 0) atomicOr(dev_status, 1);
        }
        if (p < 0 || p >= rows) p = -1;
    }
    const uint64_t row_bytes = static_cast<uint64_t>(H) * 2;
    combine_slots<U, NTL, NTS, GATED>(
        [&](int k) -> const char* {
            const int pk = __builtin_amdgcn_readlane(p, k);
            return pk < 0 ? nullptr : y + static_cast<uint64_t>(pk) * row_bytes;
        },
        g, K, out + t * row_bytes, row_bytes, slice, lane);
}

// ---------------------------------------------------------------------------
// Expert-parallel dispatch and combine over P ranks in one pass each.  The
// dispatch is rank p's pack followed by the AllToAllV of its packed rows,
// without the packed buffers: once every rank's metadata is known (the
// pack_tiles / pack_scan of all ranks, one launch of each with a grid row or
// workgroup per rank; rank p's scan writes row p of the P x P counts),
// each token row goes straight to the receive buffer of every rank owning
// one of its experts, at
//     recv_row = sum_{q < p} counts[q][r] + pos_p[t, k] - dest_offsets_p[r].
// The combine reads each slot's expert output straight from its owner's
// buffer at that row and sums in slot order as unpack does.  On several
// GPUs this is a push of the rows to the peers and a pull of the outputs.
struct EpArgs {
    const char* x[PURLIN_MAX_RANKS];        // dispatch: token rows; combine: expert outputs (receive layout)
    const int32_t* ids[PURLIN_MAX_RANKS];
    char* dst[PURLIN_MAX_RANKS];            // dispatch: receive buffers; combine: outputs
    const int32_t* tile_base[PURLIN_MAX_RANKS];
    const int32_t* lrank[PURLIN_MAX_RANKS];
    const int32_t* dest_off[PURLIN_MAX_RANKS];
    const float* gates[PURLIN_MAX_RANKS];
    const int32_t* counts;  // P x P: rows rank p sends rank r
    const int64_t* before;  // P x P: rows rank r receives from ranks < p (ep_prefix)
    const int32_t* fits;    // 1 if every receive buffer holds its rows (ep_prefix)
    int32_t* recv_pos;      // [P, T, K]
    int32_t* status;        // optional
    int64_t capacity;       // rows per receive buffer
    int T, H, K, E, P, slices;
};

// Once per dispatch, after every rank's metadata: before[p][r] = rows rank r
// receives from ranks < p, and whether every receive buffer holds what it
// receives (if not, the rows kernel writes nothing).  The status word gets
// 1 if a receive buffer is too small or a rank's routing was invalid (its
// metadata status word `words[p]`), else 0.  One workgroup; P <= 16.
__global__ __launch_bounds__(kBlock) void ep_prefix(const int32_t* __restrict__ counts, int P, int64_t capacity,
                                                    int64_t* __restrict__ before, int32_t* __restrict__ fits,
                                                    const int32_t* __restrict__ words, int32_t* __restrict__ status) {
    __shared__ int32_t m[PURLIN_MAX_RANKS * PURLIN_MAX_RANKS];
    for (int i = threadIdx.x; i < P * P; i += kBlock) m[i] = counts[i];
    __syncthreads();
    for (int i = threadIdx.x; i < P * P; i += kBlock) {
        const int p = i / P, r = i - p * P;
        int64_t b = 0;
        for (int q = 0; q < p; ++q) b += m[q * P + r];
        before[i] = b;
    }
    if (threadIdx.x == 0) {
        bool ok = true;
        for (int r = 0; r < P; ++r) {
            int64_t col = 0;
            for (int q = 0; q < P; ++q) {
                ok = ok && m[q * P + r] >= 0;
                col += m[q * P + r];
            }
            ok = ok && col <= capacity;
        }
        *fits = ok ? 1 : 0;
        int any = 0;
        for (int p = 0; p < P; ++p) any |= words[p];
        if (status) *status = (any || !ok) ? 1 : 0;
    }
}

// Every wave of rank p's token t and column slice: lane k < K forms slot k's
// receiving rank and row from the pack metadata and ep_prefix's sums; if
// some receive buffer is too small, no wave writes anything.
template <int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void ep_dispatch_rows(EpArgs a) {
    if (!*a.fits) return;  // uniform: nothing is written
    const int P = a.P;
    const uint32_t w = wave_index();
    const uint64_t per_rank = static_cast<uint64_t>(a.T) * a.slices;
    if (w >= per_rank * P) return;
    const uint32_t p = static_cast<uint32_t>(w / per_rank);
    const uint32_t rem = static_cast<uint32_t>(w - p * per_rank);
    const uint32_t t = rem / a.slices, slice = rem - t * a.slices;
    const uint32_t lane = lane_index();
    const int K = a.K, E = a.E, L = a.E / P;
    int r = 0, row = -1;
    if (lane < static_cast<uint32_t>(K)) {
        const int64_t j = static_cast<int64_t>(t) * K + lane;
        const int e = a.ids[p][j];
        const int lr = a.lrank[p][j];
        if (e >= 0 && e < E && lr >= 0) {
            r = e / L;
            const int64_t q = static_cast<int64_t>(a.tile_base[p][static_cast<int64_t>(t / kPackTileTokens) * E + e]) + lr;
            const int64_t rr = a.before[p * P + r] + q - a.dest_off[p][r];
            row = (rr >= 0 && rr < a.capacity) ? static_cast<int>(rr) : -1;
        }
        if (slice == 0) a.recv_pos[(static_cast<int64_t>(p) * a.T + t) * K + lane] = row;
    }
    const uint64_t row_bytes = static_cast<uint64_t>(a.H) * 2;
    copy_row_to_slots<U, NTL, NTS>(a.x[p] + t * row_bytes, row_bytes, slice, K, lane, [&](int k) -> char* {
        const int rk = __builtin_amdgcn_readlane(row, k);
        return rk < 0 ? nullptr : a.dst[__builtin_amdgcn_readlane(r, k)] + static_cast<uint64_t>(rk) * row_bytes;
    });
}

// Rank p's token t, one column slice: slot k's expert output is row
// recv_pos[p, t, k] of the buffer of the rank owning ids_p[t, k].
template <int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void ep_combine_rows(EpArgs a) {
    const uint32_t w = wave_index();
    const uint64_t per_rank = static_cast<uint64_t>(a.T) * a.slices;
    if (w >= per_rank * a.P) return;
    const uint32_t p = static_cast<uint32_t>(w / per_rank);
    const uint32_t rem = static_cast<uint32_t>(w - p * per_rank);
    const uint32_t t = rem / a.slices, slice = rem - t * a.slices;
    const uint32_t lane = lane_index();
    const int K = a.K, E = a.E, L = a.E / a.P;
    int r = 0, row = -1;
    float g = 0.0f;
    if (lane < static_cast<uint32_t>(K)) {
        const int64_t j = static_cast<int64_t>(t) * K + lane;
        const int e = a.ids[p][j];
        const int64_t rr = a.recv_pos[static_cast<int64_t>(p) * a.T * K + j];
        g = a.gates[p][j];
        if (e >= 0 && e < E && rr >= 0 && rr < a.capacity) {
            r = e / L;
            row = static_cast<int>(rr);
        } else if (a.status && slice == 0) {
            atomicOr(a.status, 1);
        }
    }
    const uint64_t row_bytes = static_cast<uint64_t>(a.H) * 2;
    combine_slots<U, NTL, NTS, true>(
        [&](int k) -> const char* {
            const int rk = __builtin_amdgcn_readlane(row, k);
            return rk < 0 ? nullptr : a.x[__builtin_amdgcn_readlane(r, k)] + static_cast<uint64_t>(rk) * row_bytes;
        },
        g, K, a.dst[p] + t * row_bytes, row_bytes, slice, lane);
}

// De-duplicated, one pass: rank p's token t goes once to every rank r owning
// one of its experts, at before[p][r] + (its row in p's de-duplicated
// layout) - dest_offsets_p[r]; lane r < P forms that row (recv_row[p, t, r],
// -1 for none).
template <int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void ep_dedup_dispatch_rows(EpArgs a) {
    if (!*a.fits) return;  // uniform: nothing is written
    const int P = a.P;
    const uint32_t w = wave_index();
    const uint64_t per_rank = static_cast<uint64_t>(a.T) * a.slices;
    if (w >= per_rank * P) return;
    const uint32_t p = static_cast<uint32_t>(w / per_rank);
    const uint32_t rem = static_cast<uint32_t>(w - p * per_rank);
    const uint32_t t = rem / a.slices, slice = rem - t * a.slices;
    const uint32_t lane = lane_index();
    int row = -1;
    if (lane < static_cast<uint32_t>(P)) {
        const int64_t j = static_cast<int64_t>(t) * P + lane;
        const int lr = a.lrank[p][j];
        if (lr >= 0) {
            const int64_t rr = a.before[p * P + lane] + a.tile_base[p][static_cast<int64_t>(t / kWave) * P + lane] + lr;
            row = (rr >= 0 && rr < a.capacity) ? static_cast<int>(rr) : -1;
        }
        if (slice == 0) a.recv_pos[static_cast<int64_t>(p) * a.T * P + j] = row;
    }
    const uint64_t row_bytes = static_cast<uint64_t>(a.H) * 2;
    copy_row_to_slots<U, NTL, NTS>(a.x[p] + t * row_bytes, row_bytes, slice, P, lane, [&](int r) -> char* {
        const int rr = __builtin_amdgcn_readlane(row, r);
        return rr < 0 ? nullptr : a.dst[r] + static_cast<uint64_t>(rr) * row_bytes;
    });
}

// Its combine: rank p's token t sums, in rank order, the partial output of
// every rank r with recv_row[p, t, r] >= 0, read from r's buffer.
template <int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void ep_dedup_combine_rows(EpArgs a) {
    const uint32_t w = wave_index();
    const uint64_t per_rank = static_cast<uint64_t>(a.T) * a.slices;
    if (w >= per_rank * a.P) return;
    const uint32_t p = static_cast<uint32_t>(w / per_rank);
    const uint32_t rem = static_cast<uint32_t>(w - p * per_rank);
    const uint32_t t = rem / a.slices, slice = rem - t * a.slices;
    const uint32_t lane = lane_index();
    const int P = a.P;
    int row = -1;
    if (lane < static_cast<uint32_t>(P)) {
        const int64_t rr = a.recv_pos[(static_cast<int64_t>(p) * a.T + t) * P + lane];
        if (rr >= 0 && rr < a.capacity) {
            row = static_cast<int>(rr);
        } else if (rr != -1 && a.status && slice == 0) {
            atomicOr(a.status, 1);
        }
    }
    const uint64_t row_bytes = static_cast<uint64_t>(a.H) * 2;
    combine_slots<U, NTL, NTS, false>(
        [&](int r) -> const char* {
            const int rr = __builtin_amdgcn_readlane(row, r);
            return rr < 0 ? nullptr : a.x[r] + static_cast<uint64_t>(rr) * row_bytes;
        },
        1.0f, P, a.dst[p] + t * row_bytes, row_bytes, slice, lane);
}

// Launch shapes and cache hints, measured on MI355X: the packed rows and
// the expert outputs are streams far larger than the last-level cache.
// One 16-byte vector per lane, 1 KiB column slices: many short waves hide
// the row loads best (pack 4% and the de-duplicated pack 22% faster than
// 8 KiB slices, measured in the bench pipeline at 4096 x 7168, K = 8).
// The pack reads its token rows non-temporally: in a cycle of
// ReduceScatter, AllGather (P = 8, 256 MiB per rank), pack and combine, the
// rows kernel takes the same time either way but the AllGather after it
// (which reads the ReduceScatter's output, written with cached stores) ran
// 14 us faster and the cycle 1003 -> 986 us, the 56 MiB token matrix no
// longer taking last-level cache space.  The de-duplicated and
// expert-parallel dispatches keep cached loads (de-duplicated pack of 8
// ranks 445 -> 470 us with non-temporal ones).  A wave per (token, slot)
// writing whole 14 KiB rows measured 10% faster than the slices after an
// AllGather alone but made the cycle slower (1000 -> 1030 us).
constexpr int kPackUnroll = 1;
constexpr int kDedupUnroll = 1;
// Token matrices read ahead by the pack's metadata launches: from 8 MiB
// (below, the rows kernel is latency-bound) to 128 MiB (half the 256 MB
// last-level cache, so the matrix survives until the rows kernel reads it).
constexpr uint64_t kPrefetchMinBytes = uint64_t(8) << 20;
constexpr uint64_t kPrefetchMaxBytes = uint64_t(128) << 20;
// The one-pass pack: a grid of one workgroup per compute unit of MI355X
// (256); at most two rounds of it.
constexpr int kOneGroups = 256;
constexpr int kOneMaxGroups = 2 * kOneGroups;
constexpr bool kPackNtLoad = true;
constexpr bool kDispatchNtLoad = false;  // de-duplicated and expert-parallel dispatch rows
constexpr bool kPackNtStore = true;
constexpr int kUnpackUnroll = 1;
constexpr bool kUnpackNtLoad = true;
constexpr bool kUnpackNtStore = true;

// Column slices per token: U * 64 vectors each; rows that are not a
// multiple of 16 bytes are handled by one wave per token.
int row_slices(int H, int U) {
    const uint64_t row_bytes = static_cast<uint64_t>(H) * 2;
    if (row_bytes % 16 != 0) return 1;
    const uint64_t nvec = row_bytes / 16, per = static_cast<uint64_t>(U) * kWave;
    return static_cast<int>((nvec + per - 1) / per);
}

uint64_t align256(uint64_t b) { return (b + 255) & ~uint64_t(255); }

}  // namespace

bool moe_launch_fits(int T, int H) {
    // one wave per (token, slice); wave ids are 32-bit
    const uint64_t waves = static_cast<uint64_t>(T) * std::max({row_slices(H, kPackUnroll), row_slices(H, kDedupUnroll),
                                                                row_slices(H, kUnpackUnroll)});
    return waves < (uint64_t(1) << 31);
}

uint64_t pack_workspace_bytes(int T, int K, int E) {
    const uint64_t ntiles = (static_cast<uint64_t>(T) + kPackTileTokens - 1) / kPackTileTokens;
    return align256(4 * ntiles * E) + align256(4 * static_cast<uint64_t>(T) * K) + align256(4 * ntiles);
}

PackWorkspace pack_workspace_carve(void* base, int T, int K, int E) {
    const uint64_t ntiles = (static_cast<uint64_t>(T) + kPackTileTokens - 1) / kPackTileTokens;
    char* p = static_cast<char*>(base);
    PackWorkspace ws{};
    ws.tile_base = reinterpret_cast<int32_t*>(p);
    p += align256(4 * ntiles * E);
    ws.lrank = reinterpret_cast<int32_t*>(p);
    p += align256(4 * static_cast<uint64_t>(T) * K);
    ws.tile_err = reinterpret_cast<int32_t*>(p);
    return ws;
}

hipError_t launch_pack_meta(int T, int K, int E, int P, const int32_t* ids, int32_t* dest_counts,
                            int32_t* dest_offsets, int32_t* expert_counts, int32_t* expert_offsets, int32_t* dev_status,
                            const PackWorkspace& ws, hipStream_t stream, const void* prefetch,
                            uint64_t prefetch_bytes) {
    const int ntiles = (T + kPackTileTokens - 1) / kPackTileTokens;
    // The token matrix, when given and of a size the last-level cache holds
    // well, is read by extra workgroups of both launches: the first 2/5 with
    // the tiles, the rest with the scan, one pass of four 16-byte loads per
    // thread.  Measured on MI355X in the bench step (4096 x 7168 bf16,
    // after a 2 GiB AllGather): rows kernel 103 -> 89 us, tiles 4.6 -> 8.5
    // us, scan 6.7 -> 13.5 us, the pack 115 -> 111 us (the metadata's
    // dependent loads slow down under the read traffic, so the matrix's
    // 8-9 us of reading is only partly hidden); the whole matrix read with
    // the tiles instead: 15.4 + 7.3 + 92.7 us.
    Prefetch pt{}, ps{};
    if (prefetch && ntiles > 0 && prefetch_bytes >= kPrefetchMinBytes && prefetch_bytes <= kPrefetchMaxBytes) {
        const uint64_t cut = prefetch_bytes * 2 / 5 / 16 * 16;
        const auto blocks = [](uint64_t bytes, uint32_t threads, uint32_t most) {
            const uint64_t per = static_cast<uint64_t>(threads) * 64;  // four 16-byte loads per thread
            return static_cast<uint32_t>(std::min<uint64_t>(most, (bytes + per - 1) / per));
        };
        pt = Prefetch{static_cast<const char*>(prefetch), 0, cut, blocks(cut, kBlock, 4096)};
        ps = Prefetch{static_cast<const char*>(prefetch), cut, prefetch_bytes / 16 * 16,
                      blocks(prefetch_bytes - cut, kScanThreads, 768)};
    }
    (void)hipGetLastError();
    if (ntiles > 0) {
        RankIds rids{};
        rids.ids[0] = ids;
        hipLaunchKernelGGL(pack_tiles, dim3(ntiles + pt.blocks), dim3(kBlock), static_cast<size_t>(E) * 8, stream, T,
                           K, E, rids, ws.tile_base, ws.lrank, ws.tile_err, uint64_t(0), pt);
    }
    hipLaunchKernelGGL(pack_scan, dim3(1 + ps.blocks), dim3(kScanThreads), 0, stream, ntiles, E, P, ws.tile_base,
                       ws.tile_err, expert_counts, expert_offsets, dest_counts, dest_offsets, dev_status, uint64_t(0),
                       ps);
    return hipGetLastError();
}

hipError_t launch_pack_rows(int T, int H, int K, int E, const uint16_t* x, const int32_t* ids, uint16_t* packed,
                            int32_t* pos, const PackWorkspace& ws, hipStream_t stream) {
    (void)hipGetLastError();
    if (T > 0) {
        const int slices = row_slices(H, kPackUnroll);
        const uint64_t waves = static_cast<uint64_t>(T) * slices;
        const dim3 grid(static_cast<uint32_t>((waves + kWavesPerBlock - 1) / kWavesPerBlock));
        hipLaunchKernelGGL((pack_rows<kPackUnroll, kPackNtLoad, kPackNtStore>), grid, dim3(kBlock), 0, stream, T, H,
                           K, E, slices, reinterpret_cast<const char*>(x), ids, ws.tile_base, ws.lrank, pos,
                           reinterpret_cast<char*>(packed));
    }
    return hipGetLastError();
}

int pack_onepass_tokens(int T, int H, int K, int E) {
    const uint64_t row_bytes = static_cast<uint64_t>(H) * 2;
    if (T < 1 || row_bytes % 16 != 0 || E > kOneMaxExperts) return 0;
    if (static_cast<int64_t>(T) * K > kOneMaxIds || T * K < 4) return 0;
    const uint64_t nvec = row_bytes / 16;
    const uint64_t most = static_cast<uint64_t>(kOneVec) * kOneThreads;  // x vectors a workgroup holds
    if (nvec > most) return 0;
    // as many workgroups as compute units, fewer tokens each when the rows
    // do not fit the registers, the token masks (64 bits) or the position
    // table (then the grid runs in more than one round)
    const uint64_t tw = std::min<uint64_t>({(static_cast<uint64_t>(T) + kOneGroups - 1) / kOneGroups, most / nvec,
                                            uint64_t(64), static_cast<uint64_t>(kOneMaxOwn / K)});
    if (tw < 1 || (static_cast<uint64_t>(T) + tw - 1) / tw > kOneMaxGroups) return 0;
    return static_cast<int>(tw);
}

hipError_t launch_pack(int T, int H, int K, int E, int P, const uint16_t* x, const int32_t* ids, uint16_t* packed,
                       int32_t* dest_counts, int32_t* dest_offsets, int32_t* expert_counts, int32_t* expert_offsets,
                       int32_t* pos, int32_t* dev_status, const PackWorkspace& ws, hipStream_t stream,
                       uint64_t* rec) {
    if (const int tw = pack_onepass_tokens(T, H, K, E)) {
        (void)hipGetLastError();
        const uint32_t nvec = static_cast<uint32_t>(static_cast<uint64_t>(H) * 2 / 16);
        const auto kernel = K <= kOneUnrolledSlots ? pack_onepass<kOneUnrolledSlots, kPackNtLoad, kPackNtStore>
                                                   : pack_onepass<0, kPackNtLoad, kPackNtStore>;
        int copies = kOneMaxCopies;
        while (copies > 1 && static_cast<uint64_t>(copies) * (2 * E + 1) * 4 > kOneCopyBytes) copies /= 2;
        const size_t lds = static_cast<size_t>(copies) * (2 * E + 1) * 4;
        hipLaunchKernelGGL(kernel, dim3((T + tw - 1) / tw), dim3(kOneThreads), lds, stream, T, K, E, P, tw, nvec,
                           copies, reinterpret_cast<const char*>(x), ids, reinterpret_cast<char*>(packed), pos,
                           expert_counts, expert_offsets, dest_counts, dest_offsets, dev_status, rec,
                           rec ? wall_clock_khz() : 0);
        return hipGetLastError();
    }
    const hipError_t e = launch_pack_meta(T, K, E, P, ids, dest_counts, dest_offsets, expert_counts, expert_offsets,
                                          dev_status, ws, stream, x, static_cast<uint64_t>(T) * H * 2);
    if (e != hipSuccess) return e;
    return launch_pack_rows(T, H, K, E, x, ids, packed, pos, ws, stream);
}

hipError_t launch_unpack(int T, int H, int K, const uint16_t* y, const int32_t* pos, const float* gates, uint16_t* out,
                         int32_t* dev_status, hipStream_t stream) {
    (void)hipGetLastError();
    if (dev_status) hipLaunchKernelGGL(set_status, dim3(1), dim3(1), 0, stream, dev_status);
    if (T > 0) {
        const int slices = row_slices(H, kUnpackUnroll);
        const uint64_t waves = static_cast<uint64_t>(T) * slices;
        const dim3 grid(static_cast<uint32_t>((waves + kWavesPerBlock - 1) / kWavesPerBlock));
        hipLaunchKernelGGL((unpack_rows<kUnpackUnroll, kUnpackNtLoad, kUnpackNtStore, true>), grid, dim3(kBlock), 0,
                           stream, T, H, K, slices, static_cast<int64_t>(T) * K, reinterpret_cast<const char*>(y), pos,
                           gates, reinterpret_cast<char*>(out), dev_status);
    }
    return hipGetLastError();
}

uint64_t pack_dedup_workspace_bytes(int T, int P) {
    const uint64_t ntiles = (static_cast<uint64_t>(T) + kWave - 1) / kWave;
    return align256(4 * ntiles * P) + align256(4 * static_cast<uint64_t>(T) * P) + align256(4 * ntiles);
}

hipError_t launch_pack_dedup(int T, int H, int K, int E, int P, const uint16_t* x, const int32_t* ids,
                             uint16_t* packed, int32_t* dest_counts, int32_t* dest_offsets, int32_t* row_of,
                             int32_t* dev_status, void* workspace, hipStream_t stream) {
    const int ntiles = (T + kWave - 1) / kWave;
    char* ws = static_cast<char*>(workspace);
    int32_t* tile_base = reinterpret_cast<int32_t*>(ws);
    int32_t* lrank = reinterpret_cast<int32_t*>(ws + align256(4 * static_cast<uint64_t>(ntiles) * P));
    int32_t* tile_err = reinterpret_cast<int32_t*>(ws + align256(4 * static_cast<uint64_t>(ntiles) * P) +
                                                   align256(4 * static_cast<uint64_t>(T) * P));
    (void)hipGetLastError();
    if (ntiles > 0) {
        RankIds rids{};
        rids.ids[0] = ids;
        hipLaunchKernelGGL(dedup_tiles, dim3(ntiles), dim3(kBlock), 0, stream, T, K, E, P, rids, tile_base, lrank,
                           tile_err, uint64_t(0));
    }
    hipLaunchKernelGGL(dedup_scan, dim3(1), dim3(kScanThreads), 0, stream, ntiles, P, tile_base, tile_err, dest_counts,
                       dest_offsets, dev_status, uint64_t(0));
    if (T > 0) {
        const int slices = row_slices(H, kDedupUnroll);
        const uint64_t waves = static_cast<uint64_t>(T) * slices;
        const dim3 grid(static_cast<uint32_t>((waves + kWavesPerBlock - 1) / kWavesPerBlock));
        hipLaunchKernelGGL((dedup_rows<kDedupUnroll, kDispatchNtLoad, kPackNtStore>), grid, dim3(kBlock), 0, stream, T, H,
                           P, slices, reinterpret_cast<const char*>(x), tile_base, lrank, dest_offsets, row_of,
                           reinterpret_cast<char*>(packed));
    }
    return hipGetLastError();
}

hipError_t launch_unpack_dedup(int T, int H, int P, int64_t rows, const uint16_t* y, const int32_t* row_of,
                               uint16_t* out, int32_t* dev_status, hipStream_t stream) {
    (void)hipGetLastError();
    if (dev_status) hipLaunchKernelGGL(set_status, dim3(1), dim3(1), 0, stream, dev_status);
    if (T > 0) {
        const int slices = row_slices(H, kUnpackUnroll);
        const uint64_t waves = static_cast<uint64_t>(T) * slices;
        const dim3 grid(static_cast<uint32_t>((waves + kWavesPerBlock - 1) / kWavesPerBlock));
        hipLaunchKernelGGL((unpack_rows<kUnpackUnroll, kUnpackNtLoad, kUnpackNtStore, false>), grid, dim3(kBlock), 0,
                           stream, T, H, P, slices, rows, reinterpret_cast<const char*>(y), row_of, nullptr,
                           reinterpret_cast<char*>(out), dev_status);
    }
    return hipGetLastError();
}

// Both one-pass dispatches end their workspace with before[P][P] (int64)
// and the capacity verdict.
uint64_t ep_tail_bytes(int P) {
    const uint64_t Pu = static_cast<uint64_t>(P);
    return align256(8 * Pu * Pu) + align256(4);
}

uint64_t ep_dispatch_workspace_bytes(int T, int K, int E, int P) {
    const uint64_t Pu = static_cast<uint64_t>(P);
    return Pu * pack_workspace_bytes(T, K, E) + align256(4 * Pu * Pu) + align256(4 * Pu * E) + align256(4 * Pu) +
           ep_tail_bytes(P);
}

hipError_t launch_ep_dispatch(int T, int H, int K, int E, int P, const uint16_t* const* x, const int32_t* const* ids,
                              uint16_t* const* recv, int64_t capacity, int32_t* counts, int32_t* recv_pos,
                              int32_t* dev_status, void* workspace, hipStream_t stream) {
    const uint64_t Pu = static_cast<uint64_t>(P);
    const uint64_t per = pack_workspace_bytes(T, K, E);
    char* ws = static_cast<char*>(workspace);
    int32_t* dest_off = reinterpret_cast<int32_t*>(ws + Pu * per);                          // [P][P]
    int32_t* expert_counts = reinterpret_cast<int32_t*>(ws + Pu * per + align256(4 * Pu * Pu));  // [P][E]
    int32_t* words = reinterpret_cast<int32_t*>(ws + Pu * per + align256(4 * Pu * Pu) + align256(4 * Pu * E));
    char* tail = ws + Pu * per + align256(4 * Pu * Pu) + align256(4 * Pu * E) + align256(4 * Pu);
    int64_t* before = reinterpret_cast<int64_t*>(tail);
    int32_t* fits = reinterpret_cast<int32_t*>(tail + align256(8 * Pu * Pu));
    const int ntiles = (T + kPackTileTokens - 1) / kPackTileTokens;
    EpArgs a{};
    RankIds rids{};
    (void)hipGetLastError();
    // every rank's metadata in one launch of each kind (rank p's workspace
    // at ws + p * per, its outputs at row p)
    const PackWorkspace w0 = pack_workspace_carve(ws, T, K, E);
    for (int p = 0; p < P; ++p) rids.ids[p] = ids[p];
    if (ntiles > 0)
        hipLaunchKernelGGL(pack_tiles, dim3(ntiles, P), dim3(kBlock), static_cast<size_t>(E) * 8, stream, T, K, E, rids,
                           w0.tile_base, w0.lrank, w0.tile_err, per, Prefetch{});
    hipLaunchKernelGGL(pack_scan, dim3(P), dim3(kScanThreads), 0, stream, ntiles, E, P, w0.tile_base, w0.tile_err,
                       expert_counts, static_cast<int32_t*>(nullptr), counts, dest_off, words, per, Prefetch{});
    hipLaunchKernelGGL(ep_prefix, dim3(1), dim3(kBlock), 0, stream, counts, P, capacity, before, fits, words,
                       dev_status);
    for (int p = 0; p < P; ++p) {
        const PackWorkspace w = pack_workspace_carve(ws + p * per, T, K, E);
        a.x[p] = reinterpret_cast<const char*>(x[p]);
        a.ids[p] = ids[p];
        a.dst[p] = reinterpret_cast<char*>(recv[p]);
        a.tile_base[p] = w.tile_base;
        a.lrank[p] = w.lrank;
        a.dest_off[p] = dest_off + p * P;
    }
    if (T > 0) {
        a.counts = counts;
        a.before = before;
        a.fits = fits;
        a.recv_pos = recv_pos;
        a.status = dev_status;
        a.capacity = capacity;
        a.T = T;
        a.H = H;
        a.K = K;
        a.E = E;
        a.P = P;
        a.slices = row_slices(H, kPackUnroll);
        const uint64_t waves = Pu * static_cast<uint64_t>(T) * a.slices;
        const dim3 grid(static_cast<uint32_t>((waves + kWavesPerBlock - 1) / kWavesPerBlock));
        hipLaunchKernelGGL((ep_dispatch_rows<kPackUnroll, kDispatchNtLoad, kPackNtStore>), grid, dim3(kBlock), 0, stream,
                           a);
    }
    return hipGetLastError();
}

hipError_t launch_ep_combine(int T, int H, int K, int E, int P, const uint16_t* const* y, int64_t capacity,
                             const int32_t* const* ids, const int32_t* recv_pos, const float* const* gates,
                             uint16_t* const* out, int32_t* dev_status, hipStream_t stream) {
    EpArgs a{};
    for (int p = 0; p < P; ++p) {
        a.x[p] = reinterpret_cast<const char*>(y[p]);
        a.ids[p] = ids[p];
        a.dst[p] = reinterpret_cast<char*>(out[p]);
        a.gates[p] = gates[p];
    }
    a.recv_pos = const_cast<int32_t*>(recv_pos);  // read only here
    a.status = dev_status;
    a.capacity = capacity;
    a.T = T;
    a.H = H;
    a.K = K;
    a.E = E;
    a.P = P;
    a.slices = row_slices(H, kUnpackUnroll);
    (void)hipGetLastError();
    if (dev_status) hipLaunchKernelGGL(set_status, dim3(1), dim3(1), 0, stream, dev_status);
    if (T > 0) {
        const uint64_t waves = static_cast<uint64_t>(P) * T * a.slices;
        const dim3 grid(static_cast<uint32_t>((waves + kWavesPerBlock - 1) / kWavesPerBlock));
        hipLaunchKernelGGL((ep_combine_rows<kUnpackUnroll, kUnpackNtLoad, kUnpackNtStore>), grid, dim3(kBlock), 0,
                           stream, a);
    }
    return hipGetLastError();
}

bool ep_launch_fits(int T, int H, int P) {
    const uint64_t slices = std::max(row_slices(H, kPackUnroll), row_slices(H, kUnpackUnroll));
    return static_cast<uint64_t>(P) * T * slices < (uint64_t(1) << 31);
}

uint64_t ep_dispatch_dedup_workspace_bytes(int T, int P) {
    const uint64_t Pu = static_cast<uint64_t>(P);
    return Pu * pack_dedup_workspace_bytes(T, P) + align256(4 * Pu * Pu) + align256(4 * Pu) + ep_tail_bytes(P);
}

hipError_t launch_ep_dispatch_dedup(int T, int H, int K, int E, int P, const uint16_t* const* x,
                                    const int32_t* const* ids, uint16_t* const* recv, int64_t capacity,
                                    int32_t* counts, int32_t* recv_row, int32_t* dev_status, void* workspace,
                                    hipStream_t stream) {
    const uint64_t Pu = static_cast<uint64_t>(P);
    const uint64_t per = pack_dedup_workspace_bytes(T, P);
    const int ntiles = (T + kWave - 1) / kWave;
    const uint64_t nt = static_cast<uint64_t>(ntiles);
    char* ws = static_cast<char*>(workspace);
    int32_t* dest_off = reinterpret_cast<int32_t*>(ws + Pu * per);  // [P][P]
    int32_t* words = reinterpret_cast<int32_t*>(ws + Pu * per + align256(4 * Pu * Pu));
    char* tail = ws + Pu * per + align256(4 * Pu * Pu) + align256(4 * Pu);
    int64_t* before = reinterpret_cast<int64_t*>(tail);
    int32_t* fits = reinterpret_cast<int32_t*>(tail + align256(8 * Pu * Pu));
    EpArgs a{};
    RankIds rids{};
    (void)hipGetLastError();
    // rank p's dedup workspace at ws + p * per: tile bases, local ranks, error flags
    const uint64_t lrank_at = align256(4 * nt * Pu);
    const uint64_t err_at = lrank_at + align256(4 * uint64_t(T) * Pu);
    for (int p = 0; p < P; ++p) rids.ids[p] = ids[p];
    if (ntiles > 0)
        hipLaunchKernelGGL(dedup_tiles, dim3(ntiles, P), dim3(kBlock), 0, stream, T, K, E, P, rids,
                           reinterpret_cast<int32_t*>(ws), reinterpret_cast<int32_t*>(ws + lrank_at),
                           reinterpret_cast<int32_t*>(ws + err_at), per);
    hipLaunchKernelGGL(dedup_scan, dim3(P), dim3(kScanThreads), 0, stream, ntiles, P, reinterpret_cast<int32_t*>(ws),
                       reinterpret_cast<const int32_t*>(ws + err_at), counts, dest_off, words, per);
    hipLaunchKernelGGL(ep_prefix, dim3(1), dim3(kBlock), 0, stream, counts, P, capacity, before, fits, words,
                       dev_status);
    for (int p = 0; p < P; ++p) {
        char* base = ws + p * per;
        int32_t* tile_base = reinterpret_cast<int32_t*>(base);
        int32_t* lrank = reinterpret_cast<int32_t*>(base + lrank_at);
        a.x[p] = reinterpret_cast<const char*>(x[p]);
        a.dst[p] = reinterpret_cast<char*>(recv[p]);
        a.tile_base[p] = tile_base;
        a.lrank[p] = lrank;
        a.dest_off[p] = dest_off + p * P;
    }
    if (T > 0) {
        a.counts = counts;
        a.before = before;
        a.fits = fits;
        a.recv_pos = recv_row;
        a.status = dev_status;
        a.capacity = capacity;
        a.T = T;
        a.H = H;
        a.K = K;
        a.E = E;
        a.P = P;
        a.slices = row_slices(H, kDedupUnroll);
        const uint64_t waves = Pu * static_cast<uint64_t>(T) * a.slices;
        const dim3 grid(static_cast<uint32_t>((waves + kWavesPerBlock - 1) / kWavesPerBlock));
        hipLaunchKernelGGL((ep_dedup_dispatch_rows<kDedupUnroll, kDispatchNtLoad, kPackNtStore>), grid, dim3(kBlock), 0,
                           stream, a);
    }
    return hipGetLastError();
}

hipError_t launch_ep_combine_dedup(int T, int H, int P, const uint16_t* const* y, int64_t capacity,
                                   const int32_t* recv_row, uint16_t* const* out, int32_t* dev_status,
                                   hipStream_t stream) {
    EpArgs a{};
    for (int p = 0; p < P; ++p) {
        a.x[p] = reinterpret_cast<const char*>(y[p]);
        a.dst[p] = reinterpret_cast<char*>(out[p]);
    }
    a.recv_pos = const_cast<int32_t*>(recv_row);  // read only here
    a.status = dev_status;
    a.capacity = capacity;
    a.T = T;
    a.H = H;
    a.P = P;
    a.slices = row_slices(H, kUnpackUnroll);
    (void)hipGetLastError();
    if (dev_status) hipLaunchKernelGGL(set_status, dim3(1), dim3(1), 0, stream, dev_status);
    if (T > 0) {
        const uint64_t waves = static_cast<uint64_t>(P) * T * a.slices;
        const dim3 grid(static_cast<uint32_t>((waves + kWavesPerBlock - 1) / kWavesPerBlock));
        hipLaunchKernelGGL((ep_dedup_combine_rows<kUnpackUnroll, kUnpackNtLoad, kUnpackNtStore>), grid, dim3(kBlock),
                           0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace purlin
